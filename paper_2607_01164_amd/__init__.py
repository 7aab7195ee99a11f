"""Point sampling of a learned 3D-Gaussian scalar field (W-VEG) on AMD
Instinct MI355X: a C-ABI HIP library (include/gs.h, include/gs_train.h,
csrc/) and its Python binding (gsq)."""
from .gsq import (GS_ERR_CAPACITY, GS_ERR_HIP, GS_ERR_INVALID_ARGUMENT, GS_ERR_WORKSPACE, GS_OK,  # noqa: F401
                  GS_QUERY_GRID, GS_QUERY_JITTER, GS_QUERY_POINTS, GS_QUERY_VOXELS, Gaussians, Grads, GsError, GsLibraryMissing,
                  Index, Query, alloc_backward_work, alloc_plan, backward_work_bytes, build_index, gs_build_index,
                  gs_sample, gs_sample_backward, load_library, make_grid, plan_bytes, profile_enable,
                  profile_read, profile_reset, profile_select, RawParams, alloc_loss_terms, alloc_loss_work,
                  gs_activate, gs_activate_backward, gs_loss, loss_work_bytes, read_loss_terms, ParamSet,
                  alloc_densify_work, densify_work_bytes, gs_densify, alloc_gaussian_major_work,
                  gaussian_major_work_bytes, gs_sample_gaussian_major, backward_pair_count,
                  sample_pair_counts, gs_sample_backward_noalloc, gs_plan_queries, gs_sample_planned)
