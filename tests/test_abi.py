"""The C-ABI library loads and exports every function include/*.h declares,
and its host-side validation rejects malformed arguments before any device
work (no GPU needed: nothing here launches a kernel)."""
import ctypes
import os
import re

import pytest

import paper_2607_01164_amd as gs
from paper_2607_01164_amd import gsq

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SIZE_ERR = ctypes.c_size_t(-1).value


def declared_functions():
    inc = os.path.join(ROOT, "include")
    text = "".join(open(os.path.join(inc, f)).read() for f in sorted(os.listdir(inc)) if f.endswith(".h"))
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gs_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("gs_build_index", "gs_sample", "gs_sample_backward", "gs_last_error"):
        assert n in names
    assert set(names) == set(gsq.EXPORTED)


def test_library_exports_every_declared_symbol():
    L = gs.load_library()
    for n in declared_functions():
        assert hasattr(L, n), n
    assert L.gs_version() >= 100


def test_nm_lists_the_symbols():
    import subprocess
    out = subprocess.run(["nm", "-D", "--defined-only", gsq.LIB_PATH], capture_output=True, text=True).stdout
    for n in declared_functions():
        assert re.search(rf"\bT {n}\b", out), n


def grid(cells=(8, 8, 8), lo=(0, 0, 0), hi=(1, 1, 1)):
    return gs.make_grid(cells, lo, hi)


def test_sizing_functions():
    L = gs.load_library()
    g = grid()
    a = L.gs_index_work_bytes(1000, ctypes.byref(g), 10000)
    b = L.gs_index_work_bytes(2000, ctypes.byref(g), 10000)
    c = L.gs_index_work_bytes(1000, ctypes.byref(g), 20000)
    assert 0 < a < b and a < c and a % 256 == 0
    assert L.gs_index_work_bytes(-1, ctypes.byref(g), 10) == SIZE_ERR
    assert L.gs_index_work_bytes(10, ctypes.byref(grid((0, 8, 8))), 10) == SIZE_ERR
    assert L.gs_index_work_bytes(10, ctypes.byref(grid(hi=(1, 0, 1))), 10) == SIZE_ERR
    qg = gsq.GsQuery(gs.GS_QUERY_GRID, (ctypes.c_int32 * 3)(32, 32, 32), 0, None, None)
    assert L.gs_plan_bytes(ctypes.byref(qg), ctypes.byref(g)) == 0
    assert L.gs_query_size(ctypes.byref(qg)) == 32 ** 3
    qp = gsq.GsQuery(gs.GS_QUERY_POINTS, (ctypes.c_int32 * 3)(0, 0, 0), 1000, None, 4096)
    assert L.gs_plan_bytes(ctypes.byref(qp), ctypes.byref(g)) > 1000 * 16
    assert L.gs_query_size(ctypes.byref(qp)) == 1000
    bad = gsq.GsQuery(7, (ctypes.c_int32 * 3)(0, 0, 0), 10, None, None)
    assert L.gs_query_size(ctypes.byref(bad)) == -1
    nullpts = gsq.GsQuery(gs.GS_QUERY_POINTS, (ctypes.c_int32 * 3)(0, 0, 0), 10, None, None)
    assert L.gs_query_size(ctypes.byref(nullpts)) == -1
    empty = gsq.GsQuery(gs.GS_QUERY_POINTS, (ctypes.c_int32 * 3)(0, 0, 0), 0, None, None)
    assert L.gs_query_size(ctypes.byref(empty)) == 0


def test_jitter_query_validation():
    """Training-sample queries: offsets required; without voxel ids the query
    covers every voxel, so n must be the voxel count."""
    L = gs.load_library()
    g = grid()
    dims = (ctypes.c_int32 * 3)(16, 8, 4)
    full = gsq.GsQuery(gs.GS_QUERY_JITTER, dims, 16 * 8 * 4, None, FAKE)
    assert L.gs_query_size(ctypes.byref(full)) == 16 * 8 * 4
    assert L.gs_plan_bytes(ctypes.byref(full), ctypes.byref(g)) > 512 * 16
    listed = gsq.GsQuery(gs.GS_QUERY_JITTER, dims, 100, FAKE, FAKE)
    assert L.gs_query_size(ctypes.byref(listed)) == 100
    short = gsq.GsQuery(gs.GS_QUERY_JITTER, dims, 100, None, FAKE)
    assert L.gs_query_size(ctypes.byref(short)) == -1
    no_offsets = gsq.GsQuery(gs.GS_QUERY_JITTER, dims, 100, FAKE, None)
    assert L.gs_query_size(ctypes.byref(no_offsets)) == -1
    bad_dims = gsq.GsQuery(gs.GS_QUERY_JITTER, (ctypes.c_int32 * 3)(16, 0, 4), 100, FAKE, FAKE)
    assert L.gs_query_size(ctypes.byref(bad_dims)) == -1


FAKE = 1 << 20  # a non-null, 256-aligned address that validation never dereferences


def fake_gauss(n=10):
    return gsq.GsGaussians(n, FAKE, FAKE, FAKE, FAKE, FAKE)


def fake_index(capacity=100, work_bytes=1 << 30):
    return gsq.GsIndex(FAKE, FAKE, FAKE, capacity, FAKE, work_bytes, -1, 0, grid(), 0.0)


def call_build(gauss, g, tau, idx):
    L = gs.load_library()
    return L.gs_build_index(None if gauss is None else ctypes.byref(gauss), None if g is None else ctypes.byref(g),
                            tau, None if idx is None else ctypes.byref(idx), None)


@pytest.mark.parametrize("case", ["null_gauss", "neg_n", "null_param", "null_grid", "bad_cells", "flat_box",
                                  "nan_box", "tau_zero", "tau_one", "null_index", "neg_capacity", "null_offsets",
                                  "null_keys"])
def test_build_index_rejects_bad_arguments(case):
    L = gs.load_library()
    gauss, g, tau, idx = fake_gauss(), grid(), 0.01, fake_index()
    if case == "null_gauss":
        gauss = None
    elif case == "neg_n":
        gauss = fake_gauss(-1)
    elif case == "null_param":
        gauss = gsq.GsGaussians(5, FAKE, None, FAKE, FAKE, FAKE)
    elif case == "null_grid":
        g = None
    elif case == "bad_cells":
        g = grid((8, -1, 8))
    elif case == "flat_box":
        g = grid(lo=(0, 0.5, 0), hi=(1, 0.5, 1))
    elif case == "nan_box":
        g = grid(lo=(float("nan"), 0, 0))
    elif case == "tau_zero":
        tau = 0.0
    elif case == "tau_one":
        tau = 1.0
    elif case == "null_index":
        idx = None
    elif case == "neg_capacity":
        idx = fake_index(capacity=-5)
    elif case == "null_offsets":
        idx = fake_index()
        idx.cell_offsets = None
    elif case == "null_keys":
        idx = fake_index()
        idx.keys = None
    st = call_build(gauss, g, tau, idx)
    assert st == gs.GS_ERR_INVALID_ARGUMENT
    assert L.gs_last_error().decode().startswith("gs_build_index")


def test_build_index_rejects_small_or_misaligned_workspace():
    L = gs.load_library()
    st = call_build(fake_gauss(), grid(), 0.01, fake_index(work_bytes=1000))
    assert st == gs.GS_ERR_WORKSPACE and b"workspace" in L.gs_last_error()
    idx = fake_index()
    idx.work = FAKE + 8
    assert call_build(fake_gauss(), grid(), 0.01, idx) == gs.GS_ERR_WORKSPACE


def test_sample_requires_a_built_index():
    L = gs.load_library()
    idx = fake_index()  # n_pairs = -1: never built
    q = gsq.GsQuery(gs.GS_QUERY_GRID, (ctypes.c_int32 * 3)(32, 32, 32), 0, None, None)
    st = L.gs_sample(ctypes.byref(fake_gauss()), ctypes.byref(idx), ctypes.byref(q), FAKE, FAKE, None, 0, None)
    assert st == gs.GS_ERR_INVALID_ARGUMENT and b"not been built" in L.gs_last_error()


def built_fake_index(n_gauss=10):
    idx = fake_index()
    idx.n_pairs = 50
    idx.n_gauss = n_gauss
    idx.tau = 0.01
    return idx


def test_sample_validates_queries():
    L = gs.load_library()
    idx = built_fake_index()
    # GRID dims must be multiples of the index cells
    q = gsq.GsQuery(gs.GS_QUERY_GRID, (ctypes.c_int32 * 3)(30, 32, 32), 0, None, None)
    st = L.gs_sample(ctypes.byref(fake_gauss()), ctypes.byref(idx), ctypes.byref(q), FAKE, FAKE, None, 0, None)
    assert st == gs.GS_ERR_INVALID_ARGUMENT and b"multiple" in L.gs_last_error()
    # Gaussian count must match the index
    q = gsq.GsQuery(gs.GS_QUERY_GRID, (ctypes.c_int32 * 3)(32, 32, 32), 0, None, None)
    st = L.gs_sample(ctypes.byref(fake_gauss(11)), ctypes.byref(idx), ctypes.byref(q), FAKE, FAKE, None, 0, None)
    assert st == gs.GS_ERR_INVALID_ARGUMENT and b"built for 10" in L.gs_last_error()
    # outputs must be given
    st = L.gs_sample(ctypes.byref(fake_gauss()), ctypes.byref(idx), ctypes.byref(q), None, FAKE, None, 0, None)
    assert st == gs.GS_ERR_INVALID_ARGUMENT
    # point queries need a plan of gs_plan_bytes
    qp = gsq.GsQuery(gs.GS_QUERY_POINTS, (ctypes.c_int32 * 3)(0, 0, 0), 100, None, FAKE)
    st = L.gs_sample(ctypes.byref(fake_gauss()), ctypes.byref(idx), ctypes.byref(qp), FAKE, FAKE, FAKE, 16, None)
    assert st == gs.GS_ERR_WORKSPACE and b"plan" in L.gs_last_error()
    # negative counts and unknown kinds
    qn = gsq.GsQuery(gs.GS_QUERY_POINTS, (ctypes.c_int32 * 3)(0, 0, 0), -3, None, FAKE)
    st = L.gs_sample(ctypes.byref(fake_gauss()), ctypes.byref(idx), ctypes.byref(qn), FAKE, FAKE, FAKE, 1 << 20, None)
    assert st == gs.GS_ERR_INVALID_ARGUMENT
    qk = gsq.GsQuery(9, (ctypes.c_int32 * 3)(0, 0, 0), 3, None, FAKE)
    st = L.gs_sample(ctypes.byref(fake_gauss()), ctypes.byref(idx), ctypes.byref(qk), FAKE, FAKE, FAKE, 1 << 20, None)
    assert st == gs.GS_ERR_INVALID_ARGUMENT


def test_plan_queries_and_sample_planned_validate_arguments():
    """The two halves of gs_sample check what gs_sample checks, before any
    device work; grid queries need no plan."""
    L = gs.load_library()
    g = grid((32, 32, 32))
    qg = gsq.GsQuery(gs.GS_QUERY_GRID, (ctypes.c_int32 * 3)(32, 32, 32), 0, None, None)
    assert L.gs_plan_queries(ctypes.byref(qg), ctypes.byref(g), None, 0, None) == gs.GS_OK
    qbad = gsq.GsQuery(gs.GS_QUERY_GRID, (ctypes.c_int32 * 3)(30, 32, 32), 0, None, None)
    st = L.gs_plan_queries(ctypes.byref(qbad), ctypes.byref(g), None, 0, None)
    assert st == gs.GS_ERR_INVALID_ARGUMENT and b"multiple" in L.gs_last_error()
    qp = gsq.GsQuery(gs.GS_QUERY_POINTS, (ctypes.c_int32 * 3)(0, 0, 0), 100, None, FAKE)
    st = L.gs_plan_queries(ctypes.byref(qp), ctypes.byref(g), FAKE, 16, None)
    assert st == gs.GS_ERR_WORKSPACE and b"plan" in L.gs_last_error()
    st = L.gs_plan_queries(ctypes.byref(qp), ctypes.byref(grid((1024, 1024, 1024))), FAKE, 1 << 40, None)
    assert st == gs.GS_ERR_INVALID_ARGUMENT and b"2^30" in L.gs_last_error()
    st = L.gs_plan_queries(None, ctypes.byref(g), FAKE, 1 << 20, None)
    assert st == gs.GS_ERR_INVALID_ARGUMENT
    idx = fake_index()  # never built
    st = L.gs_sample_planned(ctypes.byref(fake_gauss()), ctypes.byref(idx), ctypes.byref(qg), FAKE, FAKE, None, 0, None)
    assert st == gs.GS_ERR_INVALID_ARGUMENT and b"not been built" in L.gs_last_error()
    idx = built_fake_index()
    st = L.gs_sample_planned(ctypes.byref(fake_gauss()), ctypes.byref(idx), ctypes.byref(qp), FAKE, FAKE, FAKE, 16,
                             None)
    assert st == gs.GS_ERR_WORKSPACE and b"plan" in L.gs_last_error()
    st = L.gs_sample_planned(ctypes.byref(fake_gauss()), ctypes.byref(idx), ctypes.byref(qp), None, FAKE, FAKE,
                             1 << 20, None)
    assert st == gs.GS_ERR_INVALID_ARGUMENT


def test_ordered_queries_reject_grids_of_2_30_cells():
    """Voxel, point and jitter queries sort 32-bit keys 4 cell + quarter (the
    outside bucket last): a grid of 2^30 cells or more is refused before any
    device work, while grid queries may use it."""
    L = gs.load_library()
    big = grid((1024, 1024, 1024))
    ok = grid((1024, 1024, 1023))
    qp = gsq.GsQuery(gs.GS_QUERY_POINTS, (ctypes.c_int32 * 3)(0, 0, 0), 100, None, FAKE)
    assert L.gs_plan_bytes(ctypes.byref(qp), ctypes.byref(big)) == SIZE_ERR
    assert L.gs_plan_bytes(ctypes.byref(qp), ctypes.byref(ok)) != SIZE_ERR
    idx = built_fake_index()
    idx.grid = big
    st = L.gs_sample(ctypes.byref(fake_gauss()), ctypes.byref(idx), ctypes.byref(qp), FAKE, FAKE, FAKE, 1 << 40, None)
    assert st == gs.GS_ERR_INVALID_ARGUMENT and b"2^30" in L.gs_last_error()
    qv = gsq.GsQuery(gs.GS_QUERY_VOXELS, (ctypes.c_int32 * 3)(1024, 1024, 1024), 100, FAKE, None)
    st = L.gs_sample(ctypes.byref(fake_gauss()), ctypes.byref(idx), ctypes.byref(qv), FAKE, FAKE, FAKE, 1 << 40, None)
    assert st == gs.GS_ERR_INVALID_ARGUMENT and b"2^30" in L.gs_last_error()
    qg = gsq.GsQuery(gs.GS_QUERY_GRID, (ctypes.c_int32 * 3)(1024, 1024, 1024), 0, None, None)
    assert L.gs_plan_bytes(ctypes.byref(qg), ctypes.byref(big)) == 0


def test_pair_counts_validate_arguments():
    L = gs.load_library()
    t, c = ctypes.c_int64(7), ctypes.c_int64(7)
    q = gsq.GsQuery(gs.GS_QUERY_POINTS, (ctypes.c_int32 * 3)(0, 0, 0), 100, None, FAKE)
    st = L.gs_sample_pair_counts(ctypes.byref(fake_index()), ctypes.byref(q), FAKE, 1 << 30, FAKE, 1 << 30,
                                 ctypes.byref(t), ctypes.byref(c), None)
    assert st == gs.GS_ERR_INVALID_ARGUMENT and b"not built" in L.gs_last_error()
    assert t.value == 0 and c.value == 0
    idx = built_fake_index()
    st = L.gs_sample_pair_counts(ctypes.byref(idx), ctypes.byref(q), FAKE, 16, FAKE, 1 << 30, ctypes.byref(t),
                                 ctypes.byref(c), None)
    assert st == gs.GS_ERR_WORKSPACE and b"plan" in L.gs_last_error()
    st = L.gs_sample_pair_counts(ctypes.byref(idx), ctypes.byref(q), FAKE, 1 << 30, FAKE, 8, ctypes.byref(t),
                                 ctypes.byref(c), None)
    assert st == gs.GS_ERR_WORKSPACE
    st = L.gs_sample_pair_counts(ctypes.byref(idx), ctypes.byref(q), FAKE, 1 << 30, FAKE, 1 << 30, None,
                                 ctypes.byref(c), None)
    assert st == gs.GS_ERR_INVALID_ARGUMENT


def test_noalloc_backward_refuses_oversized_work_before_device_work():
    """The static-workspace backward checks its fixed limit on the host."""
    L = gs.load_library()
    idx = built_fake_index(n_gauss=2_000_000)
    q = gsq.GsQuery(gs.GS_QUERY_POINTS, (ctypes.c_int32 * 3)(0, 0, 0), 3_000_000, None, FAKE)
    st = L.gs_sample_backward_noalloc(ctypes.byref(fake_gauss(2_000_000)), ctypes.byref(idx), ctypes.byref(q), FAKE,
                                      1 << 40, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None)
    assert st == gs.GS_ERR_WORKSPACE and b"fixed" in L.gs_last_error()
    st = L.gs_sample_backward_noalloc(ctypes.byref(fake_gauss()), ctypes.byref(fake_index()), ctypes.byref(q), FAKE,
                                      1 << 40, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None)
    assert st == gs.GS_ERR_INVALID_ARGUMENT


def test_backward_validates_arguments():
    L = gs.load_library()
    idx = built_fake_index()
    q = gsq.GsQuery(gs.GS_QUERY_GRID, (ctypes.c_int32 * 3)(32, 32, 32), 0, None, None)
    args = [ctypes.byref(fake_gauss()), ctypes.byref(idx), ctypes.byref(q), None, 0] + [FAKE] * 9
    st = L.gs_sample_backward(*args, FAKE, 16, None)
    assert st == gs.GS_ERR_WORKSPACE
    need = L.gs_backward_work_bytes(ctypes.byref(idx), ctypes.byref(q))
    assert 0 < need < SIZE_ERR
    args_null = list(args)
    args_null[5] = None  # value
    st = L.gs_sample_backward(*args_null, FAKE, need, None)
    assert st == gs.GS_ERR_INVALID_ARGUMENT
    args_null = list(args)
    args_null[12] = None  # d_value
    st = L.gs_sample_backward(*args_null, FAKE, need, None)
    assert st == gs.GS_ERR_INVALID_ARGUMENT


def test_binding_refuses_cpu_tensors():
    import torch
    with pytest.raises(ValueError):
        gs.Gaussians(torch.zeros(3, 3), torch.ones(3, 3), torch.ones(3, 4), torch.ones(3), torch.ones(3)).c()


def test_binding_fails_loudly_without_the_library(monkeypatch):
    monkeypatch.setattr(gsq, "_LIB", None)
    monkeypatch.setattr(gsq, "LIB_PATH", "/nonexistent/libgsq.so")
    with pytest.raises(gs.GsLibraryMissing):
        gsq.load_library()


def test_training_epilogue_validation():
    """gs_train.h entry points reject malformed arguments before any launch."""
    L = gs.load_library()
    fake = ctypes.c_void_p(1 << 20)  # never dereferenced: every call below fails validation first
    assert L.gs_activate(-1, fake, fake, fake, 0.02, fake, fake, fake, None) == gs.GS_ERR_INVALID_ARGUMENT
    assert L.gs_activate(1 << 31, fake, fake, fake, 0.02, fake, fake, fake, None) == gs.GS_ERR_INVALID_ARGUMENT
    assert L.gs_activate(0, None, None, None, 0.02, None, None, None, None) == gs.GS_OK  # nothing to do
    assert L.gs_activate(5, fake, None, fake, 0.02, fake, fake, fake, None) == gs.GS_ERR_INVALID_ARGUMENT
    assert b"null" in L.gs_last_error()
    assert L.gs_activate_backward(5, fake, fake, fake, 0.0, fake, fake, None, fake, fake, fake, None) == \
        gs.GS_ERR_INVALID_ARGUMENT
    assert L.gs_activate_backward(0, None, None, None, 0.0, None, None, None, None, None, None, None) == gs.GS_OK
    # loss workspace sizing
    a, b = L.gs_loss_work_bytes(1), L.gs_loss_work_bytes(1 << 24)
    assert 0 < a <= b and a % 256 == 0 and b % 256 == 0
    assert L.gs_loss_work_bytes(0) > 0
    assert L.gs_loss_work_bytes(-1) == SIZE_ERR and L.gs_loss_work_bytes(1 << 31) == SIZE_ERR
    ok = gsq.GsLossParams(0.01, 0.1, 1.0, 1.0)
    P = ctypes.byref
    n, need = 1000, L.gs_loss_work_bytes(1000)
    args = lambda p, work=ctypes.c_void_p(1 << 20), wb=need, terms=fake, v=fake: \
        L.gs_loss(n, v, fake, fake, None, p, fake, fake, terms, work, wb, None)
    assert args(None) == gs.GS_ERR_INVALID_ARGUMENT
    assert args(P(ok), terms=None) == gs.GS_ERR_INVALID_ARGUMENT
    assert args(P(ok), v=None) == gs.GS_ERR_INVALID_ARGUMENT
    for bad in (gsq.GsLossParams(0.0, 0.1, 1, 1), gsq.GsLossParams(1.0, 0.1, 1, 1),
                gsq.GsLossParams(float("nan"), 0.1, 1, 1), gsq.GsLossParams(0.01, -0.1, 1, 1),
                gsq.GsLossParams(0.01, float("inf"), 1, 1), gsq.GsLossParams(0.01, 0.1, float("nan"), 1),
                gsq.GsLossParams(0.01, 0.1, 1, float("inf"))):
        assert args(P(bad)) == gs.GS_ERR_INVALID_ARGUMENT, (bad.tau, bad.fn_eps, bad.fn_lambda, bad.fp_lambda)
    assert args(P(ok), wb=need - 1) == gs.GS_ERR_WORKSPACE
    assert args(P(ok), work=ctypes.c_void_p((1 << 20) + 8)) == gs.GS_ERR_WORKSPACE
    assert args(P(ok), work=None) == gs.GS_ERR_WORKSPACE
    assert L.gs_loss(-1, fake, fake, fake, None, P(ok), fake, fake, fake, fake, need, None) == \
        gs.GS_ERR_INVALID_ARGUMENT


def test_densify_validation():
    """gs_densify rejects malformed arguments before any device work."""
    L = gs.load_library()
    P = ctypes.byref
    fake = 1 << 20
    prm = gsq.GsParams(fake, fake, fake, fake, fake)
    g = grid()
    q = gsq.GsQuery(gs.GS_QUERY_GRID, (ctypes.c_int32 * 3)(16, 16, 16), 0, None, None)
    ok = gsq.GsDensifyParams(0.005, 0.01, -5.0, -4.6, 100)
    need = L.gs_densify_work_bytes(1000, P(q))
    assert need != SIZE_ERR and need % 256 == 0 and need > 16 ** 3 * 16
    assert L.gs_densify_work_bytes(-1, P(q)) == SIZE_ERR
    bad_q = gsq.GsQuery(gs.GS_QUERY_VOXELS, (ctypes.c_int32 * 3)(16, 16, 16), 10, None, None)
    assert L.gs_densify_work_bytes(10, P(bad_q)) == SIZE_ERR
    n_out = ctypes.c_int64(-7)

    def call(n_in=1000, prm_in=prm, dp=ok, cap=2000, out=prm, work=fake, wb=need, qq=q, src=fake, dom=g):
        return L.gs_densify(None if prm_in is None else P(prm_in), n_in, fake, None if dom is None else P(dom),
                            P(qq), fake, fake, fake, None, None if dp is None else P(dp),
                            None if out is None else P(out), cap, src, P(n_out), work, wb, None)

    assert call(prm_in=None) == gs.GS_ERR_INVALID_ARGUMENT
    assert call(out=None) == gs.GS_ERR_INVALID_ARGUMENT
    assert call(dp=None) == gs.GS_ERR_INVALID_ARGUMENT
    assert call(dom=None) == gs.GS_ERR_INVALID_ARGUMENT
    assert call(n_in=-1) == gs.GS_ERR_INVALID_ARGUMENT and n_out.value == 0
    assert call(cap=1 << 31) == gs.GS_ERR_INVALID_ARGUMENT
    assert call(qq=bad_q) == gs.GS_ERR_INVALID_ARGUMENT
    assert call(dom=grid((0, 4, 4))) == gs.GS_ERR_INVALID_ARGUMENT
    assert call(src=None) == gs.GS_ERR_INVALID_ARGUMENT
    assert call(out=gsq.GsParams(fake, None, fake, fake, fake)) == gs.GS_ERR_INVALID_ARGUMENT
    for bad in (gsq.GsDensifyParams(0.005, 0.0, -5, -4.6, 1), gsq.GsDensifyParams(float("nan"), 0.01, -5, -4.6, 1),
                gsq.GsDensifyParams(0.005, 0.01, float("inf"), -4.6, 1),
                gsq.GsDensifyParams(0.005, 0.01, -5, float("nan"), 1), gsq.GsDensifyParams(0.005, 0.01, -5, -4.6, -1)):
        assert call(dp=bad) == gs.GS_ERR_INVALID_ARGUMENT
    assert call(wb=need - 1) == gs.GS_ERR_WORKSPACE
    assert call(work=fake + 64) == gs.GS_ERR_WORKSPACE


def test_gaussian_major_validation():
    L = gs.load_library()
    qg = gsq.GsQuery(gs.GS_QUERY_GRID, (ctypes.c_int32 * 3)(8, 8, 8), 0, None, None)
    assert L.gs_sample_gaussian_major_work_bytes(ctypes.byref(qg)) == SIZE_ERR
    qp = gsq.GsQuery(gs.GS_QUERY_POINTS, (ctypes.c_int32 * 3)(0, 0, 0), 1000, 1 << 20, 1 << 20)
    assert L.gs_sample_gaussian_major_work_bytes(ctypes.byref(qp)) == 16000
    # an unbuilt index is rejected before any device work
    idx = gsq.GsIndex()
    idx.n_pairs = -1
    gauss = gsq.GsGaussians(0, None, None, None, None, None)
    assert L.gs_sample_gaussian_major(ctypes.byref(gauss), ctypes.byref(idx), ctypes.byref(qp), None, None, None, 0,
                                      None, 0, None) == gs.GS_ERR_INVALID_ARGUMENT
