"""Pins of the oracle's training-sample positions (the structured training
of Sec. 4.2.2: one random position in each voxel every iteration): special
offsets reduce to the voxel centre and the voxel corner, and every offset in
[0, 1) stays inside its voxel."""
import numpy as np
import pytest

import oracle
import synth


@pytest.mark.parametrize("dims,lo,hi", [((8, 4, 2), (0, 0, 0), (1, 1, 1)), ((7, 5, 3), (-1.0, 0.25, 2.0), (2.0, 1.5, 3.5))])
def test_half_offsets_give_voxel_centres(dims, lo, hi):
    n = dims[0] * dims[1] * dims[2]
    u = np.full((n, 3), 0.5, np.float32)
    np.testing.assert_array_equal(oracle.jitter_positions(dims, u, lo, hi), oracle.voxel_centers(dims, lo, hi))
    ids = np.random.default_rng(3).choice(n, size=17, replace=False).astype(np.uint32)
    np.testing.assert_array_equal(oracle.jitter_positions(dims, u[:17], lo, hi, ids=ids),
                                  oracle.voxel_centers(dims, lo, hi, ids=ids))


def test_zero_offsets_give_exact_corners():
    # unit box and power-of-two dims: the corner i / 2^k is a float32
    dims = (16, 8, 4)
    n = 16 * 8 * 4
    p = oracle.jitter_positions(dims, np.zeros((n, 3), np.float32))
    t = np.arange(n)
    ijk = np.stack([t % 16, (t // 16) % 8, t // 128], axis=1)
    np.testing.assert_array_equal(p.astype(np.float64), ijk / np.array(dims, np.float64))


def test_offsets_stay_in_their_voxel():
    dims, lo, hi = (13, 9, 6), (-0.5, 0.0, 1.0), (1.5, 0.75, 2.5)
    n = 13 * 9 * 6
    u = synth.jitter_offsets(99, n)
    u[:5] = np.float32(np.nextafter(np.float32(1), np.float32(0)))  # the largest float32 below 1
    u[5:10] = 0.0
    p = oracle.jitter_positions(dims, u, lo, hi).astype(np.float64)
    t = np.arange(n)
    ijk = np.stack([t % 13, (t // 13) % 9, t // 117], axis=1)
    lo_, hi_ = np.array(lo, np.float64), np.array(hi, np.float64)
    vs = (hi_ - lo_) / np.array(dims, np.float64)
    # within the voxel, up to float32 rounding of the three operations
    slack = 4 * np.finfo(np.float32).eps * (np.abs(lo_) + np.abs(hi_))
    assert np.all(p >= lo_ + ijk * vs - slack)
    assert np.all(p <= lo_ + (ijk + 1) * vs + slack)
    # and at the fractional offset u within it, to float32 accuracy
    frac = (p - lo_) / vs - ijk
    assert np.max(np.abs(frac - u)) < 1e-4


def test_without_ids_is_every_voxel_in_order():
    dims = (5, 4, 3)
    n = 60
    u = synth.jitter_offsets(5, n)
    np.testing.assert_array_equal(oracle.jitter_positions(dims, u),
                                  oracle.jitter_positions(dims, u, ids=np.arange(n, dtype=np.uint32)))
    with pytest.raises(ValueError):
        oracle.jitter_positions(dims, u[:59])
