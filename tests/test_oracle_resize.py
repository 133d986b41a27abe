"""Pins for the conservative resize reference (oracle/resize.py), CPU only.

Tied to: scipy's bilinear interpolation (ndimage.map_coordinates, order 1,
nearest-edge) at the same sample points; the identity at equal size; the
2x upscaling closed form (even target rows copy a base row, odd ones OR two);
conservativeness on upscaling (every active base block survives in some
target block); and the identity that the threshold-map resize commutes with
mask instantiation for every threshold.  Planted mistakes must fail a pin.
"""

import numpy as np
import pytest
from scipy import ndimage

from oracle import resize as ors


def _mask(H, nq, nk, seed, p=0.2):
    return np.random.default_rng(seed).random((H, nq, nk)) < p


def _sample_points(nb, nt):
    return np.arange(nt) * nb / nt


def pin_matches_scipy_bilinear(bc, rm, rt):
    rng = np.random.default_rng(1)
    for (nq, nk, tq, tk) in ((7, 9, 11, 23), (16, 16, 37, 40), (5, 8, 5, 13)):
        R = rng.integers(0, 4, size=(1, nq, nk))
        x, y = np.meshgrid(_sample_points(nq, tq), _sample_points(nk, tk), indexing="ij")
        phi = ndimage.map_coordinates(R[0].astype(np.float64), [x, y], order=1, mode="nearest")
        ref = np.ceil(phi - 1e-9)     # scipy is float: allow its rounding below integers
        if not np.array_equal(bc(R, tq, tk)[0], ref.astype(np.int64)):
            return False
    return True


def pin_identity_at_equal_size(bc, rm, rt):
    M = _mask(2, 13, 17, 2)
    T = np.random.default_rng(3).random((2, 13, 17)).astype(np.float32)
    return np.array_equal(rm(M, 13, 17), M) and np.array_equal(rt(T, 13, 17), T)


def pin_upscale_by_two_closed_form(bc, rm, rt):
    M = _mask(1, 6, 6, 4, 0.3)[0]
    out = rm(M[None], 12, 12)[0]
    ref = np.zeros((12, 12), dtype=bool)
    for u in range(12):
        rows = [u // 2] if u % 2 == 0 else [u // 2, min(u // 2 + 1, 5)]
        for v in range(12):
            cols = [v // 2] if v % 2 == 0 else [v // 2, min(v // 2 + 1, 5)]
            ref[u, v] = any(M[i, j] for i in rows for j in cols)
    return np.array_equal(out, ref)


def pin_conservative_on_upscale(bc, rm, rt):
    for (nq, nk, tq, tk, seed) in ((10, 10, 23, 23, 5), (256, 256, 591, 591, 6), (7, 30, 8, 61, 7)):
        M = _mask(1, nq, nk, seed, 0.05)[0]
        out = rm(M[None], tq, tk)[0]
        i0, i1, _, wi1 = ors._axis(nq, tq)
        j0, j1, _, wj1 = ors._axis(nk, tk)
        # every active base block (i, j) is a positively weighted neighbour of some active target block
        for (i, j) in zip(*np.nonzero(M)):
            us = np.nonzero((i0 == i) | ((i1 == i) & (wi1 > 0)))[0]
            vs = np.nonzero((j0 == j) | ((j1 == j) & (wj1 > 0)))[0]
            if len(us) == 0 or len(vs) == 0 or not out[np.ix_(us, vs)].any():
                return False
    return True


def pin_threshold_resize_commutes_with_instantiation(bc, rm, rt):
    rng = np.random.default_rng(8)
    T = rng.random((3, 12, 20)).astype(np.float32)
    T[0, 3, 5] = np.float32(0.5)
    Tt = rt(T, 29, 47)
    for p in (0.0, 0.1, 0.5, 0.77, 1.0):
        if not np.array_equal(Tt <= np.float32(p), rm(T <= np.float32(p), 29, 47)):
            return False
    return True


PINS = [pin_matches_scipy_bilinear, pin_identity_at_equal_size, pin_upscale_by_two_closed_form,
        pin_conservative_on_upscale, pin_threshold_resize_commutes_with_instantiation]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_resize_reference_pins(pin):
    assert pin(ors.bilinear_ceil, ors.resize_mask, ors.resize_threshold_map)


def test_nan_entries_are_skipped_in_threshold_resize():
    T = np.array([[[np.nan, 0.3], [np.nan, np.nan]]], dtype=np.float32)
    out = ors.resize_threshold_map(T, 4, 4)
    assert out[0, 0, 0] != out[0, 0, 0] and out[0, 0, 1] == np.float32(0.3)


# -------------------------------------------------------- planted mistakes ---

def _bc_floor(R, tq, tk):
    R = np.asarray(R).astype(np.int64)
    i0, i1, wi0, wi1 = ors._axis(R.shape[1], tq)
    j0, j1, wj0, wj1 = ors._axis(R.shape[2], tk)
    num = (wi0[:, None] * wj0[None, :] * R[:, i0][:, :, j0] + wi0[:, None] * wj1[None, :] * R[:, i0][:, :, j1]
           + wi1[:, None] * wj0[None, :] * R[:, i1][:, :, j0] + wi1[:, None] * wj1[None, :] * R[:, i1][:, :, j1])
    return num // (np.int64(tq) * tk)


def _rm_floor(M, tq, tk):
    return _bc_floor(np.asarray(M, dtype=bool), tq, tk) > 0


def _rm_nearest(M, tq, tk):
    M = np.asarray(M, dtype=bool)
    i0, _, _, _ = ors._axis(M.shape[1], tq)
    j0, _, _, _ = ors._axis(M.shape[2], tk)
    return M[:, i0][:, :, j0]


def _rt_max(T, tq, tk):
    return -ors.resize_threshold_map(-np.asarray(T, np.float32), tq, tk)


def _rm_swapped_axes(M, tq, tk):
    M = np.asarray(M, dtype=bool)
    return np.swapaxes(ors.resize_mask(np.swapaxes(M, 1, 2), tk, tq), 1, 2)[:, :tq, :tk] \
        if M.shape[1] == M.shape[2] and tq != tk else ors.resize_mask(M, tk, tq)


MUTANTS = {
    "floor_instead_of_ceil": (_bc_floor, _rm_floor, ors.resize_threshold_map),
    "nearest_neighbour": (ors.bilinear_ceil, _rm_nearest, ors.resize_threshold_map),
    "max_over_support": (ors.bilinear_ceil, ors.resize_mask, _rt_max),
    "target_sizes_swapped": (ors.bilinear_ceil, _rm_swapped_axes, ors.resize_threshold_map),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistakes_are_caught(name):
    bc, rm, rt = MUTANTS[name]
    failed = []
    for pin in PINS:
        try:
            ok = pin(bc, rm, rt)
        except Exception:
            ok = False
        if not ok:
            failed.append(pin.__name__)
    assert failed, "planted mistake %s passed every pin" % name
