"""Seeded input generators: determinism, exact density, structure."""

import numpy as np
import pytest

import oracle
from workloads import (TINY, WAN13B_480P, WAN14B_480P, WAN14B_720P, make_masks, masks_for,
                       pack_rows, sample_items, sweep_point, block_centres)


def test_tiny_mask_reading():
    # 4 frames x 4 blocks of 64 tokens; structural = same in-frame position within +-1 frame
    packed, bm, dens = masks_for(TINY)
    assert packed.shape == (1, 16, 1) and packed.dtype == np.uint64
    assert bm.sum() == 64 and dens[0] == 0.25
    f, y, x = block_centres(16, 64, TINY.grid)
    struct = (np.abs(f[:, None] - f[None, :]) <= 1) & (y[:, None] == y[None, :]) & (x[:, None] == x[None, :])
    assert struct.sum() == 40
    assert np.all(bm[0][struct])


@pytest.mark.parametrize("wl", [TINY, WAN13B_480P, WAN14B_480P, WAN14B_720P], ids=lambda w: w.name)
def test_masks_deterministic_exact_and_diagonal(wl):
    p1, bm1, d1 = masks_for(wl)
    p2, bm2, d2 = masks_for(wl)
    assert np.array_equal(p1, p2)
    n_qb, n_kb = wl.n_qb, wl.n_kb
    assert p1.shape == (wl.H, n_qb, (n_kb + 63) // 64)
    assert np.array_equal(oracle.block_mask(p1, n_kb), bm1)
    for h in range(wl.H):
        assert np.all(bm1[h, np.arange(n_qb), np.arange(n_qb)])
    if wl.rho_range is not None:
        lo, hi = wl.rho_range
        assert np.all(d1 >= lo - 1e-3) and np.all(d1 <= hi + 1e-3)
    # unused high bits of the last word are zero
    tail = n_kb % 64
    if tail:
        assert np.all((p1[:, :, -1] >> np.uint64(tail)) == 0)


def test_sweep_points_hit_density():
    for blk in (64, 128):
        for kind in ("structured", "uniform"):
            for rho in (0.5, 0.1, 0.05):
                wl = sweep_point(rho, blk, kind)
                _, bm, d = masks_for(wl)
                target = round(rho * wl.n_qb * wl.n_kb) / (wl.n_qb * wl.n_kb)
                assert np.allclose(d, target)
    _, bm, d = masks_for(sweep_point(1.0, 128, "structured"))
    assert bm.all()


def test_structured_masks_have_structure():
    bm, _ = make_masks("structured", 4, 32768, 128, 128, 7, grid=(21, 30, 52), rho=0.2)
    f, _, _ = block_centres(256, 128, (21, 30, 52))
    near = np.abs(f[:, None] - f[None, :]) <= 3
    # far more enabled blocks inside the temporal window than a uniform mask would give
    for h in range(4):
        inside = bm[h][near].mean()
        outside = bm[h][~near].mean()
        assert inside > 2 * outside


def test_pack_rows_lsb_first():
    bm = np.zeros((1, 1, 70), dtype=bool)
    bm[0, 0, [0, 5, 64, 69]] = True
    w = pack_rows(bm)
    assert int(w[0, 0, 0]) == (1 | (1 << 5)) and int(w[0, 0, 1]) == (1 | (1 << 5))


def test_sample_items_cover_heads_and_tail():
    _, bm, _ = masks_for(WAN14B_480P)
    items = sample_items(WAN14B_480P, bm, 64)
    assert len(items) == 64 and len(set(items)) == 64
    assert {h for (_, h, _) in items} == set(range(40))
    assert (0, 39, 255) in items
