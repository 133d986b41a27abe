"""Seeded Q/K/V, masks and parity samples for a ``Workload``.

Only input generation: no attention arithmetic.  Q, K and V are N(0,1) drawn
in float32 from a seeded ``torch.Generator`` on the target device, multiplied
by a per-head scale s_h (one value per head, applied to q, k and v alike),
then rounded to bfloat16.  Reference checks read the rounded bf16 tensors back
to the host, so both sides always see the same bits.
"""

import numpy as np

from .masks import make_masks, pack_rows


def head_scales(wl):
    """Per-head input scale s_h ~ U[range] (seeded), or None for s_h = 1."""
    if wl.head_scale_range is None:
        return None
    rng = np.random.default_rng(wl.data_seed + 7919)
    lo, hi = wl.head_scale_range
    return rng.uniform(lo, hi, size=wl.H)


def masks_for(wl):
    """(packed uint64 [H, n_qb, W], bool [H, n_qb, n_kb], density [H])."""
    bm, dens = make_masks(
        wl.mask_kind, wl.H, wl.N, wl.blk_q, wl.blk_k, wl.mask_seed, grid=wl.grid,
        rho=wl.rho, rho_range=wl.rho_range, w_t=wl.w_t, n_globals=wl.n_globals)
    return pack_rows(bm), bm, dens


def qkv_for(wl, device="cpu", seed=None):
    """bf16 tensors q, k, v of shape [B, H, N, d] on ``device``."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(int(wl.data_seed if seed is None else seed))
    shape = (wl.B, wl.H, wl.N, wl.d)
    s = head_scales(wl)
    outs = []
    for _ in range(3):
        t = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
        if s is not None:
            t.mul_(torch.as_tensor(s, dtype=torch.float32, device=device).view(1, wl.H, 1, 1))
        outs.append(t.to(torch.bfloat16))
        del t
    return tuple(outs)


def bf16_to_bits(t):
    """Host uint16 view of a bf16 torch tensor's bits (copies to the host)."""
    import torch
    assert t.dtype == torch.bfloat16
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def sample_items(wl, bool_mask, n_items, seed=None):
    """Seeded (b, h, u) query blocks to check against the reference.

    Includes, for each head (up to ``n_items``), its row with the most enabled
    blocks, the last (possibly ragged) query block once, and fills the rest
    uniformly at random without repetition.
    """
    rng = np.random.default_rng(wl.sample_seed if seed is None else seed)
    counts = bool_mask.sum(axis=2)                     # [H, n_qb]
    chosen = []
    seen = set()

    def add(it):
        if it not in seen and len(chosen) < n_items:
            seen.add(it)
            chosen.append(it)

    for h in range(wl.H):
        add((int(rng.integers(wl.B)), h, int(np.argmax(counts[h]))))
    add((wl.B - 1, wl.H - 1, wl.n_qb - 1))
    total = wl.B * wl.H * wl.n_qb
    while len(chosen) < min(n_items, total):
        add((int(rng.integers(wl.B)), int(rng.integers(wl.H)), int(rng.integers(wl.n_qb))))
    return chosen
