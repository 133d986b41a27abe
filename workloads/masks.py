"""Seeded synthetic block masks shaped like the paper's static per-head masks.

The paper's masks come from an offline pipeline (WEST threshold maps, FAST
per-head thresholds, Sec. 4.1-4.2) run on Wan2.1 / HunyuanVideo weights and
calibration prompts, none of which are available here.  These generators are
stand-ins with the same structure: for every head a static block mask with a
temporal window, a spatial neighbourhood, a few "global" key-block columns,
the diagonal always on, and seeded random fill up to an exact per-head
density.  Density is the fraction of enabled blocks (Sec. 1, Fig. 1 caption;
global density in Sec. 5.1 is the same ratio measured in FLOPs).

Only input generation lives here: no attention arithmetic.  Everything draws
from ``numpy.random.default_rng(seed)`` (PCG64), which is machine-independent.
"""

import numpy as np


def n_blocks(n_tokens, blk):
    return -(-int(n_tokens) // int(blk))


def block_centres(n_blk, blk, grid):
    """(frame, y, x) of each block's centre token, frame-major flattening.

    Token t sits at frame t // (Hs*Ws), row (t % (Hs*Ws)) // Ws, column t % Ws.
    Centres past the last grid token (padding tokens) clamp to that token.
    """
    T, Hs, Ws = grid
    n_tok = T * Hs * Ws
    c = np.minimum(np.arange(n_blk) * blk + blk // 2, n_tok - 1)
    f = c // (Hs * Ws)
    r = c % (Hs * Ws)
    return f, r // Ws, r % Ws


def _diag(n_qb, n_kb, blk_q, blk_k, n_tokens):
    """Key block holding each query block's centre token (u == v when blk_q == blk_k)."""
    c = np.minimum(np.arange(n_qb) * blk_q + blk_q // 2, n_tokens - 1)
    m = np.zeros((n_qb, n_kb), dtype=bool)
    m[np.arange(n_qb), c // blk_k] = True
    return m


def _fill_random(rng, m, target):
    """Enable uniformly chosen unset blocks until exactly ``target`` are set."""
    need = int(target) - int(m.sum())
    if need > 0:
        unset = np.flatnonzero(~m.ravel())
        pick = rng.choice(unset, size=need, replace=False)
        flat = m.ravel().copy()
        flat[pick] = True
        m = flat.reshape(m.shape)
    return m


def structured_head(rng, n_tokens, blk_q, blk_k, grid, rho, w_t, n_globals):
    """One head's structured mask (bool [n_qb, n_kb]) at exact density ``rho``.

    Structural blocks: the diagonal, ``n_globals`` global key-block columns,
    and every (u, v) whose centre tokens are within ``w_t`` frames and within
    Chebyshev radius r on the latent grid.  r is the largest radius whose
    structural count stays within the target; if even r = 0 overshoots, the
    temporal window shrinks.  Random fill then reaches the exact target.
    """
    n_qb, n_kb = n_blocks(n_tokens, blk_q), n_blocks(n_tokens, blk_k)
    target = int(round(rho * n_qb * n_kb))
    base = _diag(n_qb, n_kb, blk_q, blk_k, n_tokens)
    if n_globals > 0:
        cols = rng.choice(n_kb, size=min(n_globals, n_kb), replace=False)
        base[:, cols] = True
    fq, yq, xq = block_centres(n_qb, blk_q, grid)
    fk, yk, xk = block_centres(n_kb, blk_k, grid)
    df = np.abs(fq[:, None] - fk[None, :])
    dsp = np.maximum(np.abs(yq[:, None] - yk[None, :]), np.abs(xq[:, None] - xk[None, :]))
    m = base
    n_base = int(base.sum())
    for w in range(int(w_t), -1, -1):
        cand = (df <= w) & ~base
        radii = np.sort(dsp[cand])
        # largest r with n_base + #(cand with dsp <= r) <= target
        room = target - n_base
        if room < 0 or radii.size == 0:
            continue
        if radii.size <= room:
            m = base | cand
            break
        r_lim = radii[room]            # the (room+1)-th smallest radius overshoots
        r = r_lim - 1
        if r < 0:
            continue                   # even radius 0 overshoots: shrink the window
        m = base | (cand & (dsp <= r))
        break
    return _fill_random(rng, m, target)


def uniform_head(rng, n_tokens, blk_q, blk_k, rho):
    """Diagonal plus uniformly random blocks, exact density ``rho``."""
    n_qb, n_kb = n_blocks(n_tokens, blk_q), n_blocks(n_tokens, blk_k)
    target = int(round(rho * n_qb * n_kb))
    return _fill_random(rng, _diag(n_qb, n_kb, blk_q, blk_k, n_tokens), target)


def pack_rows(bool_mask):
    """bool [H, n_qb, n_kb] -> uint64 [H, n_qb, ceil(n_kb/64)], LSB-first words.

    Block v of a row is bit (v mod 64) of word v // 64; unused high bits of the
    last word are zero.
    """
    bm = np.asarray(bool_mask, dtype=bool)
    H, n_qb, n_kb = bm.shape
    W = (n_kb + 63) // 64
    padded = np.zeros((H, n_qb, W * 64), dtype=bool)
    padded[:, :, :n_kb] = bm
    by = np.packbits(padded, axis=-1, bitorder="little")
    return np.ascontiguousarray(by).view("<u8").reshape(H, n_qb, W).astype(np.uint64)


def make_masks(kind, H, n_tokens, blk_q, blk_k, seed, grid=None, rho=None,
               rho_range=None, w_t=None, n_globals=None):
    """Per-head masks for one workload.

    kind: "structured" | "uniform" | "dense".  Per head, rho comes from
    ``rho`` (fixed) or U[rho_range]; for "structured" the temporal half-window
    is ``w_t`` or U{1,2,3}, and the number of global columns ``n_globals`` or
    U{1..4}.  Returns (bool [H, n_qb, n_kb], per-head density float64 [H]).
    """
    rng = np.random.default_rng(seed)
    n_qb, n_kb = n_blocks(n_tokens, blk_q), n_blocks(n_tokens, blk_k)
    out = np.zeros((H, n_qb, n_kb), dtype=bool)
    for h in range(H):
        if kind == "dense":
            out[h] = True
            continue
        r = float(rho) if rho is not None else float(rng.uniform(*rho_range))
        if kind == "structured":
            wt = int(w_t) if w_t is not None else int(rng.integers(1, 4))
            ng = int(n_globals) if n_globals is not None else int(rng.integers(1, 5))
            out[h] = structured_head(rng, n_tokens, blk_q, blk_k, grid, r, wt, ng)
        elif kind == "uniform":
            out[h] = uniform_head(rng, n_tokens, blk_q, blk_k, r)
        else:
            raise ValueError("unknown mask kind %r" % (kind,))
    dens = out.reshape(H, -1).mean(axis=1)
    return out, dens
