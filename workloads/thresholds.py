"""Seeded synthetic threshold maps shaped like WEST's (paper Sec. 4.1.2).

A threshold map gives, per head and block (u, v), the smallest density
threshold p at which the block joins the head's mask.  The real maps come from
calibration prompts on model weights that are not available here; these
stand-ins have the structure the paper describes and visualises: the diagonal
and a few "global" key columns enter first, then blocks in a spatio-temporal
neighbourhood of the query block in order of distance, and the remaining
blocks late and in no particular order.

Only input generation lives here.  ``p_for_density`` picks the threshold that
gives a target density (the quantile of the map), as FAST's offline search
would; it is a helper for choosing inputs, not part of the instantiation.
"""

import numpy as np

from .masks import block_centres


def threshold_maps(H, n_qb, n_kb, blk, grid, seed):
    """float32 ``[H][n_qb][n_kb]`` threshold maps with values in [0, 1]."""
    rng = np.random.default_rng(seed)
    T_, Hs, Ws = grid
    fq, yq, xq = block_centres(n_qb, blk, grid)
    fk, yk, xk = block_centres(n_kb, blk, grid)
    df = np.abs(fq[:, None] - fk[None, :]).astype(np.float64)
    dsp = np.maximum(np.abs(yq[:, None] - yk[None, :]), np.abs(xq[:, None] - xk[None, :]))
    out = np.empty((H, n_qb, n_kb), dtype=np.float32)
    for h in range(H):
        w_t = rng.uniform(1.0, 4.0)                      # temporal reach of this head
        r_s = rng.uniform(2.0, max(3.0, 0.5 * max(Hs, Ws)))  # spatial reach
        dist = df / w_t + dsp / r_s                      # 0 on the diagonal
        near = 0.5 * dist / (1.0 + dist)                 # in [0, 0.5)
        late = rng.uniform(0.3, 1.0, size=(n_qb, n_kb))  # unstructured remainder
        mix = rng.uniform(0.0, 1.0, size=(n_qb, n_kb)) < np.exp(-dist)
        t = np.where(mix, near + 0.05 * rng.random((n_qb, n_kb)), np.maximum(near, late))
        g = rng.choice(n_kb, size=rng.integers(1, 5), replace=False)
        t[:, g] = rng.uniform(0.0, 0.05, size=(n_qb, len(g)))
        d = np.minimum(np.arange(n_qb) * blk + blk // 2, T_ * Hs * Ws - 1) // blk
        t[np.arange(n_qb), np.minimum(d, n_kb - 1)] = 0.0
        out[h] = np.clip(t, 0.0, 1.0).astype(np.float32)
    return out


def p_for_density(T, rho):
    """Per-head float32 threshold whose mask ``T <= p`` has density >= rho (quantile)."""
    T = np.asarray(T, dtype=np.float32)
    H = T.shape[0]
    flat = np.sort(T.reshape(H, -1), axis=1)
    n = flat.shape[1]
    rho = np.broadcast_to(np.asarray(rho, dtype=np.float64), (H,))
    idx = np.clip(np.ceil(rho * n).astype(np.int64) - 1, 0, n - 1)
    return flat[np.arange(H), idx].astype(np.float32)


def stratified_rows(N, H, n_strata=16, per_stratum=1, seed=0):
    """Sampled query rows per head for fidelity profiling (paper Sec. 4.2.3).

    The N rows are cut into ``n_strata`` equal strata and ``per_stratum`` rows
    are drawn uniformly (without replacement) from each, so every part of the
    sequence is represented.  The paper profiles with 16 rows, about 0.05 % of
    a 32K-token map; read here as 16 strata of one row each.  Returns int32
    ``[H][n_strata * per_stratum]``, ascending per head.
    """
    rng = np.random.default_rng(seed)
    edges = np.linspace(0, N, n_strata + 1).astype(np.int64)
    out = np.empty((H, n_strata * per_stratum), dtype=np.int32)
    for h in range(H):
        picks = []
        for s in range(n_strata):
            lo, hi = int(edges[s]), int(edges[s + 1])
            n = max(hi - lo, 1)
            take = min(per_stratum, n)
            sel = rng.choice(n, size=take, replace=False) + lo
            sel = np.pad(sel, (0, per_stratum - take), mode="edge")
            picks.append(np.sort(sel))
        out[h] = np.minimum(np.concatenate(picks), N - 1)
    return out
