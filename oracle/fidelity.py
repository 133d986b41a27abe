"""Reference Hellinger fidelity of block-sparse attention (paper Sec. 4.2.1, 4.2.3).

Test infrastructure only (see ``oracle/__init__``).

FAST measures how far a sparse attention row is from the dense one with the
Hellinger distance (Sec. 4.2.1, Eq. 3)

    H(P, Q) = (1 / sqrt 2) * sqrt( sum_j (sqrt p_j - sqrt q_j)^2 )

and scores a mask by the Fidelity Score F = 1 - H (Eq. 4).  Here P is the
dense softmax row of a query token over all N keys and Q = P~ the row that
block-sparse attention produces: softmax over the keys of the enabled blocks
only (zero elsewhere), which is exactly what the CRM kernel computes.  The
masks are those of the threshold map, M_p = 1[T <= p] (Sec. 4.1.2), for each
candidate threshold p; the profile is taken on a few sampled query rows per
head (Sec. 4.2.3, stratified sampling), and a head's score for a candidate is
the mean over its sampled rows of 1 - H (reading: the mean over rows of the
per-row distance; the paper defines H for one pair of distributions).  A row
whose mask enables no key has no sparse distribution; its distance is taken as
1 (the largest value H can take).

Float64 throughout, written from the definitions: logits, dense softmax,
restricted softmax, then Eq. 3 term by term.
"""

import numpy as np

from .bits import bf16_bits_to_f64


def _f64(x):
    x = np.asarray(x)
    return bf16_bits_to_f64(x) if x.dtype == np.uint16 else x.astype(np.float64)


def hellinger(P, Q):
    """Eq. 3 for distributions along the last axis."""
    P = np.asarray(P, dtype=np.float64)
    Q = np.asarray(Q, dtype=np.float64)
    return np.sqrt(np.sum((np.sqrt(P) - np.sqrt(Q)) ** 2, axis=-1)) / np.sqrt(2.0)


def fidelity_score(P, Q):
    """Eq. 4: F = 1 - H."""
    return 1.0 - hellinger(P, Q)


def _softmax_over(s, allowed=None):
    """Softmax of logits s over the allowed positions (all if None), zero elsewhere."""
    if allowed is None:
        allowed = np.ones(s.shape, dtype=bool)
    if not allowed.any():
        return None
    t = np.where(allowed, s, -np.inf)
    t = t - t[allowed].max()
    e = np.where(allowed, np.exp(t), 0.0)
    return e / e.sum()


def logits(q_row, k, scale):
    """s_j = scale * <q, k_j> for every key j (float64)."""
    return scale * (_f64(k) @ _f64(q_row))


def dense_row(q_row, k, scale):
    """Dense softmax row of one query over all keys (float64)."""
    return _softmax_over(logits(q_row, k, scale))


def profile(q, k, rows, T, p_cands, blk, scale):
    """Fidelity profile of threshold-map masks on sampled rows.

    q, k: [B][H][N][d] (bf16 bit patterns or floats); rows: int [H][R] query
    token indices per head (shared by the batch); T: [H][n_qb][n_kb] map;
    p_cands: [K] candidate thresholds.  Returns (Hd [B][H][R][K], F [B][H][K]).
    A row's logits do not depend on the candidate, so they are formed once per
    row; each candidate then restricts and renormalises them (P~) and Eq. 3 is
    taken against the dense row P.
    """
    q = np.asarray(q)
    k = np.asarray(k)
    B, H, N, d = q.shape
    rows = np.asarray(rows)
    R = rows.shape[1]
    T = np.asarray(T, dtype=np.float32)
    p_cands = np.asarray(p_cands, dtype=np.float32)
    K = p_cands.shape[0]
    key_block = np.arange(N) // blk
    Hd = np.zeros((B, H, R, K))
    for b in range(B):
        for h in range(H):
            kf = _f64(k[b, h])
            for i in range(R):
                r = int(rows[h, i])
                s = scale * (kf @ _f64(q[b, h, r]))
                P = _softmax_over(s)
                u = r // blk
                for c in range(K):
                    on_blocks = T[h, u] <= p_cands[c]
                    Qs = _softmax_over(s, on_blocks[key_block])
                    Hd[b, h, i, c] = 1.0 if Qs is None else hellinger(P, Qs)
    return Hd, 1.0 - Hd.mean(axis=2)


def block_log_mass(q_row, k, blk, scale):
    """log sum_{j in block v} exp(s_j) for every key block v (natural log, float64).

    The per-block pooled attention mass of one query row before normalisation:
    exp(block_log_mass - logsumexp over all keys) is the probability mass the
    dense row puts on block v (the row-sampled form of the block pooling of
    Sec. 4.1.1, Eq. 1, summed instead of averaged).
    """
    s = logits(q_row, k, scale)
    N = s.shape[0]
    n_kb = -(-N // blk)
    out = np.empty(n_kb)
    for v in range(n_kb):
        sv = s[v * blk:min((v + 1) * blk, N)]
        mx = sv.max()
        out[v] = mx + np.log(np.exp(sv - mx).sum())
    return out
