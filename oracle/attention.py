"""Reference block-sparse scaled-dot-product attention, float64 on the CPU.

Test infrastructure only (see ``oracle/__init__``).

What is computed (paper Sec. 4.3.2): the CRM kernel is FlashAttention's
forward pass with its dense key-block loop replaced by a walk over the enabled
key blocks of the query block's CRM row, so each executed block is an ordinary
dense tile.  The result is therefore exactly softmax attention in which query
token i may only see the keys of enabled blocks.  Written out, for batch b,
head h and query token i < N with query block u = floor(i / blk_q):

    K_i   = { j < N : bit(h, u, floor(j / blk_k)) = 1 }        (allowed keys)
    s_ij  = scale * sum_c q_ic k_jc                              (j in K_i)
    m_i   = max_{j in K_i} s_ij
    l_i   = sum_{j in K_i} exp(s_ij - m_i)
    lse_i = m_i + ln l_i                         (natural log, scaled logits)
    out_i = sum_{j in K_i} exp(s_ij - lse_i) v_j

Readings where the paper is silent: no causal or token-level mask (video DiTs
use bidirectional full 3D attention, Sec. 1 and Sec. 2.1); a query with no
allowed key gets out = 0 and lse = -inf; keys j >= N do not exist (the last
block of a ragged sequence is short); the inputs are the exact bf16 values,
promoted to float64 before any arithmetic.

The max subtraction only keeps exp() finite; in exact arithmetic the result
does not depend on it.  There is no blocking, no online rescaling and no
reordering here: one matmul for the logits, one for the output.
"""

import numpy as np

from .bits import bf16_bits_to_f64, block_mask


def _as_f64(x):
    x = np.asarray(x)
    if x.dtype == np.uint16:
        return bf16_bits_to_f64(x)
    return x.astype(np.float64, copy=False)


def _allowed_keys(allowed_kb, blk_k, n_tokens):
    """Token-level key mask of one query block from its key-block mask."""
    allowed_kb = np.asarray(allowed_kb, dtype=bool)
    j = np.arange(n_tokens)
    return allowed_kb[j // blk_k]


def attention_block(q_rows, k, v, allowed_kb, blk_k, scale):
    """Output and lse of some query rows that share one CRM row.

    ``q_rows`` [nq, d]; ``k``, ``v`` [N, d] (float, or uint16 bf16 bits);
    ``allowed_kb`` bool [n_kb].  Returns (out [nq, d], lse [nq]).
    """
    q_rows = _as_f64(q_rows)
    k = _as_f64(k)
    v = _as_f64(v)
    n_tokens = k.shape[0]
    keys = _allowed_keys(allowed_kb, blk_k, n_tokens)
    nq, d = q_rows.shape[0], v.shape[1]
    out = np.zeros((nq, d), dtype=np.float64)
    lse = np.full(nq, -np.inf, dtype=np.float64)
    if nq == 0 or not keys.any():
        return out, lse
    s = scale * (q_rows @ k[keys].T)
    m = s.max(axis=1, keepdims=True)
    l = np.exp(s - m).sum(axis=1, keepdims=True)
    lse[:] = (m + np.log(l))[:, 0]
    p = np.exp(s - lse[:, None])
    out[:] = p @ v[keys]
    return out, lse


def _check_shapes(q, k, v, mask_bits, blk_q, blk_k):
    if q.ndim != 4 or q.shape != k.shape or q.shape != v.shape:
        raise ValueError("q, k, v must share one [B, H, N, d] shape")
    B, H, N, d = q.shape
    n_qb = -(-N // blk_q)
    n_kb = -(-N // blk_k)
    mb = np.asarray(mask_bits)
    if mb.shape[0] != H or mb.shape[1] != n_qb:
        raise ValueError("mask_bits must be [H][ceil(N/blk_q)][W]")
    return B, H, N, d, n_qb, n_kb


def attention(q, k, v, mask_bits, blk_q, blk_k, scale):
    """Full block-sparse attention.  q, k, v: [B, H, N, d] (float or bf16 bits).

    Returns out float64 [B, H, N, d] and lse float64 [B, H, N].
    """
    q = np.asarray(q)
    k = np.asarray(k)
    v = np.asarray(v)
    B, H, N, d, n_qb, n_kb = _check_shapes(q, k, v, mask_bits, blk_q, blk_k)
    bm = block_mask(mask_bits, n_kb)
    out = np.zeros((B, H, N, d), dtype=np.float64)
    lse = np.full((B, H, N), -np.inf, dtype=np.float64)
    for b in range(B):
        for h in range(H):
            kh = _as_f64(k[b, h])
            vh = _as_f64(v[b, h])
            for u in range(n_qb):
                r0, r1 = u * blk_q, min((u + 1) * blk_q, N)
                o, s = attention_block(q[b, h, r0:r1], kh, vh, bm[h, u], blk_k, scale)
                out[b, h, r0:r1] = o
                lse[b, h, r0:r1] = s
    return out, lse


def attention_sampled(q, k, v, mask_bits, blk_q, blk_k, scale, items):
    """Reference output for selected query blocks only.

    ``items`` is a sequence of (b, h, u).  Returns a list of
    (out [rows, d], lse [rows]) in the same order, rows = the valid tokens of
    query block u.  Inputs may be bf16 bit arrays; only the touched heads are
    promoted to float64.
    """
    q = np.asarray(q)
    k = np.asarray(k)
    v = np.asarray(v)
    B, H, N, d, n_qb, n_kb = _check_shapes(q, k, v, mask_bits, blk_q, blk_k)
    bm = block_mask(mask_bits, n_kb)
    res = []
    cache = {}
    for (b, h, u) in items:
        if (b, h) not in cache:
            cache.clear()
            cache[(b, h)] = (_as_f64(k[b, h]), _as_f64(v[b, h]))
        kh, vh = cache[(b, h)]
        r0, r1 = u * blk_q, min((u + 1) * blk_q, N)
        res.append(attention_block(q[b, h, r0:r1], kh, vh, bm[h, u], blk_k, scale))
    return res
