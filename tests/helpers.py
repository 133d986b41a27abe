"""Shared helpers for the GPU parity tests: tolerances and reference runs."""

import numpy as np

import oracle

# Tolerances fixed for the forward pass: out max-abs 2e-2, mean-abs 2e-3; lse max-abs 1e-3.
OUT_MAX_ABS = 2e-2
OUT_MEAN_ABS = 2e-3
LSE_MAX_ABS = 1e-3
# Where a bf16 output cannot come within OUT_MAX_ABS of the exact value (its
# half-ulp exceeds 1e-2 once |out| >= 8), the bound is the half-ulp plus the
# arithmetic allowance below.
BF16_FLOOR_EXTRA = 4e-3


def bf16_half_ulp(x):
    """Half a unit in the last place of bf16 (8 significant bits) at |x|."""
    ax = np.maximum(np.abs(np.asarray(x, dtype=np.float64)), 2.0 ** -126)
    return 2.0 ** (np.floor(np.log2(ax)) - 8)


# Unit roundoff of bf16: 8 significant bits, round to nearest even, so the
# relative error of one rounding is at most half an ulp over the value, 2^-8
# (pinned by tests/test_tolerances.py).
BF16_UNIT_ROUNDOFF = 2.0 ** -8


def compare(out_gpu, lse_gpu, out_ref, lse_ref, pv_abs=None):
    """Element-wise comparison; returns a stats dict (raises AssertionError on failure).

    pv_abs, when given, is the reference attention applied to |v| (the same
    weights on the absolute values).  P is rounded to bf16 before the P V
    product, which moves out_ic by at most the unit roundoff times
    sum_j P_ij |v_jc| / sum_j P_ij, so the arithmetic allowance beside the
    output's own half-ulp is that bound plus 1e-3 for the fp32 arithmetic,
    instead of the fixed BF16_FLOOR_EXTRA."""
    out_gpu = np.asarray(out_gpu, dtype=np.float64)
    out_ref = np.asarray(out_ref, dtype=np.float64)
    lse_gpu = np.asarray(lse_gpu, dtype=np.float64)
    lse_ref = np.asarray(lse_ref, dtype=np.float64)
    assert out_gpu.shape == out_ref.shape and lse_gpu.shape == lse_ref.shape
    err = np.abs(out_gpu - out_ref)
    if pv_abs is None:
        extra = BF16_FLOOR_EXTRA
    else:
        extra = BF16_UNIT_ROUNDOFF * np.asarray(pv_abs, dtype=np.float64) + 1e-3
    allowed = np.maximum(OUT_MAX_ABS, bf16_half_ulp(out_ref) + extra)
    fin_ref = np.isfinite(lse_ref)
    assert np.array_equal(np.isfinite(lse_gpu), fin_ref), "lse finiteness differs"
    assert np.all(np.isneginf(lse_gpu[~fin_ref])), "empty rows must have lse = -inf"
    lse_err = np.abs(lse_gpu[fin_ref] - lse_ref[fin_ref])
    stats = dict(
        out_max_abs=float(err.max()) if err.size else 0.0,
        out_mean_abs=float(err.mean()) if err.size else 0.0,
        lse_max_abs=float(lse_err.max()) if lse_err.size else 0.0,
        n_bf16_floor=int((allowed > OUT_MAX_ABS).sum()),
        out_max_abs_excl_floor=float(err[allowed <= OUT_MAX_ABS].max()) if err.size else 0.0,
    )
    assert np.all(np.isfinite(out_gpu)), "non-finite output"
    bad = err > allowed
    assert not bad.any(), "out error %.3g at %s exceeds bound (stats %s)" % (
        err[bad].max(), np.argwhere(bad)[0].tolist(), stats)
    assert stats["out_mean_abs"] <= OUT_MEAN_ABS, stats
    assert stats["lse_max_abs"] <= LSE_MAX_ABS, stats
    return stats


def compare_strict(out_gpu, lse_gpu, out_ref, lse_ref):
    """The plain bounds with no allowance for rounding the output: out max-abs
    <= OUT_MAX_ABS and mean-abs <= OUT_MEAN_ABS over every checked element,
    lse max-abs <= LSE_MAX_ABS over the finite ones.  For float32 outputs."""
    out_gpu = np.asarray(out_gpu, dtype=np.float64)
    out_ref = np.asarray(out_ref, dtype=np.float64)
    lse_gpu = np.asarray(lse_gpu, dtype=np.float64)
    lse_ref = np.asarray(lse_ref, dtype=np.float64)
    assert out_gpu.shape == out_ref.shape and lse_gpu.shape == lse_ref.shape
    assert np.all(np.isfinite(out_gpu)), "non-finite output"
    fin_ref = np.isfinite(lse_ref)
    assert np.array_equal(np.isfinite(lse_gpu), fin_ref), "lse finiteness differs"
    err = np.abs(out_gpu - out_ref)
    lse_err = np.abs(lse_gpu[fin_ref] - lse_ref[fin_ref])
    stats = dict(out_max_abs=float(err.max()) if err.size else 0.0,
                 out_mean_abs=float(err.mean()) if err.size else 0.0,
                 lse_max_abs=float(lse_err.max()) if lse_err.size else 0.0)
    assert stats["out_max_abs"] <= OUT_MAX_ABS, stats
    assert stats["out_mean_abs"] <= OUT_MEAN_ABS, stats
    assert stats["lse_max_abs"] <= LSE_MAX_ABS, stats
    return stats


def gather_rows(t, items, blk_q, N):
    """Rows of the (b, h, u) query blocks of a [B, H, N, ...] device tensor, on the host,
    concatenated in item order."""
    parts = []
    for (b, h, u) in items:
        r0, r1 = u * blk_q, min((u + 1) * blk_q, N)
        parts.append(t[b, h, r0:r1].float().cpu().numpy())
    return np.concatenate(parts)


def to_bits(t):
    """bf16 torch tensor -> host uint16 bit array."""
    import torch
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def reference_items(q, k, v, packed, blk_q, blk_k, scale, items):
    """Reference (out, lse) for (b, h, u) query blocks, reading device tensors per head."""
    B, H, N, d = q.shape
    n_kb = -(-N // blk_k)
    res = {}
    by_head = {}
    for it in items:
        by_head.setdefault((it[0], it[1]), []).append(it[2])
    for (b, h), us in sorted(by_head.items()):
        kb = to_bits(k[b, h])
        vb = to_bits(v[b, h])
        for u in us:
            allowed = oracle.block_mask(packed[h:h + 1, u:u + 1], n_kb)[0, 0]
            r0, r1 = u * blk_q, min((u + 1) * blk_q, N)
            qb = to_bits(q[b, h, r0:r1])
            res[(b, h, u)] = oracle.attention_block(qb, kb, vb, allowed, blk_k, scale)
    return res
