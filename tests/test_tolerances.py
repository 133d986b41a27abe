"""Pins of the constants the parity bounds are built from (CPU only).

The bound on the effect of rounding P to bf16 uses bf16's unit roundoff, and
the out bound beside it uses half a bf16 ulp at |ref|.  Both are checked here
against torch's own float32 -> bfloat16 conversion (round to nearest even), so
that a constant off by a factor of two fails.  The comparison itself
(helpers.compare) is checked both ways on a small case: it accepts an emulation
of the kernel's arithmetic at input scale 2, and it rejects references with a
planted mistake (a dropped block, a shifted lse, a flipped sign, a transposed
operand).
"""

import numpy as np
import pytest
import torch

from helpers import BF16_UNIT_ROUNDOFF, bf16_half_ulp


def _round_bf16(x):
    return torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()


def test_unit_roundoff_is_the_largest_relative_error_of_one_rounding():
    rng = np.random.default_rng(5)
    x = (rng.uniform(1.0, 2.0, 1 << 20) * 2.0 ** rng.integers(-60, 60, 1 << 20)).astype(np.float32)
    rel = np.abs(_round_bf16(x) - x.astype(np.float64)) / np.abs(x.astype(np.float64))
    assert rel.max() <= BF16_UNIT_ROUNDOFF
    assert rel.max() > 0.99 * BF16_UNIT_ROUNDOFF    # attained: a smaller constant would fail
    # just above 1 the error is exactly the unit roundoff (ties go to even: down to 1)
    tie = np.array([1.0 + 2.0 ** -8], dtype=np.float32)
    assert _round_bf16(tie)[0] == 1.0


def test_half_ulp_bounds_the_absolute_error_of_one_rounding():
    rng = np.random.default_rng(6)
    x = (rng.standard_normal(1 << 20) * 2.0 ** rng.integers(-20, 20, 1 << 20)).astype(np.float32)
    err = np.abs(_round_bf16(x) - x.astype(np.float64))
    hu = bf16_half_ulp(x)
    assert np.all(err <= hu)
    assert (err / hu).max() > 0.99
    assert bf16_half_ulp(np.array([4.5]))[0] == 2.0 ** -6    # ulp on [4, 8) is 2^-5


# ------------------------------------------------ the parity comparison itself ---

def _bits(x):
    """float -> bf16 bit pattern (round to nearest even), as the GPU tests pass them."""
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(
        torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def _from_bits(b):
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _small_case(scale_in, seed=11):
    from workloads import pack_rows
    rng = np.random.default_rng(seed)
    B, H, N, d, blk = 1, 2, 300, 64, 64
    n_b = -(-N // blk)
    bm = rng.random((H, n_b, n_b)) < 0.5
    bm[:, np.arange(n_b), np.arange(n_b)] = True
    q, k, v = (_bits(rng.standard_normal((B, H, N, d)) * scale_in) for _ in range(3))
    return q, k, v, bm, pack_rows(bm), blk, 1.0 / d ** 0.5


def _kernel_arithmetic(q, k, v, bm, blk, scale):
    """The attention kernel's arithmetic, emulated: fp32 logits, exact row maximum in
    the log2 domain, P rounded to bf16 before P V, fp32 sums, out rounded to bf16."""
    qf, kf, vf = (_from_bits(t).astype(np.float32) for t in (q, k, v))
    B, H, N, d = qf.shape
    c = np.float32(scale * 1.4426950408889634)
    out = np.zeros((B, H, N, d))
    lse = np.full((B, H, N), -np.inf)
    idx = np.arange(N) // blk
    for b in range(B):
        for h in range(H):
            allow = bm[h][idx][:, idx]
            s = np.where(allow, qf[b, h] @ kf[b, h].T, -np.inf).astype(np.float32)
            m = (s.max(1, keepdims=True) * c).astype(np.float32)
            p = np.exp2((s * c - m).astype(np.float32)).astype(np.float32)
            pb = _from_bits(_bits(p))
            l = p.astype(np.float64).sum(1, keepdims=True)
            out[b, h] = _from_bits(_bits(pb @ vf[b, h].astype(np.float64) / l))
            lse[b, h] = (m[:, 0] + np.log2(l[:, 0])) * np.log(2.0)
    return out, lse


def test_compare_accepts_the_kernel_arithmetic_at_high_input_scale():
    import oracle
    from helpers import compare
    q, k, v, bm, packed, blk, scale = _small_case(scale_in=2.0)
    ref_out, ref_lse = oracle.attention(q, k, v, packed, blk, blk, scale)
    pv_abs, _ = oracle.attention(q, k, v & np.uint16(0x7FFF), packed, blk, blk, scale)
    out, lse = _kernel_arithmetic(q, k, v, bm, blk, scale)
    compare(out, lse, ref_out, ref_lse, pv_abs=pv_abs)
    compare(out, lse, ref_out, ref_lse)


@pytest.mark.parametrize("plant", ["drop_block", "lse_shift", "sign", "transpose_v"])
def test_compare_rejects_planted_mistakes_in_the_reference(plant):
    """Mistakes planted in the reference (on the CPU) must fail the comparison."""
    import oracle
    from helpers import compare
    from workloads import pack_rows
    q, k, v, bm, packed, blk, scale = _small_case(scale_in=1.0)
    out, lse = oracle.attention(q, k, v, packed, blk, blk, scale)
    ref_out, ref_lse = out.copy(), lse.copy()
    if plant == "drop_block":       # one enabled off-diagonal block missing from the reference
        bm2 = bm.copy()
        u, w = [(u, w) for u in range(bm.shape[1]) for w in range(bm.shape[2])
                if bm[0, u, w] and u != w][0]
        bm2[0, u, w] = False
        ref_out, ref_lse = oracle.attention(q, k, v, pack_rows(bm2), blk, blk, scale)
    elif plant == "lse_shift":      # lse off by 2e-3 (a wrong log base would be far more)
        ref_lse = ref_lse + 2e-3
    elif plant == "sign":           # one element with the wrong sign
        i = np.unravel_index(np.argmax(np.abs(ref_out)), ref_out.shape)
        ref_out[i] = -ref_out[i]
    elif plant == "transpose_v":    # v's token and feature axes mixed up in one head
        vt = v.copy()
        vt[0, 0, :64, :] = v[0, 0, :64, :].T
        ref_out, ref_lse = oracle.attention(q, k, vt, packed, blk, blk, scale)
    with pytest.raises(AssertionError):
        compare(out, lse, ref_out, ref_lse)
