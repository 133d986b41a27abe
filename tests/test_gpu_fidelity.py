"""Fidelity profile on the GPU (sa_fidelity_profile) vs the float64 reference.

Tolerance, derived from the arithmetic: logits come from bf16 products summed in
fp32 (relative error ~1e-6 of sum |q_c k_c|, i.e. ~1e-5 in a logit at these
scales), and exp/log are single precision, so a dropped mass carries a relative
error of order 1e-5; H = sqrt(x / (1 + sqrt(1 - x))) halves relative errors.
|H_gpu - H_ref| <= 1e-4 and |F_gpu - F_ref| <= 1e-4 leave a 10x margin.  The
per-block log-masses are checked like lse (1e-3 absolute).
"""

import numpy as np
import pytest

from oracle import fidelity as ofid
from helpers import to_bits
from workloads import WAN14B_720P, p_for_density, qkv_for, stratified_rows, threshold_maps

pytestmark = pytest.mark.gpu

H_TOL = 1e-4
LSE_TOL = 1e-3


def _torch():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch


def _gpu_profile(q, k, rows, T, p, blk, scale):
    torch = _torch()
    from paper_2606_23019_amd import binding
    hel, fid, blk_lse = binding.fidelity_profile(
        q, k, torch.from_numpy(np.ascontiguousarray(rows, dtype=np.int32)).cuda(),
        torch.from_numpy(np.ascontiguousarray(T, dtype=np.float32)).cuda(),
        torch.from_numpy(np.ascontiguousarray(p, dtype=np.float32)).cuda(), blk, scale)
    torch.cuda.synchronize()
    return hel.cpu().numpy(), fid.cpu().numpy(), blk_lse.cpu().numpy()


def _rand_qkv(B, H, N, d, seed, scale=1.0):
    torch = _torch()
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    return tuple((torch.randn((B, H, N, d), generator=g, device="cuda") * scale).to(torch.bfloat16)
                 for _ in range(2))


CASES = [
    # (B, H, N, d, blk, R, K, seed)
    (1, 2, 1000, 64, 64, 16, 6, 1),     # ragged
    (2, 3, 777, 128, 128, 5, 3, 2),     # ragged, last block 9 keys
    (1, 1, 130, 128, 128, 1, 1, 3),     # last block 2 keys
    (1, 2, 4096, 128, 128, 32, 10, 4),  # R at its maximum
    (1, 1, 2048, 64, 128, 7, 64, 5),    # K at its maximum
]


@pytest.mark.parametrize("B,H,N,d,blk,R,K,seed", CASES)
def test_fidelity_parity_small(B, H, N, d, blk, R, K, seed):
    n = -(-N // blk)
    q, k = _rand_qkv(B, H, N, d, seed, scale=1.5)
    T = threshold_maps(H, n, n, blk, (4, 10, -(-N // 40)), seed=seed)
    rows = stratified_rows(N, H, n_strata=R, seed=seed)
    rng = np.random.default_rng(seed)
    p = np.sort(rng.uniform(-0.05, 1.0, K)).astype(np.float32)
    scale = d ** -0.5
    hel, fid, blk_lse = _gpu_profile(q, k, rows, T, p, blk, scale)
    qb, kb = to_bits(q), to_bits(k)
    ref_h, ref_f = ofid.profile(qb, kb, rows, T, p, blk, scale)
    assert np.abs(hel - ref_h).max() <= H_TOL, np.abs(hel - ref_h).max()
    assert np.abs(fid - ref_f).max() <= H_TOL, np.abs(fid - ref_f).max()
    for b in range(B):
        for h in range(H):
            for i in range(R):
                ref = ofid.block_log_mass(qb[b, h, rows[h, i]], kb[b, h], blk, scale)
                assert np.abs(blk_lse[b, h, i] - ref).max() <= LSE_TOL


def test_fidelity_edge_thresholds_and_rows():
    # rows at 0 and N - 1; candidates below every entry (nothing kept: H = 1),
    # at the top (everything kept: H = 0), a tie with map entries, and NaN
    B, H, N, d, blk = 1, 2, 900, 128, 128
    n = -(-N // blk)
    q, k = _rand_qkv(B, H, N, d, 11)
    T = threshold_maps(H, n, n, blk, (3, 10, 30), seed=11)
    T[1, 0, 3] = np.float32(0.375)
    rows = np.array([[0, 450, 899], [899, 1, 128]], dtype=np.int32)
    p = np.array([-1.0, 0.0, 0.375, 1.0, np.nan], dtype=np.float32)
    hel, fid, _ = _gpu_profile(q, k, rows, T, p, blk, d ** -0.5)
    ref_h, ref_f = ofid.profile(to_bits(q), to_bits(k), rows, T, p, blk, d ** -0.5)
    assert np.array_equal(hel[..., 0], np.ones_like(hel[..., 0]))
    assert np.array_equal(hel[..., 4], np.ones_like(hel[..., 4]))
    assert np.all(hel[..., 3] == 0.0)
    assert np.abs(hel - ref_h).max() <= H_TOL and np.abs(fid - ref_f).max() <= H_TOL
    assert np.all(np.diff(fid[..., :4], axis=-1) >= -H_TOL)


def test_fidelity_full_720p_sampled_heads():
    # 14B-720p shape: 40 heads x 75648 tokens, 16 stratified rows, 16 candidates;
    # every head on the GPU, three heads checked against the reference
    torch = _torch()
    wl = WAN14B_720P
    q, k, _ = qkv_for(wl, device="cuda")
    T = threshold_maps(wl.H, wl.n_qb, wl.n_kb, wl.blk_q, wl.grid, seed=wl.mask_seed)
    rows = stratified_rows(wl.N, wl.H, seed=wl.sample_seed)
    p = np.linspace(0.0, 1.0, 16).astype(np.float32)
    hel, fid, _ = _gpu_profile(q, k, rows, T, p, wl.blk_q, wl.scale)
    assert np.all(np.isfinite(hel)) and np.all((fid >= 0) & (fid <= 1))
    for h in (0, 17, 39):
        ref_h, ref_f = ofid.profile(to_bits(q[:, h:h + 1]), to_bits(k[:, h:h + 1]), rows[h:h + 1],
                                    T[h:h + 1], p, wl.blk_q, wl.scale)
        assert np.abs(hel[:, h:h + 1] - ref_h).max() <= H_TOL
        assert np.abs(fid[:, h:h + 1] - ref_f).max() <= H_TOL
    del q, k
    torch.cuda.empty_cache()
