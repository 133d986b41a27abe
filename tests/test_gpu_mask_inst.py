"""Mask instantiation on the GPU (sa_mask_instantiate) vs the reference: bit-exact."""

import numpy as np
import pytest

import oracle
from helpers import compare, to_bits
from workloads import WAN14B_720P, threshold_maps, p_for_density

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch


def _run(T, p, dirty=True):
    torch = _torch()
    from paper_2606_23019_amd import binding
    Td = torch.from_numpy(np.ascontiguousarray(T, dtype=np.float32)).cuda()
    pd = torch.from_numpy(np.ascontiguousarray(p, dtype=np.float32)).cuda()
    n_p, (H, n_qb, n_kb) = p.shape[0], T.shape
    out = torch.full((n_p, H, n_qb, (n_kb + 63) // 64), -0x5A5A5A5A5A5A5A5B if dirty else 0,
                     dtype=torch.int64, device="cuda")
    binding.mask_instantiate(Td, pd, out=out)
    torch.cuda.synchronize()
    return out.cpu().numpy().view(np.uint64)


SHAPES = [
    # (H, n_qb, n_kb, n_p, seed)
    (1, 1, 1, 1, 1),
    (2, 3, 63, 1, 2),
    (2, 3, 64, 2, 3),
    (3, 5, 65, 3, 4),
    (4, 7, 130, 1, 5),
    (2, 4, 591, 5, 6),
    (1, 2, 4097, 2, 7),     # 65 words: two chunks of the row loop
    (2, 2, 65535, 1, 8),    # largest supported row
    (3, 6, 256, 16, 9),     # one full set of 16 thresholds per wavefront
    (2, 5, 300, 17, 10),    # 16 + 1: a second set of one threshold
    (4, 9, 591, 50, 11),    # the 50 timesteps of one layer: 4 sets, the last of 2
]


@pytest.mark.parametrize("H,n_qb,n_kb,n_p,seed", SHAPES)
def test_instantiate_bit_exact(H, n_qb, n_kb, n_p, seed):
    rng = np.random.default_rng(seed)
    T = rng.random((H, n_qb, n_kb)).astype(np.float32)
    p = rng.random((n_p, H)).astype(np.float32)
    got = _run(T, p)
    ref = oracle.instantiate_packed(T, p)
    assert got.shape == ref.shape and np.array_equal(got, ref)


def test_instantiate_ties_nan_and_extremes():
    T = np.array([[[0.0, 0.5, np.nan, 1.0, 0.5, np.inf, -np.inf] * 20]], dtype=np.float32)
    p = np.array([[0.5], [np.nan], [-1.0], [np.inf], [0.0]], dtype=np.float32)
    got = _run(T, p)
    assert np.array_equal(got, oracle.instantiate_packed(T, p))


def test_instantiate_full_720p_maps():
    # 14B-720p shape: 40 heads of 591 x 591 blocks, per-head densities, 4 timesteps
    wl = WAN14B_720P
    T = threshold_maps(wl.H, wl.n_qb, wl.n_kb, wl.blk_q, wl.grid, seed=wl.mask_seed)
    rng = np.random.default_rng(wl.sample_seed)
    p = np.stack([p_for_density(T, rng.uniform(0.05, 0.3, wl.H)) for _ in range(4)])
    got = _run(T, p)
    assert np.array_equal(got, oracle.instantiate_packed(T, p))


def test_instantiated_masks_drive_attention():
    # instantiate on the GPU, run the CRM path on those bits, check against the
    # reference attention on the reference-instantiated mask
    torch = _torch()
    from paper_2606_23019_amd import binding
    B, H, N, d, blk = 1, 3, 1000, 128, 128
    n = -(-N // blk)
    T = threshold_maps(H, n, n, blk, (4, 10, 25), seed=77)
    p = p_for_density(T, np.array([0.2, 0.5, 0.8]))[None]
    bits = binding.mask_instantiate(torch.from_numpy(T).cuda(), torch.from_numpy(p).cuda())
    g = torch.Generator(device="cuda")
    g.manual_seed(78)
    q, k, v = (torch.randn((B, H, N, d), generator=g, device="cuda").to(torch.bfloat16)
               for _ in range(3))
    out, lse = binding.bsattn_fwd(q, k, v, bits[0].contiguous(), blk, blk)
    torch.cuda.synchronize()
    ref_mask = oracle.instantiate_packed(T, p)[0]
    ro, rl = oracle.attention(to_bits(q), to_bits(k), to_bits(v), ref_mask, blk, blk, d ** -0.5)
    print(compare(out.float().cpu().numpy(), lse.cpu().numpy(), ro, rl))
