"""Maskless dense path (sa_dense_attn_fwd) vs the float64 reference and vs the CRM path."""

import numpy as np
import pytest

import oracle
from helpers import compare, to_bits
from workloads import pack_rows, sample_items

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch


def _rand_qkv(B, H, N, d, seed, scale=1.0):
    torch = _torch()
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    return tuple((torch.randn((B, H, N, d), generator=g, device="cuda") * scale).to(torch.bfloat16)
                 for _ in range(3))


def _ones(H, N, blk):
    n = -(-N // blk)
    return pack_rows(np.ones((H, n, n), dtype=bool))


DENSE_CASES = [
    # (B, H, N, d, blk, seed)
    (1, 1, 64, 64, 64, 1),        # one block
    (2, 3, 1000, 64, 64, 2),      # ragged
    (1, 2, 1000, 128, 64, 3),
    (2, 2, 1000, 64, 128, 4),
    (1, 2, 777, 128, 128, 5),     # ragged, last block 9 keys
    (1, 1, 130, 128, 128, 6),     # last block 2 keys
    (1, 2, 4096, 128, 128, 7),    # several tiles, no tail
]


@pytest.mark.parametrize("B,H,N,d,blk,seed", DENSE_CASES)
def test_dense_parity_vs_reference(B, H, N, d, blk, seed):
    torch = _torch()
    from paper_2606_23019_amd import binding
    q, k, v = _rand_qkv(B, H, N, d, seed, scale=1.5)
    out, lse = binding.dense_attn_fwd(q, k, v, blk)
    torch.cuda.synchronize()
    ref_out, ref_lse = oracle.attention(to_bits(q), to_bits(k), to_bits(v), _ones(H, N, blk), blk,
                                        blk, 1.0 / d ** 0.5)
    print(compare(out.float().cpu().numpy(), lse.cpu().numpy(), ref_out, ref_lse))


@pytest.mark.parametrize("B,H,N,d,blk,seed", DENSE_CASES)
def test_dense_equals_crm_path_with_all_ones_mask(B, H, N, d, blk, seed):
    # same kernel, same ascending key-block order: identical bits
    torch = _torch()
    from paper_2606_23019_amd import binding
    q, k, v = _rand_qkv(B, H, N, d, 100 + seed)
    o1, l1 = binding.dense_attn_fwd(q, k, v, blk)
    o2, l2 = binding.bsattn_fwd(q, k, v, _ones(H, N, blk), blk, blk)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_dense_full_size_sampled():
    # 14B-480p shape (H40, N32768, d128) at 0 % sparsity, sampled query blocks
    torch = _torch()
    from paper_2606_23019_amd import binding
    from workloads import WAN14B_480P, qkv_for
    wl = WAN14B_480P
    q, k, v = qkv_for(wl, device="cuda")
    out, lse = binding.dense_attn_fwd(q, k, v, wl.blk_q, wl.scale)
    torch.cuda.synchronize()
    bm = np.ones((wl.H, wl.n_qb, wl.n_kb), dtype=bool)
    items = sample_items(wl, bm, 16)
    go, gl, ro, rl = [], [], [], []
    allowed = np.ones(wl.n_kb, dtype=bool)
    for (b, h, u) in items:
        r0, r1 = u * wl.blk_q, min((u + 1) * wl.blk_q, wl.N)
        ref = oracle.attention_block(to_bits(q[b, h, r0:r1]), to_bits(k[b, h]), to_bits(v[b, h]),
                                     allowed, wl.blk_k, wl.scale)
        go.append(out[b, h, r0:r1].float().cpu().numpy())
        gl.append(lse[b, h, r0:r1].cpu().numpy())
        ro.append(ref[0])
        rl.append(ref[1])
    print(compare(np.concatenate(go), np.concatenate(gl), np.concatenate(ro), np.concatenate(rl)))
    assert torch.isfinite(out).all().item() and torch.isfinite(lse).all().item()
    del q, k, v, out, lse
    torch.cuda.empty_cache()
