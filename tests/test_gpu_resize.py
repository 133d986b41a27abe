"""Conservative resize on the GPU (sa_resize_mask, sa_resize_threshold_map) vs the reference: bit-exact."""

import numpy as np
import pytest

import oracle
from oracle import resize as ors
from workloads import WAN14B_480P, WAN14B_720P, pack_rows, threshold_maps

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch


SIZES = [
    # (H, nq, nk, tq, tk, seed)
    (1, 1, 1, 5, 5, 1),          # one block grows into a 5 x 5 map
    (2, 7, 9, 11, 23, 2),
    (1, 6, 6, 12, 12, 3),        # exact 2x
    (3, 20, 30, 7, 11, 4),       # downscale (samples some rows)
    (2, 13, 17, 13, 17, 5),      # equal size
    (2, 40, 70, 100, 130, 6),    # crosses word boundaries
    (40, WAN14B_480P.n_qb, WAN14B_480P.n_kb, WAN14B_720P.n_qb, WAN14B_720P.n_kb, 7),  # 480p -> 720p
    (1, 2, 3000, 3, 8192, 8),    # mask: widest target with the column table in LDS
    (1, 3, 100, 4, 9000, 9),     # mask: target too wide for the table (points computed per word)
    (2, 5, 4100, 7, 5000, 10),   # base rows of 65 words, target rows of 79
    (3, 9, 11, 17, 13, 11),      # 17 target rows: a workgroup's last wavefront has fewer rows
]


@pytest.mark.parametrize("H,nq,nk,tq,tk,seed", SIZES)
def test_resize_threshold_map_bit_exact(H, nq, nk, tq, tk, seed):
    torch = _torch()
    from paper_2606_23019_amd import binding
    T = np.random.default_rng(seed).random((H, nq, nk)).astype(np.float32)
    T.reshape(-1)[::97] = np.nan
    got = binding.resize_threshold_map(torch.from_numpy(T).cuda(), tq, tk)
    torch.cuda.synchronize()
    ref = ors.resize_threshold_map(T, tq, tk)
    assert np.array_equal(got.cpu().numpy(), ref, equal_nan=True)


@pytest.mark.parametrize("H,nq,nk,tq,tk,seed", SIZES)
def test_resize_mask_bit_exact(H, nq, nk, tq, tk, seed):
    torch = _torch()
    from paper_2606_23019_amd import binding
    M = np.random.default_rng(seed).random((H, nq, nk)) < 0.15
    packed = pack_rows(M)
    packed[..., -1] |= np.uint64(0xFFFF000000000000) if nk % 64 and nk % 64 <= 48 else np.uint64(0)
    got = binding.resize_mask(packed, nk, tq, tk)
    torch.cuda.synchronize()
    ref = oracle.pack_crm(ors.resize_mask(M, tq, tk))
    assert np.array_equal(got.cpu().numpy().view(np.uint64), ref)


def test_resize_commutes_with_instantiation_on_gpu():
    # 480p threshold maps -> 720p: instantiating the resized map equals resizing the mask
    torch = _torch()
    from paper_2606_23019_amd import binding
    a, b = WAN14B_480P, WAN14B_720P
    T = threshold_maps(a.H, a.n_qb, a.n_kb, a.blk_q, a.grid, seed=a.mask_seed)
    Td = torch.from_numpy(T).cuda()
    p = torch.from_numpy(np.random.default_rng(9).uniform(0.05, 0.6, (3, a.H)).astype(np.float32)).cuda()
    lhs = binding.mask_instantiate(binding.resize_threshold_map(Td, b.n_qb, b.n_kb), p)
    masks = binding.mask_instantiate(Td, p)
    rhs = torch.stack([binding.resize_mask(masks[i], a.n_kb, b.n_qb, b.n_kb) for i in range(3)])
    torch.cuda.synchronize()
    assert torch.equal(lhs, rhs)
