"""sa_bsattn_fwd_noalloc (the entry point that allocates nothing) against
sa_bsattn_fwd, both called through the raw C ABI on device buffers the test
allocates beforehand.  Two calls in a row, the second on a smaller problem,
so the second runs on the scratch contents the first left behind; both must
equal the allocating call bit for bit.  A problem whose workspace exceeds the
fixed scratch is rejected on the host with SA_ERR_TOO_LARGE and writes
nothing."""

import ctypes

import numpy as np
import pytest

from workloads import pack_rows

pytestmark = pytest.mark.gpu


def _case(torch, B, H, N, d, blk, seed, p):
    rng = np.random.default_rng(seed)
    n = -(-N // blk)
    bm = rng.random((H, n, n)) < p
    for h in range(H):
        bm[h, np.arange(n), np.arange(n)] = True
    packed = np.ascontiguousarray(pack_rows(bm)).view(np.int64)
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    q, k, v = ((torch.randn((B, H, N, d), generator=g, device="cuda") * 1.5).to(torch.bfloat16)
               for _ in range(3))
    mask = torch.from_numpy(packed.copy()).cuda()
    return q, k, v, mask


def _call(lib, fn, torch, q, k, v, mask, blk, out, lse):
    B, H, N, d = q.shape
    P = ctypes.c_void_p
    stream = P(torch.cuda.current_stream().cuda_stream)
    return getattr(lib, fn)(P(q.data_ptr()), P(k.data_ptr()), P(v.data_ptr()),
                            P(mask.data_ptr()), P(out.data_ptr()), P(lse.data_ptr()), B, H, N, d,
                            blk, blk, ctypes.c_float(1.0 / d ** 0.5), stream)


def test_noalloc_matches_allocating_call_twice_then_rejects_too_large():
    import torch
    from paper_2606_23019_amd import binding
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    lib = binding.load(build_if_missing=False)
    for (B, H, N, d, blk, seed, p) in [(2, 6, 4000, 128, 128, 71, 0.4),   # ragged, B > 1
                                       (1, 3, 1000, 64, 64, 72, 0.3)]:    # smaller, other tile
        q, k, v, mask = _case(torch, B, H, N, d, blk, seed, p)
        ref_out = torch.empty_like(q)
        ref_lse = torch.empty((B, H, N), dtype=torch.float32, device="cuda")
        out = torch.full_like(q, 3.0)
        lse = torch.full((B, H, N), 5.0, dtype=torch.float32, device="cuda")
        assert _call(lib, "sa_bsattn_fwd", torch, q, k, v, mask, blk, ref_out, ref_lse) == 0
        assert _call(lib, "sa_bsattn_fwd_noalloc", torch, q, k, v, mask, blk, out, lse) == 0
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), ref_out.view(torch.int16)), (B, H, N, d, blk)
        assert torch.equal(lse, ref_lse), (B, H, N, d, blk)
    # H 40 at 720p-like N 75648 with 128 x 128 blocks needs 56 MB: fits; 64 x 64 blocks at
    # N 32768 and H 70 need 70 * 512 * 512 * 4 = 73 MB: rejected before any launch
    B, H, N, d, blk = 1, 70, 32768, 64, 64
    n = N // blk
    P = ctypes.c_void_p
    big = 1 << 40   # never dereferenced: the size check comes before any device work
    st = lib.sa_bsattn_fwd_noalloc(P(big), P(big + (1 << 33)), P(big + (2 << 33)),
                                   P(big + (3 << 33)), P(big + (4 << 33)), P(big + (5 << 33)),
                                   B, H, N, d, blk, blk, ctypes.c_float(0.125), None)
    assert st == binding.SA_ERR_TOO_LARGE
    assert "scratch" in binding.status_string(st)
    assert n == 512
