"""The C-ABI library loads, exports every declared symbol, and rejects bad
arguments on the host before touching the GPU (no compute calls here)."""

import ctypes

import numpy as np
import os
import re

import pytest

from paper_2606_23019_amd import binding

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include",
                      "sa_bsattn.h")


def declared_symbols():
    txt = open(HEADER).read()
    return re.findall(r"SA_API\s+[\w\s\*]+?\b(sa_\w+)\s*\(", txt)


def test_header_declares_the_boundary():
    names = declared_symbols()
    for n in ("sa_bsattn_fwd", "sa_mask_prepass", "sa_schedule", "sa_bsattn_plan_create",
              "sa_bsattn_fwd_plan", "sa_bsattn_plan_destroy", "sa_status_string"):
        assert n in names
    assert set(names) == set(binding.SIGNATURES)


def test_library_exports_every_declared_symbol(lib):
    for name in declared_symbols():
        assert hasattr(lib, name), name


def test_status_strings(lib):
    assert binding.status_string(0) == "ok"
    assert "invalid" in binding.status_string(1)
    assert "unsupported" in binding.status_string(2)
    assert binding.status_string(99) == "unknown status"
    assert lib.sa_version() >= 100


# Fake device addresses: validation rejects these calls before any HIP call.
A = 1 << 40
MB = 1 << 30


def _fwd(lib, q=A, k=A + MB, v=A + 2 * MB, m=A + 3 * MB, out=A + 4 * MB, lse=A + 5 * MB,
         B=1, H=2, N=256, d=128, bq=128, bk=128, scale=0.088):
    P = ctypes.c_void_p
    return lib.sa_bsattn_fwd(P(q), P(k), P(v), P(m), P(out), P(lse), B, H, N, d, bq, bk,
                             ctypes.c_float(scale), None)


@pytest.mark.parametrize("kw,code", [
    (dict(q=0), binding.SA_ERR_INVALID_ARG),
    (dict(m=0), binding.SA_ERR_INVALID_ARG),
    (dict(lse=0), binding.SA_ERR_INVALID_ARG),
    (dict(q=A + 8), binding.SA_ERR_INVALID_ARG),             # misaligned
    (dict(m=A + 3 * MB + 4), binding.SA_ERR_INVALID_ARG),    # misaligned mask
    (dict(out=A + 16), binding.SA_ERR_INVALID_ARG),          # out overlaps q
    (dict(lse=A + 2 * MB + 64), binding.SA_ERR_INVALID_ARG),  # lse overlaps v
    (dict(lse=A + 4 * MB + 64), binding.SA_ERR_INVALID_ARG),  # lse overlaps out
    (dict(B=0), binding.SA_ERR_INVALID_ARG),
    (dict(N=0), binding.SA_ERR_INVALID_ARG),
    (dict(scale=0.0), binding.SA_ERR_INVALID_ARG),
    (dict(scale=float("nan")), binding.SA_ERR_INVALID_ARG),
    (dict(scale=float("inf")), binding.SA_ERR_INVALID_ARG),
    (dict(d=96), binding.SA_ERR_UNSUPPORTED),
    (dict(bq=64, bk=32), binding.SA_ERR_UNSUPPORTED),
    (dict(bq=256, bk=128), binding.SA_ERR_UNSUPPORTED),
    (dict(bq=32, bk=32), binding.SA_ERR_UNSUPPORTED),
    (dict(N=64 * 65536, bq=64, bk=64), binding.SA_ERR_UNSUPPORTED),  # n_kb > 65535
])
def test_fwd_rejects_bad_arguments_on_host(lib, kw, code):
    assert _fwd(lib, **kw) == code


def test_other_entry_points_reject_bad_arguments(lib):
    P = ctypes.c_void_p
    assert lib.sa_mask_prepass(None, 1, 1, 1, P(A), P(A + MB), None) == binding.SA_ERR_INVALID_ARG
    assert lib.sa_mask_prepass(P(A), 1, 1, 70000, P(A + MB), P(A + 2 * MB), None) == \
        binding.SA_ERR_UNSUPPORTED
    assert lib.sa_schedule(P(A), 0, 1, 1, P(A + MB), None) == binding.SA_ERR_INVALID_ARG
    h = P()
    assert lib.sa_bsattn_plan_create(P(A), 1, 1, 100, 64, 96, None, ctypes.byref(h)) == \
        binding.SA_ERR_UNSUPPORTED
    assert h.value is None
    assert lib.sa_bsattn_plan_create(P(A), 1, 1, 100, 64, 64, None, None) == \
        binding.SA_ERR_INVALID_ARG
    assert lib.sa_bsattn_fwd_plan(None, P(A), P(A), P(A), P(A), P(A), 128, ctypes.c_float(1.0),
                                  None) == binding.SA_ERR_INVALID_ARG
    n = ctypes.c_int64()
    assert lib.sa_bsattn_plan_stats(None, ctypes.byref(n)) == binding.SA_ERR_INVALID_ARG
    assert lib.sa_bsattn_plan_destroy(None) == binding.SA_ERR_INVALID_ARG


def test_f32out_entry_points_reject_bad_arguments_on_host(lib):
    P = ctypes.c_void_p

    def call(q=A, out=A + 4 * MB, lse=A + 5 * MB, d=128):
        return lib.sa_bsattn_fwd_f32out(P(q), P(A + MB), P(A + 2 * MB), P(A + 3 * MB), P(out),
                                        P(lse), 1, 2, 256, d, 128, 128, ctypes.c_float(0.088),
                                        None)
    # every call carries at least one invalid argument
    out_bf16_bytes = 2 * 256 * 128 * 2
    assert call(q=0) == binding.SA_ERR_INVALID_ARG
    assert call(out=A + 4 * MB + 8) == binding.SA_ERR_INVALID_ARG          # misaligned out
    assert call(d=96) == binding.SA_ERR_UNSUPPORTED
    # lse just past a bf16 out of this shape: inside the float32 out, so rejected
    assert call(lse=A + 4 * MB + out_bf16_bytes) == binding.SA_ERR_INVALID_ARG
    # an fp32 out starting half its size before v overlaps v
    assert call(out=A + 2 * MB - out_bf16_bytes) == binding.SA_ERR_INVALID_ARG
    assert lib.sa_bsattn_fwd_plan_f32out(None, P(A), P(A), P(A), P(A), P(A), 128,
                                         ctypes.c_float(1.0), None) == binding.SA_ERR_INVALID_ARG


def _dense(lib, q=A, k=A + MB, v=A + 2 * MB, out=A + 4 * MB, lse=A + 5 * MB,
           B=1, H=2, N=256, d=128, blk=128, scale=0.088):
    P = ctypes.c_void_p
    return lib.sa_dense_attn_fwd(P(q), P(k), P(v), P(out), P(lse), B, H, N, d, blk,
                                 ctypes.c_float(scale), None)


# every case carries at least one invalid argument: validation must stop it
@pytest.mark.parametrize("kw,code", [
    (dict(q=0), binding.SA_ERR_INVALID_ARG),
    (dict(v=0), binding.SA_ERR_INVALID_ARG),
    (dict(out=0), binding.SA_ERR_INVALID_ARG),
    (dict(lse=A + 5 * MB + 2), binding.SA_ERR_INVALID_ARG),   # misaligned lse
    (dict(k=A + MB + 8), binding.SA_ERR_INVALID_ARG),         # misaligned k
    (dict(out=A + 2 * MB + 32), binding.SA_ERR_INVALID_ARG),  # out overlaps v
    (dict(H=0), binding.SA_ERR_INVALID_ARG),
    (dict(scale=-1.0), binding.SA_ERR_INVALID_ARG),
    (dict(d=32), binding.SA_ERR_UNSUPPORTED),
    (dict(blk=256), binding.SA_ERR_UNSUPPORTED),
    (dict(N=64 * 65536, blk=64), binding.SA_ERR_UNSUPPORTED),
])
def test_dense_rejects_bad_arguments_on_host(lib, kw, code):
    assert _dense(lib, **kw) == code


def _inst(lib, T=A, p=A + MB, n_p=2, H=3, n_qb=4, n_kb=100, bits=A + 2 * MB):
    P = ctypes.c_void_p
    return lib.sa_mask_instantiate(P(T), P(p), n_p, H, n_qb, n_kb, P(bits), None)


# every case carries at least one invalid argument: validation must stop it
@pytest.mark.parametrize("kw,code", [
    (dict(T=0), binding.SA_ERR_INVALID_ARG),
    (dict(p=0), binding.SA_ERR_INVALID_ARG),
    (dict(bits=0), binding.SA_ERR_INVALID_ARG),
    (dict(T=A + 2), binding.SA_ERR_INVALID_ARG),          # misaligned map
    (dict(bits=A + 2 * MB + 4), binding.SA_ERR_INVALID_ARG),  # misaligned words
    (dict(bits=A + 64), binding.SA_ERR_INVALID_ARG),      # output overlaps the map
    (dict(bits=A + MB - 8), binding.SA_ERR_INVALID_ARG),  # output runs into p
    (dict(n_p=0), binding.SA_ERR_INVALID_ARG),
    (dict(H=0), binding.SA_ERR_INVALID_ARG),
    (dict(n_kb=0), binding.SA_ERR_INVALID_ARG),
    (dict(n_kb=65536), binding.SA_ERR_UNSUPPORTED),
])
def test_instantiate_rejects_bad_arguments_on_host(lib, kw, code):
    assert _inst(lib, **kw) == code


def _fid(lib, q=A, k=A + MB, rows=A + 2 * MB, R=16, T=A + 3 * MB, p=A + 4 * MB, K=8,
         lse=A + 5 * MB, hel=A + 6 * MB, fid=A + 7 * MB, B=1, H=2, N=1000, d=128, blk=128,
         scale=0.088):
    P = ctypes.c_void_p
    return lib.sa_fidelity_profile(P(q), P(k), P(rows), R, P(T), P(p), K, P(lse), P(hel), P(fid),
                                   B, H, N, d, blk, ctypes.c_float(scale), None)


# every case carries at least one invalid argument: validation must stop it
@pytest.mark.parametrize("kw,code", [
    (dict(q=0), binding.SA_ERR_INVALID_ARG),
    (dict(rows=0), binding.SA_ERR_INVALID_ARG),
    (dict(T=0), binding.SA_ERR_INVALID_ARG),
    (dict(fid=0), binding.SA_ERR_INVALID_ARG),
    (dict(k=A + MB + 8), binding.SA_ERR_INVALID_ARG),        # misaligned k
    (dict(hel=A + 6 * MB + 2), binding.SA_ERR_INVALID_ARG),  # misaligned output
    (dict(lse=A + 3 * MB + 16), binding.SA_ERR_INVALID_ARG),  # blk_lse overlaps T
    (dict(hel=A + 5 * MB + 64), binding.SA_ERR_INVALID_ARG),  # outputs overlap
    (dict(R=0), binding.SA_ERR_INVALID_ARG),
    (dict(K=0), binding.SA_ERR_INVALID_ARG),
    (dict(scale=0.0), binding.SA_ERR_INVALID_ARG),
    (dict(R=33), binding.SA_ERR_UNSUPPORTED),
    (dict(K=65), binding.SA_ERR_UNSUPPORTED),
    (dict(B=2, H=40000), binding.SA_ERR_UNSUPPORTED),
    (dict(d=96), binding.SA_ERR_UNSUPPORTED),
    (dict(blk=32), binding.SA_ERR_UNSUPPORTED),
])
def test_fidelity_rejects_bad_arguments_on_host(lib, kw, code):
    assert _fid(lib, **kw) == code


def test_layout_entry_rejects_bad_arguments_on_host(lib):
    P = ctypes.c_void_p

    G = 1 << 34  # spacing wide enough that the large-H case does not overlap

    def call(layout=1, H=2, d=128, q=A):
        return lib.sa_bsattn_fwd_layout(P(q), P(A + G), P(A + 2 * G), P(A + 3 * G),
                                        P(A + 4 * G), P(A + 5 * G), 1, H, 256, d, 128, 128,
                                        ctypes.c_float(0.088), layout, None)
    # every call carries at least one invalid argument
    assert call(layout=2) == binding.SA_ERR_INVALID_ARG
    assert call(layout=-1) == binding.SA_ERR_INVALID_ARG
    assert call(q=0) == binding.SA_ERR_INVALID_ARG
    assert call(d=96) == binding.SA_ERR_UNSUPPORTED
    assert call(H=65536, d=128) == binding.SA_ERR_UNSUPPORTED   # row stride too large for a tile


@pytest.mark.parametrize("fn", ["sa_resize_mask", "sa_resize_threshold_map"])
def test_resize_rejects_bad_arguments_on_host(lib, fn):
    P = ctypes.c_void_p
    f = getattr(lib, fn)
    # every call carries at least one invalid argument
    assert f(None, 1, 4, 4, P(A + MB), 8, 8, None) == binding.SA_ERR_INVALID_ARG
    assert f(P(A), 1, 4, 4, None, 8, 8, None) == binding.SA_ERR_INVALID_ARG
    assert f(P(A + 2), 1, 4, 4, P(A + MB), 8, 8, None) == binding.SA_ERR_INVALID_ARG
    assert f(P(A), 0, 4, 4, P(A + MB), 8, 8, None) == binding.SA_ERR_INVALID_ARG
    assert f(P(A), 1, 4, 4, P(A + MB), 0, 8, None) == binding.SA_ERR_INVALID_ARG
    assert f(P(A), 1, 4, 4, P(A + 8), 8, 8, None) == binding.SA_ERR_INVALID_ARG   # overlap
    assert f(P(A), 1, 4, 70000, P(A + MB), 8, 8, None) == binding.SA_ERR_UNSUPPORTED
    assert f(P(A), 1, 4, 4, P(A + MB), 8, 70000, None) == binding.SA_ERR_UNSUPPORTED


# ------------------------------------------- binding size checks (host only) ---

def test_binding_rejects_mismatched_sizes_before_any_device_call():
    import torch
    from paper_2606_23019_amd import binding
    q = torch.zeros((1, 2, 256, 64), dtype=torch.bfloat16)
    good_mask = np.zeros((2, 2, 1), dtype=np.uint64)          # H=2, n_qb=2 (blk 128), W=1
    with pytest.raises(ValueError):
        binding.bsattn_fwd(q, q, q, np.zeros((2, 1, 1), dtype=np.uint64), 128, 128)  # short mask
    with pytest.raises(ValueError):
        binding.bsattn_fwd(q, q[:, :1], q, good_mask, 128, 128)                      # k shape
    with pytest.raises(ValueError):
        binding.bsattn_fwd(q, q, q, good_mask, 128, 128,
                           lse=torch.zeros((1, 2, 255)))                              # lse shape
    with pytest.raises(ValueError):
        binding.bsattn_fwd_f32out(q, q, q, np.zeros((2, 1, 1), dtype=np.uint64), 128, 128)
    with pytest.raises(ValueError):
        binding.bsattn_fwd_f32out(q, q, q, good_mask, 128, 128,
                                  out=torch.zeros((1, 2, 255, 64)))                   # out shape
    with pytest.raises(ValueError):
        binding.bsattn_fwd_bnhd(q, q, q, np.zeros((256, 2, 1), dtype=np.uint64), 128, 128)
    with pytest.raises(ValueError):
        binding.dense_attn_fwd(q, q, q[..., :32])
    with pytest.raises(ValueError):
        binding.mask_prepass(torch.zeros((2, 2, 2), dtype=torch.int64), 2, 2, 2)     # 2 words for 1
    with pytest.raises(ValueError):
        binding.bsattn_fwd_prepared(q, q, q, torch.zeros(4, dtype=torch.int32),
                                    torch.zeros(7, dtype=torch.int32),
                                    torch.zeros(4, dtype=torch.int32), 128, 128)
    with pytest.raises(ValueError):
        binding.fidelity_profile(q, q, torch.zeros((2, 4), dtype=torch.int32),
                                 torch.zeros((2, 3, 2)), torch.zeros(3), 128)         # T shape


def test_noalloc_rejects_on_host(lib):
    """The allocation-free call checks its arguments, then the workspace size
    against the fixed scratch, before any device work."""
    P = ctypes.c_void_p
    f = ctypes.c_float(0.125)
    args = [P(A), P(A + MB), P(A + 2 * MB), P(A + 3 * MB), P(A + 4 * MB), P(A + 5 * MB)]
    assert lib.sa_bsattn_fwd_noalloc(P(0), *args[1:], 1, 2, 256, 128, 128, 128, f, None) == \
        binding.SA_ERR_INVALID_ARG
    assert lib.sa_bsattn_fwd_noalloc(*args, 1, 2, 256, 96, 128, 128, f, None) == \
        binding.SA_ERR_UNSUPPORTED
    # H 70, N 32768, 64 x 64 blocks: 70 * 512 * 512 * 4 bytes of lists alone exceed 64 MiB
    T = 1 << 33
    big = [P(A + i * T) for i in range(6)]
    assert lib.sa_bsattn_fwd_noalloc(*big, 1, 70, 32768, 64, 64, 64, f, None) == \
        binding.SA_ERR_TOO_LARGE
    assert "scratch" in binding.status_string(binding.SA_ERR_TOO_LARGE)
