"""ctypes binding of ``libsa_bsattn.so`` (C ABI declared in include/sa_bsattn.h).

Argument marshalling only: every step of the forward pass runs in the HIP
library.  PyTorch supplies device buffers and the current stream.  There is no
fallback: if the library cannot be loaded the functions raise.
"""

import ctypes
import os

import numpy as np

from . import build as _build

SA_OK = 0
SA_ERR_INVALID_ARG = 1
SA_ERR_UNSUPPORTED = 2
SA_ERR_HIP = 3
SA_ERR_TOO_LARGE = 4
SA_LAYOUT_BHND = 0
SA_LAYOUT_BNHD = 1

_LIB = None

_P = ctypes.c_void_p
_I = ctypes.c_int
_F = ctypes.c_float

# name -> (restype, argtypes); mirrors include/sa_bsattn.h
SIGNATURES = {
    "sa_status_string": (ctypes.c_char_p, [_I]),
    "sa_version": (_I, []),
    "sa_bsattn_fwd": (_I, [_P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _F, _P]),
    "sa_mask_prepass": (_I, [_P, _I, _I, _I, _P, _P, _P]),
    "sa_schedule": (_I, [_P, _I, _I, _I, _P, _P]),
    "sa_bsattn_fwd_prepared": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _F, _P]),
    "sa_bsattn_plan_create": (_I, [_P, _I, _I, _I, _I, _I, _P, ctypes.POINTER(_P)]),
    "sa_bsattn_fwd_plan": (_I, [_P, _P, _P, _P, _P, _P, _I, _F, _P]),
    "sa_bsattn_fwd_f32out": (_I, [_P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _F, _P]),
    "sa_bsattn_fwd_noalloc": (_I, [_P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _F, _P]),
    "sa_bsattn_fwd_plan_f32out": (_I, [_P, _P, _P, _P, _P, _P, _I, _F, _P]),
    "sa_bsattn_plan_stats": (_I, [_P, ctypes.POINTER(ctypes.c_int64)]),
    "sa_bsattn_plan_destroy": (_I, [_P]),
    "sa_dense_attn_fwd": (_I, [_P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _F, _P]),
    "sa_mask_instantiate": (_I, [_P, _P, _I, _I, _I, _I, _P, _P]),
    "sa_bsattn_fwd_layout": (_I, [_P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _F, _I, _P]),
    "sa_resize_mask": (_I, [_P, _I, _I, _I, _P, _I, _I, _P]),
    "sa_resize_threshold_map": (_I, [_P, _I, _I, _I, _P, _I, _I, _P]),
    "sa_fidelity_profile": (_I, [_P, _P, _P, _I, _P, _P, _I, _P, _P, _P, _I, _I, _I, _I, _I, _F,
                                 _P]),
}


class SAError(RuntimeError):
    def __init__(self, fn, status):
        self.status = status
        super().__init__("%s failed: %s (status %d)" % (fn, status_string(status), status))


def library_path():
    return _build.LIB_PATH


def load(build_if_missing=True):
    """Load the library (building it in-tree only if it is absent)."""
    global _LIB
    if _LIB is not None:
        return _LIB
    path = library_path()
    if not os.path.exists(path):
        if not build_if_missing:
            raise RuntimeError("HIP library %s is not built" % path)
        _build.build()
    lib = ctypes.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _LIB = lib
    return lib


def status_string(status):
    return load().sa_status_string(int(status)).decode()


def _check(fn, status):
    if status != SA_OK:
        raise SAError(fn, status)


# --------------------------------------------------------------- tensors ---

def _torch():
    import torch
    return torch


def _dev_ptr(t, dtype, name):
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch tensor" % name)
    if t.device.type != "cuda":
        raise ValueError("%s must be on the GPU, got %s" % (name, t.device))
    if t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    return ctypes.c_void_p(t.data_ptr())


def _need(cond, msg):
    """Size checks on the host: the C ABI takes raw pointers and cannot see buffer sizes."""
    if not cond:
        raise ValueError(msg)


def _same_shape(ref, others, names):
    for t, n in zip(others, names):
        _need(tuple(t.shape) == tuple(ref.shape), "%s has shape %s, expected %s"
              % (n, tuple(t.shape), tuple(ref.shape)))


def _outputs(q, out, lse, lse_shape, out_dtype=None):
    torch = _torch()
    if out is None:
        out = torch.empty_like(q, dtype=out_dtype or q.dtype)
    _need(tuple(out.shape) == tuple(q.shape), "out must have the shape of q")
    if lse is None:
        lse = torch.empty(lse_shape, dtype=torch.float32, device=q.device)
    _need(tuple(lse.shape) == tuple(lse_shape), "lse must have shape %s" % (tuple(lse_shape),))
    return out, lse


def _mask_words(m, H, n_qb, n_kb):
    _need(m.numel() == H * n_qb * ((n_kb + 63) // 64),
          "mask has %d words, expected H * n_qb * ceil(n_kb / 64) = %d"
          % (m.numel(), H * n_qb * ((n_kb + 63) // 64)))


def _stream(stream):
    torch = _torch()
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _used_on(stream, *tensors):
    """Tensors made here and used by work on a stream other than the current one:
    the caching allocator must not hand their memory out again before that
    stream's work on them is done (it only tracks the current stream by itself)."""
    if stream is None:
        return
    torch = _torch()
    if stream == torch.cuda.current_stream():
        return
    for t in tensors:
        t.record_stream(stream)


def mask_to_device(mask_bits, device="cuda"):
    """uint64 numpy [H, n_qb, W] -> int64 torch tensor (same bits) on ``device``."""
    torch = _torch()
    if isinstance(mask_bits, torch.Tensor):
        return mask_bits.to(device).contiguous()
    m = np.ascontiguousarray(mask_bits, dtype=np.uint64).view(np.int64)
    return torch.from_numpy(m.copy()).to(device)


def _fwd_oneshot(fn, out_dtype, q, k, v, mask_bits, blk_q, blk_k, scale, out, lse, stream):
    torch = _torch()
    lib = load()
    B, H, N, d = q.shape
    _same_shape(q, (k, v), ("k", "v"))
    if scale is None:
        scale = 1.0 / float(d) ** 0.5
    m = mask_to_device(mask_bits, q.device)
    if m.dtype == torch.uint64:
        m = m.view(torch.int64)
    _mask_words(m, H, -(-N // int(blk_q)), -(-N // int(blk_k)))
    out, lse = _outputs(q, out, lse, (B, H, N), out_dtype)
    st = getattr(lib, fn)(
        _dev_ptr(q, torch.bfloat16, "q"), _dev_ptr(k, torch.bfloat16, "k"),
        _dev_ptr(v, torch.bfloat16, "v"), _dev_ptr(m, torch.int64, "mask_bits"),
        _dev_ptr(out, out_dtype, "out"), _dev_ptr(lse, torch.float32, "lse"),
        B, H, N, d, int(blk_q), int(blk_k), float(scale), _stream(stream))
    _check(fn, st)
    _used_on(stream, m, out, lse)
    return out, lse


def bsattn_fwd(q, k, v, mask_bits, blk_q, blk_k, scale=None, out=None, lse=None, stream=None):
    """One-shot forward: ``sa_bsattn_fwd``.  q, k, v: bf16 [B, H, N, d] on the GPU.

    mask_bits: int64/uint64 device tensor (or numpy uint64) [H, n_qb, W].
    Returns (out bf16 [B, H, N, d], lse float32 [B, H, N]).
    """
    return _fwd_oneshot("sa_bsattn_fwd", _torch().bfloat16, q, k, v, mask_bits, blk_q, blk_k,
                        scale, out, lse, stream)


def bsattn_fwd_f32out(q, k, v, mask_bits, blk_q, blk_k, scale=None, out=None, lse=None,
                      stream=None):
    """``sa_bsattn_fwd_f32out``: as ``bsattn_fwd`` with out float32 [B, H, N, d]."""
    return _fwd_oneshot("sa_bsattn_fwd_f32out", _torch().float32, q, k, v, mask_bits, blk_q,
                        blk_k, scale, out, lse, stream)


def bsattn_fwd_bnhd(q, k, v, mask_bits, blk_q, blk_k, scale=None, out=None, lse=None,
                    stream=None):
    """``sa_bsattn_fwd_layout`` with q, k, v, out in [B, N, H, d]; lse is [B, H, N]."""
    torch = _torch()
    lib = load()
    B, N, H, d = q.shape
    _same_shape(q, (k, v), ("k", "v"))
    if scale is None:
        scale = 1.0 / float(d) ** 0.5
    m = mask_to_device(mask_bits, q.device)
    if m.dtype == torch.uint64:
        m = m.view(torch.int64)
    _mask_words(m, H, -(-N // int(blk_q)), -(-N // int(blk_k)))
    out, lse = _outputs(q, out, lse, (B, H, N))
    st = lib.sa_bsattn_fwd_layout(
        _dev_ptr(q, torch.bfloat16, "q"), _dev_ptr(k, torch.bfloat16, "k"),
        _dev_ptr(v, torch.bfloat16, "v"), _dev_ptr(m, torch.int64, "mask_bits"),
        _dev_ptr(out, torch.bfloat16, "out"), _dev_ptr(lse, torch.float32, "lse"),
        B, H, N, d, int(blk_q), int(blk_k), float(scale), SA_LAYOUT_BNHD, _stream(stream))
    _check("sa_bsattn_fwd_layout", st)
    _used_on(stream, m, out, lse)
    return out, lse


def dense_attn_fwd(q, k, v, blk=128, scale=None, out=None, lse=None, stream=None):
    """``sa_dense_attn_fwd``: maskless attention (every key block enabled)."""
    torch = _torch()
    lib = load()
    B, H, N, d = q.shape
    _same_shape(q, (k, v), ("k", "v"))
    if scale is None:
        scale = 1.0 / float(d) ** 0.5
    out, lse = _outputs(q, out, lse, (B, H, N))
    st = lib.sa_dense_attn_fwd(
        _dev_ptr(q, torch.bfloat16, "q"), _dev_ptr(k, torch.bfloat16, "k"),
        _dev_ptr(v, torch.bfloat16, "v"), _dev_ptr(out, torch.bfloat16, "out"),
        _dev_ptr(lse, torch.float32, "lse"), B, H, N, d, int(blk), float(scale), _stream(stream))
    _check("sa_dense_attn_fwd", st)
    _used_on(stream, out, lse)
    return out, lse


def mask_instantiate(T, p, out=None, stream=None):
    """``sa_mask_instantiate``: CRM masks 1[T <= p] for every threshold set.

    T: float32 device tensor [H, n_qb, n_kb]; p: float32 device tensor [n_p, H].
    Returns int64 (uint64 bits) [n_p, H, n_qb, W].
    """
    torch = _torch()
    lib = load()
    H, n_qb, n_kb = T.shape
    n_p = p.shape[0]
    if tuple(p.shape) != (n_p, H):
        raise ValueError("p must be [n_p, H]")
    W = (n_kb + 63) // 64
    if out is None:
        out = torch.empty((n_p, H, n_qb, W), dtype=torch.int64, device=T.device)
    _need(out.numel() == n_p * H * n_qb * W, "out must hold n_p * H * n_qb * W words")
    st = lib.sa_mask_instantiate(_dev_ptr(T, torch.float32, "T"), _dev_ptr(p, torch.float32, "p"),
                                 n_p, H, n_qb, n_kb, _dev_ptr(out, torch.int64, "mask_bits"),
                                 _stream(stream))
    _check("sa_mask_instantiate", st)
    _used_on(stream, out)
    return out


def fidelity_profile(q, k, rows, T, p, blk, scale=None, stream=None):
    """``sa_fidelity_profile``: returns (hellinger [B,H,R,K], fidelity [B,H,K], blk_lse [B,H,R,n_kb]).

    rows: int32 device tensor [H, R]; T: float32 device [H, n_qb, n_kb]; p: float32 device [K].
    """
    torch = _torch()
    lib = load()
    B, H, N, d = q.shape
    _same_shape(q, (k,), ("k",))
    _need(rows.dim() == 2 and rows.shape[0] == H, "rows must be [H, R]")
    R = rows.shape[1]
    _need(p.dim() == 1, "p must be [K]")
    K = p.shape[0]
    n_kb = (N + blk - 1) // blk
    _need(tuple(T.shape) == (H, n_kb, n_kb), "T must be [H, n_qb, n_kb] = %s" % ((H, n_kb, n_kb),))
    if scale is None:
        scale = 1.0 / float(d) ** 0.5
    dev = q.device
    blk_lse = torch.empty((B, H, R, n_kb), dtype=torch.float32, device=dev)
    hel = torch.empty((B, H, R, K), dtype=torch.float32, device=dev)
    fid = torch.empty((B, H, K), dtype=torch.float32, device=dev)
    st = lib.sa_fidelity_profile(
        _dev_ptr(q, torch.bfloat16, "q"), _dev_ptr(k, torch.bfloat16, "k"),
        _dev_ptr(rows, torch.int32, "rows"), R, _dev_ptr(T, torch.float32, "T"),
        _dev_ptr(p, torch.float32, "p"), K, _dev_ptr(blk_lse, torch.float32, "blk_lse"),
        _dev_ptr(hel, torch.float32, "hellinger"), _dev_ptr(fid, torch.float32, "fidelity"),
        B, H, N, d, int(blk), float(scale), _stream(stream))
    _check("sa_fidelity_profile", st)
    _used_on(stream, blk_lse, hel, fid)
    return hel, fid, blk_lse


def resize_threshold_map(T, n_qb_out, n_kb_out, stream=None):
    """``sa_resize_threshold_map``: float32 [H, n_qb, n_kb] -> [H, n_qb_out, n_kb_out]."""
    torch = _torch()
    lib = load()
    H, n_qb, n_kb = T.shape
    out = torch.empty((H, n_qb_out, n_kb_out), dtype=torch.float32, device=T.device)
    st = lib.sa_resize_threshold_map(_dev_ptr(T, torch.float32, "T"), H, n_qb, n_kb,
                                     _dev_ptr(out, torch.float32, "T_out"), n_qb_out, n_kb_out,
                                     _stream(stream))
    _check("sa_resize_threshold_map", st)
    _used_on(stream, out)
    return out


def resize_mask(mask_bits, n_kb, n_qb_out, n_kb_out, stream=None):
    """``sa_resize_mask``: CRM int64 [H, n_qb, W] (n_kb key blocks) -> [H, n_qb_out, W_out]."""
    torch = _torch()
    lib = load()
    m = mask_to_device(mask_bits)
    if m.dtype == torch.uint64:
        m = m.view(torch.int64)
    H, n_qb, _ = m.shape
    _mask_words(m, H, n_qb, n_kb)
    out = torch.full((H, n_qb_out, (n_kb_out + 63) // 64), -1, dtype=torch.int64, device=m.device)
    st = lib.sa_resize_mask(_dev_ptr(m, torch.int64, "mask_bits"), H, n_qb, n_kb,
                            _dev_ptr(out, torch.int64, "mask_out"), n_qb_out, n_kb_out,
                            _stream(stream))
    _check("sa_resize_mask", st)
    _used_on(stream, m, out)
    return out


def mask_prepass(mask_bits, H, n_qb, n_kb, stream=None):
    """``sa_mask_prepass``: returns (counts int32 [H*n_qb], lists int32 [H*n_qb, n_kb])."""
    torch = _torch()
    lib = load()
    m = mask_to_device(mask_bits, mask_bits.device if isinstance(mask_bits, torch.Tensor) else "cuda")
    if m.dtype == torch.uint64:
        m = m.view(torch.int64)
    _mask_words(m, H, n_qb, n_kb)
    counts = torch.full((H * n_qb,), -1, dtype=torch.int32, device=m.device)
    lists = torch.full((H * n_qb, n_kb), -1, dtype=torch.int32, device=m.device)
    st = lib.sa_mask_prepass(_dev_ptr(m, torch.int64, "mask_bits"), H, n_qb, n_kb,
                             _dev_ptr(counts, torch.int32, "counts"),
                             _dev_ptr(lists, torch.int32, "lists"), _stream(stream))
    _check("sa_mask_prepass", st)
    _used_on(stream, m, counts, lists)
    return counts, lists


def schedule(counts, B, H, n_qb, stream=None):
    """``sa_schedule``: returns order int32 [B*H*n_qb]."""
    torch = _torch()
    lib = load()
    _need(counts.numel() == H * n_qb, "counts must hold H * n_qb entries")
    order = torch.full((B * H * n_qb,), -1, dtype=torch.int32, device=counts.device)
    st = lib.sa_schedule(_dev_ptr(counts, torch.int32, "counts"), B, H, n_qb,
                         _dev_ptr(order, torch.int32, "order"), _stream(stream))
    _check("sa_schedule", st)
    _used_on(stream, order)
    return order


def bsattn_fwd_prepared(q, k, v, counts, lists, order, blk_q, blk_k, scale=None, out=None,
                        lse=None, stream=None):
    """``sa_bsattn_fwd_prepared``: attention kernel on a given pre-pass and schedule."""
    torch = _torch()
    lib = load()
    B, H, N, d = q.shape
    _same_shape(q, (k, v), ("k", "v"))
    n_qb, n_kb = -(-N // int(blk_q)), -(-N // int(blk_k))
    _need(counts.numel() == H * n_qb, "counts must hold H * n_qb entries")
    _need(lists.numel() == H * n_qb * n_kb, "lists must hold H * n_qb * n_kb entries")
    _need(order.numel() == B * H * n_qb, "order must hold B * H * n_qb entries")
    if scale is None:
        scale = 1.0 / float(d) ** 0.5
    out, lse = _outputs(q, out, lse, (B, H, N))
    st = lib.sa_bsattn_fwd_prepared(
        _dev_ptr(q, torch.bfloat16, "q"), _dev_ptr(k, torch.bfloat16, "k"),
        _dev_ptr(v, torch.bfloat16, "v"), _dev_ptr(counts, torch.int32, "counts"),
        _dev_ptr(lists, torch.int32, "lists"), _dev_ptr(order, torch.int32, "order"),
        _dev_ptr(out, torch.bfloat16, "out"), _dev_ptr(lse, torch.float32, "lse"),
        B, H, N, d, int(blk_q), int(blk_k), float(scale), _stream(stream))
    _check("sa_bsattn_fwd_prepared", st)
    _used_on(stream, out, lse)
    return out, lse


class Plan:
    """Static-mask plan (``sa_bsattn_plan_*``): pre-pass and schedule done once."""

    def __init__(self, mask_bits, B, H, N, blk_q, blk_k, stream=None):
        torch = _torch()
        self._lib = load()
        self._m = mask_to_device(mask_bits)
        if self._m.dtype == torch.uint64:
            self._m = self._m.view(torch.int64)
        _mask_words(self._m, H, -(-N // int(blk_q)), -(-N // int(blk_k)))
        self.B, self.H, self.N, self.blk_q, self.blk_k = B, H, N, blk_q, blk_k
        h = ctypes.c_void_p()
        st = self._lib.sa_bsattn_plan_create(_dev_ptr(self._m, torch.int64, "mask_bits"), B, H, N,
                                             blk_q, blk_k, _stream(stream), ctypes.byref(h))
        _check("sa_bsattn_plan_create", st)
        self._h = h

    @property
    def executed_blocks(self):
        n = ctypes.c_int64()
        _check("sa_bsattn_plan_stats", self._lib.sa_bsattn_plan_stats(self._h, ctypes.byref(n)))
        return n.value

    def _fwd(self, fn, out_dtype, q, k, v, scale, out, lse, stream):
        torch = _torch()
        B, H, N, d = q.shape
        if (B, H, N) != (self.B, self.H, self.N):
            raise ValueError("q shape %s does not match the plan" % (tuple(q.shape),))
        _same_shape(q, (k, v), ("k", "v"))
        if scale is None:
            scale = 1.0 / float(d) ** 0.5
        out, lse = _outputs(q, out, lse, (B, H, N), out_dtype)
        st = getattr(self._lib, fn)(
            self._h, _dev_ptr(q, torch.bfloat16, "q"), _dev_ptr(k, torch.bfloat16, "k"),
            _dev_ptr(v, torch.bfloat16, "v"), _dev_ptr(out, out_dtype, "out"),
            _dev_ptr(lse, torch.float32, "lse"), d, float(scale), _stream(stream))
        _check(fn, st)
        _used_on(stream, out, lse)
        return out, lse

    def __call__(self, q, k, v, scale=None, out=None, lse=None, stream=None):
        """``sa_bsattn_fwd_plan``: (out bf16 [B, H, N, d], lse float32 [B, H, N])."""
        return self._fwd("sa_bsattn_fwd_plan", _torch().bfloat16, q, k, v, scale, out, lse,
                         stream)

    def fwd_f32out(self, q, k, v, scale=None, out=None, lse=None, stream=None):
        """``sa_bsattn_fwd_plan_f32out``: as the call, with out float32."""
        return self._fwd("sa_bsattn_fwd_plan_f32out", _torch().float32, q, k, v, scale, out, lse,
                         stream)

    def close(self):
        if getattr(self, "_h", None):
            self._lib.sa_bsattn_plan_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
