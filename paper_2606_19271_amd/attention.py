"""Torch-facing binding of the C ABI (ts_attn_fwd, ts_attn_fwd_varlen, ts_attn_fwd_kvcache,
ts_attn_fwd_kvcache_noalloc): argument marshalling only.

Every step of the computation runs in libts_attn.so on the tensors' device and on torch's current
stream of that device; nothing here computes attention, and there is no fallback path.
"""
import ctypes

import numpy as np
import torch

from . import _lib


def default_scale(d):
    """1/sqrt(d) rounded to float32 (the conventional softmax temperature)."""
    return float(np.float32(1.0) / np.sqrt(np.float32(d)))


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr())


def _check_tensor(name, t, ndim):
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % name)
    if t.dtype != torch.bfloat16 or t.dim() != ndim or not t.is_cuda or not t.is_contiguous():
        raise ValueError("%s must be a contiguous bfloat16 GPU tensor with %d dims" % (name, ndim))


def ts_attn_fwd(q, k, v, scale=None, out=None):
    """Dense batch: q, k, v are [B, L, H, d]; returns o = softmax(scale q k^T) v per sequence."""
    for name, t in (("q", q), ("k", k), ("v", v)):
        _check_tensor(name, t, 4)
    if k.shape != q.shape or v.shape != q.shape or k.device != q.device or v.device != q.device:
        raise ValueError("q, k, v must have one shape and device")
    B, L, H, d = q.shape
    if out is None:
        out = torch.empty_like(q)
    else:
        _check_tensor("out", out, 4)
        if out.shape != q.shape or out.device != q.device:
            raise ValueError("out must match q")
    s = default_scale(d) if scale is None else float(scale)
    lib = _lib.load()
    with torch.cuda.device(q.device):
        stream = torch.cuda.current_stream(q.device).cuda_stream
        rc = lib.ts_attn_fwd(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _lib.i32("B", B),
                             _lib.i32("L", L), _lib.i32("H", H), _lib.i32("d", d), s,
                             ctypes.c_void_p(stream))
    _lib.check(rc)
    return out


def ts_attn_fwd_varlen(q, k, v, cu_seqlens, max_seqlen, scale=None, out=None):
    """Packed batch: q, k, v are [T, H, d]; cu_seqlens is an int32 GPU tensor of nseq+1
    offsets (segment s = tokens [cu[s], cu[s+1])); max_seqlen bounds every segment length.
    Returns o with attention restricted to each segment."""
    for name, t in (("q", q), ("k", k), ("v", v)):
        _check_tensor(name, t, 3)
    if k.shape != q.shape or v.shape != q.shape or k.device != q.device or v.device != q.device:
        raise ValueError("q, k, v must have one shape and device")
    if (not isinstance(cu_seqlens, torch.Tensor) or cu_seqlens.dtype != torch.int32
            or cu_seqlens.dim() != 1 or cu_seqlens.numel() < 1 or cu_seqlens.device != q.device
            or not cu_seqlens.is_contiguous()):
        raise ValueError("cu_seqlens must be a contiguous int32 tensor on q's device")
    T, H, d = q.shape
    if out is None:
        out = torch.empty_like(q)
    else:
        _check_tensor("out", out, 3)
        if out.shape != q.shape or out.device != q.device:
            raise ValueError("out must match q")
    s = default_scale(d) if scale is None else float(scale)
    lib = _lib.load()
    with torch.cuda.device(q.device):
        stream = torch.cuda.current_stream(q.device).cuda_stream
        rc = lib.ts_attn_fwd_varlen(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(cu_seqlens),
                                    _lib.i32("nseq", cu_seqlens.numel() - 1),
                                    _lib.i32("max_seqlen", max_seqlen), _lib.i32("T", T),
                                    _lib.i32("H", H), _lib.i32("d", d), s, ctypes.c_void_p(stream))
    _lib.check(rc)
    return out


def _check_offsets(name, cu, device):
    if (not isinstance(cu, torch.Tensor) or cu.dtype != torch.int32 or cu.dim() != 1
            or cu.numel() < 1 or cu.device != device or not cu.is_contiguous()):
        raise ValueError("%s must be a contiguous int32 tensor on q's device" % name)


def ts_attn_fwd_kvcache(q, k, v, cu_seqlens_q, cu_seqlens_k, max_seqlen_q, max_seqlen_k,
                        scale=None, out=None, lse=None, return_lse=False, num_splits=0):
    """Chunk queries against per-session key/value caches.

    q is [Tq, H, d] and k, v are [Tk, H, d] (bfloat16, same device); segment s has queries
    q[cu_seqlens_q[s]:cu_seqlens_q[s+1]] and keys/values k, v[cu_seqlens_k[s]:cu_seqlens_k[s+1]]
    (int32 GPU tensors of nseq+1 offsets), and every query attends to every key of its segment.
    Returns o [Tq, H, d], or (o, lse) with lse float32 [Tq, H] (natural log-sum-exp of the scaled
    scores) when return_lse is set or an lse tensor is passed.  num_splits: 0 lets the library
    choose, 1..16 forces that many key ranges per query tile (merged by their log-sum-exp).
    """
    return _kvcache("ts_attn_fwd_kvcache", q, k, v, cu_seqlens_q, cu_seqlens_k, max_seqlen_q,
                    max_seqlen_k, scale, out, lse, return_lse, num_splits)


def ts_attn_fwd_kvcache_noalloc(q, k, v, cu_seqlens_q, cu_seqlens_k, max_seqlen_q, max_seqlen_k,
                                scale=None, out=None, lse=None, return_lse=False, num_splits=0):
    """ts_attn_fwd_kvcache without any device allocation inside the library: its scratch is a
    static 32 MiB array per device, shared by every call on that device (calls that overlap on
    one device race).  Pass `out` (and `lse`) to allocate nothing on the torch side either."""
    return _kvcache("ts_attn_fwd_kvcache_noalloc", q, k, v, cu_seqlens_q, cu_seqlens_k,
                    max_seqlen_q, max_seqlen_k, scale, out, lse, return_lse, num_splits)


def _kvcache(entry, q, k, v, cu_seqlens_q, cu_seqlens_k, max_seqlen_q, max_seqlen_k, scale, out,
             lse, return_lse, num_splits):
    for name, t in (("q", q), ("k", k), ("v", v)):
        _check_tensor(name, t, 3)
    if (k.shape != v.shape or k.shape[1:] != q.shape[1:] or k.device != q.device
            or v.device != q.device):
        raise ValueError("k and v must be [Tk, H, d] with q's H, d and device")
    _check_offsets("cu_seqlens_q", cu_seqlens_q, q.device)
    _check_offsets("cu_seqlens_k", cu_seqlens_k, q.device)
    if cu_seqlens_q.numel() != cu_seqlens_k.numel():
        raise ValueError("cu_seqlens_q and cu_seqlens_k must have the same length")
    Tq, H, d = q.shape
    Tk = k.shape[0]
    if out is None:
        out = torch.empty_like(q)
    else:
        _check_tensor("out", out, 3)
        if out.shape != q.shape or out.device != q.device:
            raise ValueError("out must match q")
    if lse is None and return_lse:
        lse = torch.empty((Tq, H), dtype=torch.float32, device=q.device)
    if lse is not None:
        if (not isinstance(lse, torch.Tensor) or lse.dtype != torch.float32 or lse.shape != (Tq, H)
                or lse.device != q.device or not lse.is_contiguous()):
            raise ValueError("lse must be a contiguous float32 [Tq, H] tensor on q's device")
    s = default_scale(d) if scale is None else float(scale)
    lib = _lib.load()
    with torch.cuda.device(q.device):
        stream = torch.cuda.current_stream(q.device).cuda_stream
        rc = getattr(lib, entry)(_ptr(q), _ptr(k), _ptr(v), _ptr(out),
                                 _ptr(lse) if lse is not None else ctypes.c_void_p(None),
                                 _ptr(cu_seqlens_q), _ptr(cu_seqlens_k),
                                 _lib.i32("nseq", cu_seqlens_q.numel() - 1),
                                 _lib.i32("max_seqlen_q", max_seqlen_q),
                                 _lib.i32("max_seqlen_k", max_seqlen_k), _lib.i32("Tq", Tq),
                                 _lib.i32("Tk", Tk), _lib.i32("H", H), _lib.i32("d", d), s,
                                 _lib.i32("num_splits", num_splits), ctypes.c_void_p(stream))
    _lib.check(rc)
    return (out, lse) if lse is not None else out
