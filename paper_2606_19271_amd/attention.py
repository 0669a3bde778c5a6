"""Torch-facing binding of ts_attn_fwd / ts_attn_fwd_varlen: argument marshalling only.

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
        rc = lib.ts_attn_fwd(_ptr(q), _ptr(k), _ptr(v), _ptr(out), B, L, H, d, s,
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
                                    cu_seqlens.numel() - 1, int(max_seqlen), T, H, d, s,
                                    ctypes.c_void_p(stream))
    _lib.check(rc)
    return out
