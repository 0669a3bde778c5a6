"""Torch-facing binding of ts_state_copy: the session-state copies of suspend (device -> pinned
host), resume (pinned host -> device) and packed-batch compaction (device -> device).

Argument marshalling only: the copy runs in libts_attn.so's kernel on torch's current stream of
the current device.  A session's rows of a packed token-major tensor [T, H, d] are one byte range
(rows cu[s]..cu[s+1] of H * d elements), so a suspend of several sessions is one call with one
range per (session, tensor).
"""
import ctypes

import numpy as np
import torch

from . import _lib


def pack_ranges(row_offsets, sessions, row_bytes, dst_start=0):
    """Ranges (src_offset, dst_offset, nbytes) that place the rows [row_offsets[s],
    row_offsets[s+1]) of each listed session back to back from byte dst_start, in list order.
    row_offsets is a host sequence of nseq+1 row indices.  Returns (ranges, next free offset)."""
    out = []
    pos = int(dst_start)
    for s in sessions:
        first, last = int(row_offsets[s]), int(row_offsets[s + 1])
        size = (last - first) * int(row_bytes)
        out.append((first * int(row_bytes), pos, size))
        pos += size
    return out, pos


def ts_state_copy(src, dst, ranges):
    """dst.bytes[d : d + n] = src.bytes[s : s + n] for every (s, d, n) in ranges (byte offsets
    into the two contiguous tensors, multiples of 16).  src and dst are GPU tensors of the
    current device or pinned CPU tensors (torch.empty(..., pin_memory=True)); they must not
    overlap.  Asynchronous on the current stream: synchronize before reading a host dst."""
    for name, t in (("src", src), ("dst", dst)):
        if not isinstance(t, torch.Tensor) or not t.is_contiguous():
            raise ValueError("%s must be a contiguous tensor" % name)
        if not t.is_cuda and not t.is_pinned():
            raise ValueError("%s must be a GPU tensor or a pinned CPU tensor" % name)
    r = np.ascontiguousarray(np.asarray(ranges, dtype=np.int64).reshape(-1, 3))
    dev = src.device if src.is_cuda else (dst.device if dst.is_cuda else torch.device("cuda", torch.cuda.current_device()))
    lib = _lib.load()
    with torch.cuda.device(dev):
        stream = torch.cuda.current_stream(dev).cuda_stream
        rc = lib.ts_state_copy(ctypes.c_void_p(src.data_ptr()), src.numel() * src.element_size(),
                               ctypes.c_void_p(dst.data_ptr()), dst.numel() * dst.element_size(),
                               ctypes.c_void_p(r.ctypes.data), _lib.i32("nranges", r.shape[0]),
                               ctypes.c_void_p(stream))
    _lib.check(rc)
    return dst
