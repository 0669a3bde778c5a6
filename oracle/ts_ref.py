"""ctypes front end of the fp64 C oracle (ts_ref.c).

Test infrastructure only.  Inputs are numpy arrays laid out token-major [T, H, d]: either float64,
or uint16 holding bfloat16 bit patterns (widened exactly inside the C code).  cu_seqlens is an
int32 array of nseq+1 segment offsets; segment s holds tokens [cu[s], cu[s+1]).  The attention it
computes is the plain definition written out in ts_ref.c's header.
"""
import ctypes
import os

import numpy as np

from . import build as _build

_lib = None

_ERRORS = {1: "bad argument", 2: "bad cu_seqlens (must start at 0 and be nondecreasing)",
           3: "row index out of range", 4: "out of memory"}


def load(rebuild=False):
    """Load libts_ref.so, compiling it first when it is missing or rebuild is set."""
    global _lib
    if _lib is not None and not rebuild:
        return _lib
    if rebuild or not os.path.exists(_build.LIB):
        _build.build()
    lib = ctypes.CDLL(_build.LIB)
    p = ctypes.c_void_p
    i32, i64, f64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_double
    for name in ("ts_ref_attn_rows_bf16", "ts_ref_attn_rows_f64"):
        fn = getattr(lib, name)
        fn.argtypes = [p, p, p, p, i32, i32, i32, f64, p, p, i64, p]
        fn.restype = ctypes.c_int
    lib.ts_ref_attn_weights_f64.argtypes = [p, p, p, p, i32, i32, i32, f64, i64, i32, p, p]
    lib.ts_ref_attn_weights_f64.restype = ctypes.c_int
    for name in ("ts_ref_attn_kv_rows_bf16", "ts_ref_attn_kv_rows_f64"):
        fn = getattr(lib, name)
        fn.argtypes = [p, p, p, p, p, i32, i32, i32, f64, p, p, i64, p, p]
        fn.restype = ctypes.c_int
    lib.ts_ref_num_threads.argtypes = []
    lib.ts_ref_num_threads.restype = ctypes.c_int
    _lib = lib
    return lib


def _ptr(a):
    return ctypes.c_void_p(a.ctypes.data)


def _prep(q, k, v, cu_seqlens):
    q, k, v = (np.ascontiguousarray(x) for x in (q, k, v))
    if q.ndim != 3 or k.shape != q.shape or v.shape != q.shape:
        raise ValueError("q, k, v must share one [T, H, d] shape")
    if not (q.dtype == k.dtype == v.dtype) or q.dtype not in (np.uint16, np.float64):
        raise ValueError("q, k, v must all be uint16 (bf16 bits) or all float64")
    cu = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
    if cu.ndim != 1 or cu.size < 2 or cu[-1] != q.shape[0]:
        raise ValueError("cu_seqlens must have nseq+1 >= 2 entries ending at T")
    return q, k, v, cu


def num_threads():
    return load().ts_ref_num_threads()


def attn_rows(q, k, v, cu_seqlens, scale, row_t, row_h):
    """O[row_t[r], row_h[r], :] for every r, as a float64 array [nrows, d]."""
    lib = load()
    q, k, v, cu = _prep(q, k, v, cu_seqlens)
    T, H, d = q.shape
    row_t = np.ascontiguousarray(row_t, dtype=np.int64)
    row_h = np.ascontiguousarray(row_h, dtype=np.int32)
    if row_t.shape != row_h.shape or row_t.ndim != 1:
        raise ValueError("row_t and row_h must be 1-D and of equal length")
    out = np.empty((row_t.size, d), dtype=np.float64)
    fn = lib.ts_ref_attn_rows_bf16 if q.dtype == np.uint16 else lib.ts_ref_attn_rows_f64
    rc = fn(_ptr(q), _ptr(k), _ptr(v), _ptr(cu), cu.size - 1, H, d, float(scale),
            _ptr(row_t), _ptr(row_h), row_t.size, _ptr(out))
    if rc:
        raise RuntimeError("oracle: " + _ERRORS.get(rc, str(rc)))
    return out


def attn_full(q, k, v, cu_seqlens, scale):
    """The whole output O as a float64 array [T, H, d]."""
    T, H, d = np.shape(q)
    tt, hh = np.meshgrid(np.arange(T, dtype=np.int64), np.arange(H, dtype=np.int32), indexing="ij")
    return attn_rows(q, k, v, cu_seqlens, scale, tt.ravel(), hh.ravel()).reshape(T, H, d)


def attn_weights(q, k, v, cu_seqlens, scale, t, h):
    """(weights, out): the softmax weights of row (t, h) over its segment and O[t, h, :]."""
    lib = load()
    q, k, v, cu = _prep(q, k, v, cu_seqlens)
    if q.dtype != np.float64:
        raise ValueError("attn_weights takes float64 inputs")
    T, H, d = q.shape
    s = int(np.searchsorted(cu, t, side="right") - 1)
    w = np.empty(max(int(cu[s + 1] - cu[s]), 1), dtype=np.float64)
    out = np.empty(d, dtype=np.float64)
    rc = lib.ts_ref_attn_weights_f64(_ptr(q), _ptr(k), _ptr(v), _ptr(cu), cu.size - 1, H, d,
                                     float(scale), int(t), int(h), _ptr(w), _ptr(out))
    if rc:
        raise RuntimeError("oracle: " + _ERRORS.get(rc, str(rc)))
    return w[: int(cu[s + 1] - cu[s])], out


def _prep_kv(q, k, v, cu_q, cu_k):
    q, k, v = (np.ascontiguousarray(x) for x in (q, k, v))
    if q.ndim != 3 or k.ndim != 3 or k.shape != v.shape or k.shape[1:] != q.shape[1:]:
        raise ValueError("q must be [Tq, H, d] and k, v [Tk, H, d]")
    if not (q.dtype == k.dtype == v.dtype) or q.dtype not in (np.uint16, np.float64):
        raise ValueError("q, k, v must all be uint16 (bf16 bits) or all float64")
    cq = np.ascontiguousarray(cu_q, dtype=np.int32)
    ck = np.ascontiguousarray(cu_k, dtype=np.int32)
    if cq.ndim != 1 or cq.size < 2 or cq.shape != ck.shape:
        raise ValueError("cu_q and cu_k must both have nseq+1 >= 2 entries")
    if cq[-1] != q.shape[0] or ck[-1] != k.shape[0]:
        raise ValueError("cu_q must end at Tq and cu_k at Tk")
    return q, k, v, cq, ck


def attn_kv_rows(q, k, v, cu_q, cu_k, scale, row_t, row_h):
    """Chunk queries against per-segment key ranges (ts_ref.c, ts_ref_attn_kv_rows_*).

    q is [Tq, H, d]; k, v are [Tk, H, d]; segment s has queries cu_q[s]:cu_q[s+1] and keys
    cu_k[s]:cu_k[s+1].  Returns (out [nrows, d], lse [nrows]) as float64 for the rows
    (query token row_t[r], head row_h[r]); lse is the natural log-sum-exp of the scaled scores.
    """
    lib = load()
    q, k, v, cq, ck = _prep_kv(q, k, v, cu_q, cu_k)
    H, d = q.shape[1], q.shape[2]
    row_t = np.ascontiguousarray(row_t, dtype=np.int64)
    row_h = np.ascontiguousarray(row_h, dtype=np.int32)
    if row_t.shape != row_h.shape or row_t.ndim != 1:
        raise ValueError("row_t and row_h must be 1-D and of equal length")
    out = np.empty((row_t.size, d), dtype=np.float64)
    lse = np.empty(row_t.size, dtype=np.float64)
    fn = lib.ts_ref_attn_kv_rows_bf16 if q.dtype == np.uint16 else lib.ts_ref_attn_kv_rows_f64
    rc = fn(_ptr(q), _ptr(k), _ptr(v), _ptr(cq), _ptr(ck), cq.size - 1, H, d, float(scale),
            _ptr(row_t), _ptr(row_h), row_t.size, _ptr(out), _ptr(lse))
    if rc:
        raise RuntimeError("oracle: " + _ERRORS.get(rc, str(rc)))
    return out, lse


def attn_kv_full(q, k, v, cu_q, cu_k, scale):
    """(O [Tq, H, d], lse [Tq, H]) of chunk-vs-cache attention, float64."""
    Tq, H, d = np.shape(q)
    tt, hh = np.meshgrid(np.arange(Tq, dtype=np.int64), np.arange(H, dtype=np.int32), indexing="ij")
    out, lse = attn_kv_rows(q, k, v, cu_q, cu_k, scale, tt.ravel(), hh.ravel())
    return out.reshape(Tq, H, d), lse.reshape(Tq, H)
