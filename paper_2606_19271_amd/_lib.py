"""ctypes loader of libts_attn.so and the raw C ABI (include/ts_attn.h)."""
import ctypes
import os

from .build import LIB

TS_OK = 0
STATUS_NAMES = ["TS_OK", "TS_ERR_NULL", "TS_ERR_SHAPE", "TS_ERR_HEAD_DIM", "TS_ERR_SCALE",
                "TS_ERR_ALIGN", "TS_ERR_ALIAS", "TS_ERR_UNSUPPORTED", "TS_ERR_HIP",
                "TS_ERR_NOMEM", "TS_ERR_SEGMENTS", "TS_ERR_MEMORY", "TS_ERR_CAPTURE",
                "TS_ERR_SCRATCH"]
globals().update({name: i for i, name in enumerate(STATUS_NAMES)})

_lib = None


class TsAttnError(RuntimeError):
    """A non-zero ts_status returned by the library."""

    def __init__(self, status, message):
        super().__init__(message)
        self.status = status


def load():
    """The loaded library; raises if it has not been built (there is no fallback path)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB):
        raise ImportError("libts_attn.so is not built (%s); run __graft_entry__.build()" % LIB)
    lib = ctypes.CDLL(LIB)
    p, i32, f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float
    lib.ts_attn_fwd.argtypes = [p, p, p, p, i32, i32, i32, i32, f32, p]
    lib.ts_attn_fwd.restype = ctypes.c_int
    lib.ts_attn_fwd_varlen.argtypes = [p, p, p, p, p, i32, i32, i32, i32, i32, f32, p]
    lib.ts_attn_fwd_varlen.restype = ctypes.c_int
    lib.ts_attn_fwd_kvcache.argtypes = [p, p, p, p, p, p, p] + [i32] * 7 + [f32, i32, p]
    lib.ts_attn_fwd_kvcache.restype = ctypes.c_int
    lib.ts_attn_fwd_kvcache_noalloc.argtypes = lib.ts_attn_fwd_kvcache.argtypes
    lib.ts_attn_fwd_kvcache_noalloc.restype = ctypes.c_int
    i64 = ctypes.c_int64
    lib.ts_state_copy.argtypes = [p, i64, p, i64, p, i32, p]
    lib.ts_state_copy.restype = ctypes.c_int
    lib.ts_attn_status_str.argtypes = [ctypes.c_int]
    lib.ts_attn_status_str.restype = ctypes.c_char_p
    lib.ts_attn_abi_version.argtypes = []
    lib.ts_attn_abi_version.restype = ctypes.c_int
    _lib = lib
    return lib


def i32(name, x):
    """x as a C int32 argument; ctypes would silently wrap a larger value, so refuse it."""
    x = int(x)
    if not -(1 << 31) <= x < (1 << 31):
        raise ValueError("%s = %d does not fit the C ABI's int32" % (name, x))
    return x


def status_str(status):
    return load().ts_attn_status_str(int(status)).decode()


def check(status):
    if status != TS_OK:
        raise TsAttnError(status, status_str(status))
