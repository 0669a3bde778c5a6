"""MI355X (gfx950) fused segment-local attention for packed video-diffusion serving batches.

The compute lives in libts_attn.so (hand-written HIP kernels behind the C ABI of
include/ts_attn.h); the closed-loop session scheduler lives in libts_sched.so (host C++ behind
include/ts_sched.h).  This package only marshals arguments into those ABIs.
"""
from .attention import (ts_attn_fwd, ts_attn_fwd_kvcache, ts_attn_fwd_kvcache_noalloc,  # noqa: F401
                        ts_attn_fwd_varlen, default_scale)
from ._lib import TsAttnError, load, status_str  # noqa: F401
from .state import pack_ranges, ts_state_copy  # noqa: F401
from .sched import Scheduler, SchedError, load_sched  # noqa: F401


def abi_version():
    return load().ts_attn_abi_version()
