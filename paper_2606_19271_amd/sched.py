"""ctypes binding of libts_sched.so (include/ts_sched.h): the closed-loop session scheduler of the
paper (Sec. 5, Alg. 1, App. A).  Argument marshalling only; every decision is taken in the C++
library, and a missing library raises instead of falling back to anything else."""
import ctypes
import os

import numpy as np

from .build import SCHED_LIB

MAX_K = 64
MAX_LEVELS = 16
ARRIVE, DEPART, ACTIVATE, IDLE = 0, 1, 2, 3
STATUS_NAMES = ["TS_SCHED_OK", "TS_SCHED_ERR_ARG", "TS_SCHED_ERR_SESSION", "TS_SCHED_ERR_NOMEM"]


class _Params(ctypes.Structure):
    _fields_ = [("K", ctypes.c_int32), ("m_min", ctypes.c_int32), ("m_max", ctypes.c_int32),
                ("m_init", ctypes.c_int32), ("chunk_latency", ctypes.c_double * (MAX_K + 1)),
                ("eta", ctypes.c_double), ("mig_alpha_ms", ctypes.c_double),
                ("mig_beta_ms_per_byte", ctypes.c_double), ("delta", ctypes.c_double),
                ("window", ctypes.c_int32), ("levels", ctypes.c_int32),
                ("level_bound", ctypes.c_double * MAX_LEVELS),
                ("level_lambda", ctypes.c_double * MAX_LEVELS),
                ("level_rho", ctypes.c_double * MAX_LEVELS)]


class _Decision(ctypes.Structure):
    _fields_ = [("m", ctypes.c_int32), ("m_target", ctypes.c_int32), ("placed", ctypes.c_int32),
                ("migrations", ctypes.c_int32), ("pending", ctypes.c_int32),
                ("n_req", ctypes.c_int32), ("level", ctypes.c_int32),
                ("bottleneck_ms", ctypes.c_double), ("rho_max", ctypes.c_double),
                ("rho_hat", ctypes.c_double), ("lambda_", ctypes.c_double),
                ("volatility", ctypes.c_double)]


DECISION_KEYS = ["m", "m_target", "placed", "migrations", "pending", "n_req", "level",
                 "bottleneck_ms", "rho_max", "rho_hat", "lambda", "volatility"]


class SchedError(RuntimeError):
    def __init__(self, status):
        name = STATUS_NAMES[status] if 0 <= status < len(STATUS_NAMES) else str(status)
        super().__init__(name)
        self.status = status


_lib = None


def load_sched():
    """The loaded scheduler library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(SCHED_LIB):
        raise ImportError("libts_sched.so is not built (%s); run __graft_entry__.build()" % SCHED_LIB)
    lib = ctypes.CDLL(SCHED_LIB)
    p, i32 = ctypes.c_void_p, ctypes.c_int32
    lib.ts_sched_create.argtypes = [ctypes.POINTER(_Params), ctypes.POINTER(p)]
    lib.ts_sched_create.restype = ctypes.c_int
    lib.ts_sched_destroy.argtypes = [p]
    lib.ts_sched_destroy.restype = None
    lib.ts_sched_step.argtypes = [p, i32, p, p, p, ctypes.POINTER(_Decision)]
    lib.ts_sched_step.restype = ctypes.c_int
    lib.ts_sched_placement.argtypes = [p, p, p, i32, ctypes.POINTER(i32)]
    lib.ts_sched_placement.restype = ctypes.c_int
    lib.ts_sched_gpus.argtypes = [p, p, p, i32, ctypes.POINTER(i32)]
    lib.ts_sched_gpus.restype = ctypes.c_int
    lib.ts_sched_abi_version.argtypes = []
    lib.ts_sched_abi_version.restype = ctypes.c_int
    _lib = lib
    return lib


def _check(status):
    if status != 0:
        raise SchedError(status)


def _i32(name, x):
    """x for an int32 field or argument; ctypes would silently wrap a larger value."""
    x = int(x)
    if not -(1 << 31) <= x < (1 << 31):
        raise ValueError("%s = %d does not fit int32" % (name, x))
    return x


class Scheduler:
    """One scheduler instance (ts_sched_create / ts_sched_destroy).

    chunk_latency[n] is the per-chunk latency in ms of a GPU hosting n = 0..K sessions; the level
    table (level_bound: L-1 increasing volatility bounds, level_lambda and level_rho: L values)
    maps the volatility sigma(t) to (lambda, rho_hat).  kappa = alpha + beta * state bytes."""

    def __init__(self, K, m_min, m_max, m_init, chunk_latency, eta, alpha=0.0, beta=0.0,
                 delta=0.1, window=8, level_bound=(), level_lambda=(0.2,), level_rho=(0.7,)):
        lib = load_sched()
        if len(chunk_latency) != K + 1 or not 1 <= K <= MAX_K:
            raise ValueError("chunk_latency needs K + 1 entries, 1 <= K <= %d" % MAX_K)
        L = len(level_rho)
        if not 1 <= L <= MAX_LEVELS or len(level_lambda) != L or len(level_bound) != L - 1:
            raise ValueError("level table: L rho and lambda values and L - 1 bounds, L <= %d"
                             % MAX_LEVELS)
        prm = _Params()
        prm.K, prm.m_min = _i32("K", K), _i32("m_min", m_min)
        prm.m_max, prm.m_init = _i32("m_max", m_max), _i32("m_init", m_init)
        for n, x in enumerate(chunk_latency):
            prm.chunk_latency[n] = float(x)
        prm.eta, prm.mig_alpha_ms, prm.mig_beta_ms_per_byte = float(eta), float(alpha), float(beta)
        prm.delta, prm.window, prm.levels = float(delta), _i32("window", window), L
        for i in range(L):
            prm.level_lambda[i], prm.level_rho[i] = float(level_lambda[i]), float(level_rho[i])
        for i in range(L - 1):
            prm.level_bound[i] = float(level_bound[i])
        h = ctypes.c_void_p()
        _check(lib.ts_sched_create(ctypes.byref(prm), ctypes.byref(h)))
        self._lib, self._h, self.K = lib, h, K
        self._dec = _Decision()

    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            self._lib.ts_sched_destroy(self._h)
            self._h = None

    def __del__(self):
        self.close()

    @staticmethod
    def pack(changes):
        """(kinds int32, ids int64, bytes int64) arrays of a list of (kind, id, bytes) tuples."""
        a = np.asarray(changes, dtype=np.int64).reshape(-1, 3)
        return (np.ascontiguousarray(a[:, 0], dtype=np.int32), np.ascontiguousarray(a[:, 1]),
                np.ascontiguousarray(a[:, 2]))

    def step_packed(self, kinds, ids, nbytes):
        """One decision epoch from packed arrays (contiguous int32 kinds, int64 ids and int64
        state bytes, one entry per change, as pack() makes them); returns the raw
        ts_sched_decision, which the next call overwrites."""
        n = len(kinds)
        for name, a, dt in (("kinds", kinds, np.int32), ("ids", ids, np.int64),
                            ("nbytes", nbytes, np.int64)):
            if (not isinstance(a, np.ndarray) or a.dtype != dt or a.ndim != 1 or len(a) != n
                    or not a.flags["C_CONTIGUOUS"]):
                raise ValueError("%s must be a contiguous 1-d %s array of %d entries"
                                 % (name, np.dtype(dt).name, n))
        _check(self._lib.ts_sched_step(self._h, n, kinds.ctypes.data if n else None,
                                       ids.ctypes.data if n else None,
                                       nbytes.ctypes.data if n else None, ctypes.byref(self._dec)))
        return self._dec

    def step(self, changes):
        """One decision epoch (ts_sched_step): the session changes, then Alg. 1; a dict of the
        decision."""
        d = self.step_packed(*self.pack(changes))
        return {"m": d.m, "m_target": d.m_target, "placed": d.placed, "migrations": d.migrations,
                "pending": d.pending, "n_req": d.n_req, "level": d.level,
                "bottleneck_ms": d.bottleneck_ms, "rho_max": d.rho_max, "rho_hat": d.rho_hat,
                "lambda": d.lambda_, "volatility": d.volatility}

    def placement(self):
        """[(session id, GPU id or -1)] in increasing session id."""
        cnt = ctypes.c_int32()
        _check(self._lib.ts_sched_placement(self._h, None, None, 0, ctypes.byref(cnt)))
        ids = np.zeros(max(cnt.value, 1), np.int64)
        gpus = np.zeros(max(cnt.value, 1), np.int32)
        _check(self._lib.ts_sched_placement(self._h, ids.ctypes.data, gpus.ctypes.data, cnt.value,
                                            ctypes.byref(cnt)))
        return [(int(i), int(g)) for i, g in zip(ids[:cnt.value], gpus[:cnt.value])]

    def gpu_loads(self):
        """[(GPU id, sessions on it)] in increasing GPU id."""
        cnt = ctypes.c_int32()
        _check(self._lib.ts_sched_gpus(self._h, None, None, 0, ctypes.byref(cnt)))
        g = np.zeros(max(cnt.value, 1), np.int32)
        n = np.zeros(max(cnt.value, 1), np.int32)
        _check(self._lib.ts_sched_gpus(self._h, g.ctypes.data, n.ctypes.data, cnt.value,
                                       ctypes.byref(cnt)))
        return [(int(a), int(b)) for a, b in zip(g[:cnt.value], n[:cnt.value])]
