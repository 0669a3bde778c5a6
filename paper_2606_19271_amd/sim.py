"""Event simulator around the scheduler library: replays a trace of decision epochs (each a list
of (kind, session id, state bytes) changes, as produced for the paper's evaluation traces) through
ts_sched_step and accounts what the paper evaluates the scheduler by (Sec. 7): GPU cost (GPU
time provisioned), the worst-case per-chunk latency of the served sessions against a latency
target, migrations, sessions left waiting, and the wall time of every decision."""
import time

import numpy as np

from .sched import Scheduler


def replay(scheduler: Scheduler, trace, epoch_seconds=5.0, latency_slo_ms=None,
           chunk_latency=None):
    """Runs every epoch of `trace` through `scheduler`; returns a summary dict and the per-epoch
    arrays (decision wall time in ms, budget M, bottleneck latency L in ms).

    With `chunk_latency` (the scheduler's l(0..K)), each epoch's bottleneck is also compared with
    the optimum of the min-max placement problem under the same budget, the quantity the paper
    compares its rebalancing against by exhaustive search (Sec. 7.4).  With a latency that depends
    only on a GPU's load and never falls as the load grows, that optimum is l(ceil(N / M)) for N
    placed sessions on M GPUs: every placement has a GPU with at least that many sessions, and the
    balanced placement attains it."""
    packed = [Scheduler.pack(ch) for ch in trace]
    n = len(packed)
    ms = np.zeros(n)
    m = np.zeros(n, np.int64)
    L = np.zeros(n)
    opt = np.zeros(n)
    migrations = placed = pending_epochs = 0
    for t, (kinds, ids, nbytes) in enumerate(packed):
        t0 = time.perf_counter_ns()
        d = scheduler.step_packed(kinds, ids, nbytes)
        ms[t] = (time.perf_counter_ns() - t0) * 1e-6
        m[t], L[t] = d.m, d.bottleneck_ms
        if chunk_latency is not None and d.m > 0:
            opt[t] = chunk_latency[-(-(d.n_req - d.pending) // d.m)]
        migrations += d.migrations
        placed += d.placed
        pending_epochs += d.pending > 0
    summary = {
        "epochs": n, "changes": int(sum(len(k) for k, _, _ in packed)),
        "decision_ms_mean": float(ms.mean()) if n else 0.0,
        "decision_ms_p99": float(np.percentile(ms, 99)) if n else 0.0,
        "decision_ms_max": float(ms.max()) if n else 0.0,
        "gpu_seconds": float(m.sum() * epoch_seconds), "m_mean": float(m.mean()) if n else 0.0,
        "m_max": int(m.max()) if n else 0, "latency_max_ms": float(L.max()) if n else 0.0,
        "latency_mean_ms": float(L.mean()) if n else 0.0, "migrations": int(migrations),
        "placed": int(placed), "epochs_with_waiting_sessions": int(pending_epochs),
    }
    if latency_slo_ms is not None:
        summary["latency_pass_rate"] = float(np.mean(L <= latency_slo_ms)) if n else 1.0
    if chunk_latency is not None:
        ok = opt > 0
        gap = L[ok] / opt[ok] - 1.0
        summary["gap_to_minmax_optimum_mean"] = float(gap.mean()) if gap.size else 0.0
        summary["gap_to_minmax_optimum_max"] = float(gap.max()) if gap.size else 0.0
    return summary, {"decision_ms": ms, "m": m, "bottleneck_ms": L, "optimum_ms": opt}
