"""Event simulator around the scheduler library: replays a trace of decision epochs (each a list
of (kind, session id, state bytes) changes, as produced for the paper's evaluation traces) through
ts_sched_step and accounts what the paper evaluates the scheduler by (Sec. 7): GPU cost (GPU
time provisioned), the worst-case per-chunk latency of the served sessions against a latency
target, migrations, sessions left waiting, and the wall time of every decision."""
import time

import numpy as np

from .sched import Scheduler


def replay(scheduler: Scheduler, trace, epoch_seconds=5.0, latency_slo_ms=None):
    """Runs every epoch of `trace` through `scheduler`; returns a summary dict and the per-epoch
    arrays (decision wall time in ms, budget M, bottleneck latency L in ms)."""
    packed = [Scheduler.pack(ch) for ch in trace]
    n = len(packed)
    ms = np.zeros(n)
    m = np.zeros(n, np.int64)
    L = np.zeros(n)
    migrations = placed = pending_epochs = 0
    for t, (kinds, ids, nbytes) in enumerate(packed):
        t0 = time.perf_counter_ns()
        d = scheduler.step_packed(kinds, ids, nbytes)
        ms[t] = (time.perf_counter_ns() - t0) * 1e-6
        m[t], L[t] = d.m, d.bottleneck_ms
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
    return summary, {"decision_ms": ms, "m": m, "bottleneck_ms": L}
