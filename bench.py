"""Benchmark of the fused segment-local attention on one MI355X.

One step = one call of the fused attention over a whole workload (by default the 32760-token,
40-head, d=128 latent of a large video DiT: 21 frames x 30 x 52), inputs already resident in HBM.
Prints one JSON line:
  value         attention TFLOP/s = sum_s 4 L_s^2 d H / (wall time per step)
  roofline      the kernel's algorithmic flops / its average launch time (HIP events on the
                launch stream) against the dense bf16 MFMA peak of MI355X; traffic = HBM bytes per
                launch from a committed rocprofv3 FETCH_SIZE/WRITE_SIZE measurement of the same
                kernel source (null when the kernel source changed since)
  cpu_baseline  the fp64 oracle timed on this host's cores on a bounded row sample of the same
                workload, in the same unit; the sampled rows also serve as a parity check
  config.gemm_bf16_reference  context: torch.matmul's bf16 rate on a 16384^3 product, same device
                and run (the sustainable MFMA rate at this device's power cap), and value over it
  config.sdpa_flash_reference  context, dense workloads: torch's flash scaled_dot_product_attention
                on the same inputs, same device and run, and value over it
Other workloads (--workload): the dense and packed self-attention cases of workloads.WORKLOADS,
and the chunk-vs-cache cases of workloads.KV_WORKLOADS (ts_attn_fwd_kvcache with the library's
automatic key splits: flops = sum_s 4 Lq_s Lk_s d H; the events bracket the whole call, i.e. the
planning, attention and, when split, merge kernels).
--workload sched_scale times the closed-loop session scheduler (host code, libts_sched.so): the
decision time of every epoch of a T5-shaped trace on clusters of 4 to 256 GPUs, and of a scale-out
that rebalances half a cluster's sessions (value = the worst decision at 256 GPUs, in ms).
--workload offload_kv times the session-state copy path instead: suspending the two largest
sessions of the kv_chunk batch (their K and V rows, 1.25 GB) to pinned host memory with
ts_state_copy (value = GB/s device -> host; the resume rate host -> device is reported beside it),
against the host link's 64 GB/s per direction (PCIe 5.0 x16).
Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--cpu-seconds S]
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6  # 256 CU x 4096 dense bf16 flop/clk x 2.4 GHz
KERNEL_SOURCE = os.path.join(ROOT, "paper_2606_19271_amd", "csrc", "attn_kernels.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
METRIC = "attention TFLOPS (4·L²·d·H) + % bf16 MFMA peak at L=32760,H=40,d=128"


def kernel_sha():
    with open(KERNEL_SOURCE, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def traffic_bytes(workload):
    """HBM bytes per launch measured by rocprofv3 for this exact kernel source, else None."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    e = t.get(workload)
    if not e or e.get("kernel_sha") != kernel_sha():
        return None
    return e.get("bytes_per_launch")


def cpu_baseline(w, q, k, v, o_gpu, seconds):
    """Times the oracle on batches of sampled rows until `seconds` of CPU time have elapsed."""
    import numpy as np

    import workloads as W
    from oracle import ts_ref

    ts_ref.load()
    kv = isinstance(w, W.KvWorkload)
    if kv:
        row_t, row_h = W.sample_kv_rows(w, n_random=4096, seed=999)
    else:
        row_t, row_h = W.sample_rows(w, n_random=4096, seed=999)
    # each (token, head) row once (a small call's sample would otherwise repeat rows)
    _, first = np.unique(row_t * w.H + row_h, return_index=True)
    row_t, row_h = row_t[first], row_h[first]
    perm = np.random.default_rng(7).permutation(row_t.size)
    row_t, row_h = row_t[perm], row_h[perm]
    qb, kb, vb = W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v)
    cu = w.cu_q if kv else w.cu_seqlens
    seg_len = np.diff(w.cu_k) if kv else np.diff(cu)  # keys each row attends to
    seg_of = np.searchsorted(cu, row_t, side="right") - 1
    done, flops, t_total, batch = 0, 0.0, 0.0, 64
    refs = []
    while t_total < seconds and done < row_t.size:
        sl = slice(done, min(done + batch, row_t.size))
        t0 = time.perf_counter()
        if kv:
            refs.append(ts_ref.attn_kv_rows(qb, kb, vb, w.cu_q, w.cu_k, w.scale, row_t[sl],
                                            row_h[sl])[0])
        else:
            refs.append(ts_ref.attn_rows(qb, kb, vb, cu, w.scale, row_t[sl], row_h[sl]))
        t_total += time.perf_counter() - t0
        flops += float(np.sum(4.0 * seg_len[seg_of[sl]] * w.d))
        done = sl.stop
        batch = min(batch * 2, 1024)
    ref = np.concatenate(refs)
    got = o_gpu[row_t[:done], row_h[:done]].astype(np.float64)
    err = np.abs(got - ref)
    return {
        "value": flops / t_total / 1e12,
        "unit": "TFLOP/s",
        "cores": ts_ref.num_threads(),
        "kind": "oracle",
        "sample": "%d (token, head) rows of %s (%.3g fp64 GFLOP of the %.3g GFLOP call), %.1f s"
                  % (done, w.name, flops / 1e9, w.flops / 1e9, t_total),
    }, {"rows": int(done), "max_abs": float(err.max()), "mean_abs": float(err.mean())}


def input_rounding(w, o_gpu):
    """Reported, not gated: the error of the GPU output (computed from the inputs rounded once to
    bf16) against the fp64 oracle on those bf16 inputs -- the kernel's own error -- and against
    the oracle on the unrounded fp32 draws, which adds the effect of rounding the inputs."""
    import numpy as np
    import torch

    import workloads as W
    from oracle import ts_ref

    out = {}
    for name, (q, k, v) in (("oracle_on_bf16_inputs", W.make_inputs(w)),
                            ("oracle_on_fp32_inputs", W.make_inputs_f32(w))):
        if q.dtype == torch.bfloat16:
            ref = ts_ref.attn_full(W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v), w.cu_seqlens,
                                   w.scale)
        else:
            ref = ts_ref.attn_full(*(x.double().numpy() for x in (q, k, v)), w.cu_seqlens, w.scale)
        err = np.abs(o_gpu.astype(np.float64).reshape(ref.shape) - ref)
        out[name] = {"max_abs": float(err.max()), "mean_abs": float(err.mean())}
    return out


def gemm_reference(torch, dev, n=16384, reps=4):
    """Context only: the bf16 rate of a plain n^3 matrix product by torch.matmul (hipBLASLt)
    on the same device and run, timed after the attention.  MI355X runs these MFMA-bound loads
    at a power-capped clock, so this rate, not the nominal peak, is what the device sustains."""
    a = torch.randn(n, n, device=dev, dtype=torch.bfloat16)
    b = torch.randn(n, n, device=dev, dtype=torch.bfloat16)
    c = a @ b
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        c = a @ b
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del a, b, c
    return {"n": n, "ms": ms, "tflops": 2.0 * n ** 3 / (ms * 1e-3) / 1e12}


def sdpa_reference(torch, qd, kd, vd, w, reps=5):
    """Context only: torch's scaled_dot_product_attention on the same dense workload, same device
    and run, restricted to its flash backend (so it never drops to the unfused math path); its
    [B, H, L, d] operands are contiguous copies of the [T, H, d] inputs.  Returns the backend's
    time and rate, or why it could not run."""
    from torch.nn.attention import SDPBackend, sdpa_kernel
    try:
        q, k, v = (x.view(1, w.T, w.H, w.d).transpose(1, 2).contiguous() for x in (qd, kd, vd))
        with sdpa_kernel(SDPBackend.FLASH_ATTENTION):
            o = torch.nn.functional.scaled_dot_product_attention(q, k, v, scale=w.scale)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                o = torch.nn.functional.scaled_dot_product_attention(q, k, v, scale=w.scale)
            e1.record()
            torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        del q, k, v, o
        torch.cuda.empty_cache()
        return {"backend": "flash", "ms": ms, "tflops": w.flops / (ms * 1e-3) / 1e12}
    except Exception as e:  # noqa: BLE001 -- a missing backend is reported, not fatal
        torch.cuda.empty_cache()
        return {"unavailable": str(e).splitlines()[0][:200] if str(e) else type(e).__name__}


PCIE5_X16_GBS = 64.0  # one direction, 32 GT/s x 16 lanes


def bench_offload(args, torch, np, ts, W):
    """Suspend / resume of session state: the K and V rows of two sessions of kv_chunk."""
    w = W.KV_WORKLOADS["kv_chunk"]
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev).manual_seed(w.seed)  # state bytes: any seeded pattern
    row = w.H * w.d * 2
    kd = torch.randint(-32768, 32767, (w.Tk * w.H * w.d,), generator=g, dtype=torch.int16, device=dev)
    vd = torch.randint(-32768, 32767, (w.Tk * w.H * w.d,), generator=g, dtype=torch.int16, device=dev)
    sessions = [4, 3]
    rk, end_k = ts.pack_ranges(w.cu_k, sessions, row)
    rv, end_v = ts.pack_ranges(w.cu_k, sessions, row, dst_start=end_k)
    host = torch.empty(end_v, dtype=torch.uint8, pin_memory=True)
    kb, vb = kd.view(torch.uint8), vd.view(torch.uint8)
    k_back, v_back = torch.empty_like(kb), torch.empty_like(vb)
    back_k = [(d, s, n) for s, d, n in rk]
    back_v = [(d, s, n) for s, d, n in rv]

    def offload():
        ts.ts_state_copy(kb, host, rk)
        ts.ts_state_copy(vb, host, rv)

    def resume():
        ts.ts_state_copy(host, k_back, back_k)
        ts.ts_state_copy(host, v_back, back_v)

    def timed(fn, steps):
        stream = torch.cuda.current_stream(dev)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        e0.record(stream)
        for _ in range(steps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) / steps, e0.elapsed_time(e1) * 1e-3 / steps

    for _ in range(args.warmup):
        offload()
        resume()
    wall_off, ev_off = timed(offload, args.steps)
    wall_res, ev_res = timed(resume, args.steps)
    nbytes = end_v
    ok = bool(torch.equal(k_back[rk[0][0]:rk[0][0] + rk[0][2]], kb[rk[0][0]:rk[0][0] + rk[0][2]]))

    # context: the driver's copy engine on the same contiguous bytes (hipMemcpyAsync)
    def sdma():
        for (s0, d0, n), src in [(r, kb) for r in rk] + [(r, vb) for r in rv]:
            host[d0:d0 + n].copy_(src[s0:s0 + n], non_blocking=True)
    sdma()
    wall_sdma, _ = timed(sdma, max(1, args.steps // 2))

    result = {
        "metric": "session-state offload GB/s (K and V rows of 2 sessions, device -> pinned host)",
        "value": nbytes / wall_off / 1e9, "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": wall_off * 1e3, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "u8", "data": "synthetic",
        "config": {"workload": "offload_kv", "sessions": sessions,
                   "keys": [w.k_seqlens[s] for s in sessions], "H": w.H, "d": w.d,
                   "bytes_per_step": nbytes, "resume_GBps": nbytes / wall_res / 1e9,
                   "hipMemcpyAsync_offload_GBps": nbytes / wall_sdma / 1e9,
                   "round_trip_exact": ok},
        "roofline": {"bound": "host-link", "achieved": nbytes / ev_off / 1e9,
                     "peak": PCIE5_X16_GBS, "unit": "GB/s",
                     "frac": nbytes / ev_off / 1e9 / PCIE5_X16_GBS, "traffic": None},
    }
    if not args.no_cpu_baseline:
        from oracle import state_copy as SC
        n_sample = 256 << 20
        src = np.random.default_rng(1).integers(0, 256, n_sample, dtype=np.uint8)
        dst = np.zeros(n_sample, np.uint8)
        t0, done = time.perf_counter(), 0
        while time.perf_counter() - t0 < min(args.cpu_seconds, 5.0):
            SC.copy_ranges(src, dst, [(0, 0, n_sample)])
            done += n_sample
        dt = time.perf_counter() - t0
        result["cpu_baseline"] = {"value": done / dt / 1e9, "unit": "GB/s", "cores": 1,
                                  "kind": "oracle",
                                  "sample": "numpy range copy of 256 MiB host -> host, %.1f s" % dt}
    print(json.dumps(result), flush=True)


def bench_sched(args):
    """Decision time of the closed-loop scheduler (host code) at growing cluster sizes."""
    import numpy as np

    import workloads as W
    from paper_2606_19271_amd.sched import Scheduler
    from paper_2606_19271_amd.sim import replay
    import json as _json

    golden = _json.load(open(os.path.join(ROOT, "tests", "golden", "app_a_volatility_levels.json")))
    vols = [r["volatility"] for r in golden["levels"]]
    levels = dict(level_bound=[(a + b) / 2.0 for a, b in zip(vols[:-1], vols[1:])],
                  level_lambda=[r["lambda"] for r in golden["levels"]],
                  level_rho=[r["rho"] for r in golden["levels"]])
    mig = W.SCHED_MIGRATION

    def make(M, m_min=1, m_init=None, **kw):
        prm = dict(levels)
        prm.update(kw)
        return Scheduler(W.SCHED_K, m_min, M, M // 2 if m_init is None else m_init,
                         W.SCHED_LATENCY_MS, mig["eta"], mig["alpha"], mig["beta"], 0.1,
                         W.SCHED_WINDOW, **prm)

    per_m = {}
    for M in W.SCHED_CLUSTERS:
        trace = W.sched_trace(M)
        runs = []
        for _ in range(max(1, args.steps)):
            summary, _ = replay(make(M), trace, latency_slo_ms=670.0,
                                chunk_latency=W.SCHED_LATENCY_MS)
            runs.append(summary)
        best = min(runs, key=lambda r: r["decision_ms_max"])
        # the heaviest single decision: M/2 full GPUs, then a scale-out to M that rebalances half
        # of the sessions onto the new GPUs
        full = [(W.EV_ARRIVE, i, W.SCHED_STATE_BYTES[0]) for i in range(W.SCHED_K * (M // 2))]
        s = make(M, m_min=M // 2, m_init=M // 2, level_bound=[], level_lambda=[0.2],
                 level_rho=[0.5])
        kinds, ids, nb = Scheduler.pack(full)
        t0 = time.perf_counter_ns()
        d = s.step_packed(kinds, ids, nb)
        burst_ms = (time.perf_counter_ns() - t0) * 1e-6
        best.update({"scale_out_epoch_ms": burst_ms, "scale_out_migrations": d.migrations,
                     "scale_out_sessions": len(full), "scale_out_m": d.m})
        per_m[M] = best
    top = per_m[max(W.SCHED_CLUSTERS)]
    worst = max(top["decision_ms_max"], top["scale_out_epoch_ms"])
    result = {
        "metric": "scheduler decision time per epoch at 256 GPUs (max over a T5-shaped trace and "
                  "a half-cluster scale-out), ms",
        "value": worst, "unit": "ms", "n_gpus": 1, "steps": args.steps, "warmup": 0,
        "ms_per_step": top["decision_ms_mean"], "higher_is_better": False, "scaling": "weak",
        "vs_baseline": None, "dtype": "f64", "data": "synthetic",
        "config": {"workload": "sched_scale", "K": W.SCHED_K,
                   "latency_ms": "250 + 50 n", "migration": mig, "epoch_s": 5,
                   "paper_claim_ms": {"<=64 GPUs": 15, "256 GPUs": 100},
                   "per_cluster": {str(M): per_m[M] for M in W.SCHED_CLUSTERS}},
        "roofline": None,
    }
    if not args.no_cpu_baseline:
        from oracle import sched_ref as SR
        M = 16
        trace = W.sched_trace(M)
        ref = SR.SchedRef(W.SCHED_K, 1, M, M // 2, W.SCHED_LATENCY_MS, mig["eta"], mig["alpha"],
                          mig["beta"], 0.1, W.SCHED_WINDOW, levels["level_bound"],
                          levels["level_lambda"], levels["level_rho"])
        t0, worst_ref, done = time.perf_counter(), 0.0, 0
        for ch in trace:
            t1 = time.perf_counter()
            ref.step(ch)
            worst_ref = max(worst_ref, (time.perf_counter() - t1) * 1e3)
            done += 1
            if time.perf_counter() - t0 > min(args.cpu_seconds, 20.0):
                break
        result["cpu_baseline"] = {"value": worst_ref, "unit": "ms", "cores": 1, "kind": "oracle",
                                  "sample": "oracle, max decision time over the first %d epochs "
                                            "of the 16-GPU trace (the 256-GPU case is out of its "
                                            "reach)" % done}
    print(json.dumps(result), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="dit_large")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-gemm-reference", action="store_true",
                    help="skip the context timing of a plain bf16 matrix product")
    ap.add_argument("--no-sdpa-reference", action="store_true",
                    help="skip the context timing of torch's flash attention (dense workloads)")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="instead of attention, time a plain device copy of this many bytes "
                         "(calibrates rocprofv3 FETCH_SIZE/WRITE_SIZE against known traffic)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the attention of a packed batch runs on the GPU "
              "that holds its sessions, with no exchange between GPUs; run with --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    if args.workload == "sched_scale":
        bench_sched(args)
        return

    import numpy as np
    import torch

    import paper_2606_19271_amd as ts
    import workloads as W

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.copy_bytes:
        src = torch.ones(args.copy_bytes // 2, dtype=torch.bfloat16, device=dev)
        dst = torch.empty_like(src)
        for _ in range(args.warmup):
            dst.copy_(src)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        dt = (time.perf_counter() - t0) / args.steps
        print(json.dumps({"copy_bytes": src.numel() * 2, "ms": dt * 1e3,
                          "GB/s_read_plus_write": 2 * src.numel() * 2 / dt / 1e9}), flush=True)
        return

    kv = args.workload in W.KV_WORKLOADS
    if args.workload == "offload_kv":
        bench_offload(args, torch, np, ts, W)
        return
    w = W.KV_WORKLOADS[args.workload] if kv else W.WORKLOADS[args.workload]
    q, k, v = W.make_kv_inputs(w) if kv else W.make_inputs(w)
    qd, kd, vd = q.to(dev), k.to(dev), v.to(dev)
    if kv:
        cuq, cuk = torch.tensor(w.cu_q, device=dev), torch.tensor(w.cu_k, device=dev)
    else:
        cu = torch.tensor(w.cu_seqlens, device=dev)
    dense = not kv and len(w.seqlens) == 1
    out = torch.empty_like(qd)

    def step():
        if kv:
            ts.ts_attn_fwd_kvcache(qd, kd, vd, cuq, cuk, w.max_q, w.max_k, out=out)
        elif dense:
            ts.ts_attn_fwd(qd.view(1, w.T, w.H, w.d), kd.view(1, w.T, w.H, w.d),
                           vd.view(1, w.T, w.H, w.d), out=out.view(1, w.T, w.H, w.d))
        else:
            ts.ts_attn_fwd_varlen(qd, kd, vd, cu, w.max_seqlen, out=out)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream(dev)
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        starts[i].record(stream)
        step()
        ends[i].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    launch_ms = [s.elapsed_time(e) for s, e in zip(starts, ends)]
    ms_per_step = wall / args.steps * 1e3
    value = w.flops / (ms_per_step * 1e-3) / 1e12
    kernel_ms = float(np.mean(launch_ms))
    achieved = w.flops / (kernel_ms * 1e-3) / 1e12
    traffic = traffic_bytes(w.name)
    gemm = None if args.no_gemm_reference else gemm_reference(torch, dev)
    sdpa = None if args.no_sdpa_reference or not dense else sdpa_reference(torch, qd, kd, vd, w)

    result = {
        "metric": METRIC,
        "value": value,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name,
                   **({"query_segments": list(w.q_seqlens), "key_segments": list(w.k_seqlens),
                       "Tq": w.Tq, "Tk": w.Tk} if kv else {"segments": list(w.seqlens), "T": w.T}),
                   "H": w.H, "d": w.d,
                   "causal": False, "flops_per_call": w.flops, "hbm_bytes_per_call": w.hbm_bytes,
                   "kernel_ms_mean": kernel_ms, "kernel_ms_min": float(np.min(launch_ms)),
                   "kernel_ms_max": float(np.max(launch_ms)),
                   "pct_bf16_peak": 100.0 * achieved / PEAK_BF16_TFLOPS,
                   # HBM bytes per launch from the rocprofv3 FETCH_SIZE / WRITE_SIZE passes of this
                   # kernel source (null when they were taken on another source), over the launch
                   "hbm_GBps_rocprof": None if traffic is None else traffic / (kernel_ms * 1e-3) / 1e9,
                   **({"gemm_bf16_reference": gemm,
                       "value_over_gemm": value / gemm["tflops"]} if gemm else {}),
                   **({"sdpa_flash_reference": sdpa,
                       "value_over_sdpa": value / sdpa["tflops"] if "tflops" in sdpa else None}
                      if sdpa else {})},
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS, "traffic": traffic},
    }
    if w.name == "tiny":
        result["config"]["input_rounding"] = input_rounding(w, out.float().cpu().numpy())
    if not args.no_cpu_baseline:
        o_host = out.float().cpu().numpy()
        del qd, kd, vd
        base, parity = cpu_baseline(w, q, k, v, o_host, args.cpu_seconds)
        result["cpu_baseline"] = base
        result["parity_sample"] = parity
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
