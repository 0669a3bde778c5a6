"""GPU parity of the HIP path (through the C ABI) against the fp64 oracle, on seeded inputs.

Full-tensor comparison where the oracle finishes in seconds (several query/key tiles plus ragged
tails); sampled rows at the full workload sizes, in the same launch configuration the benchmark
times; bitwise properties (dense == packed, segment independence, determinism); invariants whose
exact answer is known; and the error paths of the packed entry point.
"""
import os
import sys

import numpy as np
import pytest
import torch

import workloads as W
from metrics import assert_parity, assert_rows, errors
from oracle import ts_ref

pytestmark = pytest.mark.gpu

ts = pytest.importorskip("paper_2606_19271_amd")


def say(*a):
    print("[gpu-test]", *a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ts.load()
    return torch.device("cuda:0")


def draw(seqlens, H, d, seed, k_offset=False, scale_q=1.0):
    w = W.Workload("custom", tuple(seqlens), H, d, seed, k_offset)
    q, k, v = W.make_inputs(w)
    if scale_q != 1.0:
        q = (q.float() * scale_q).to(torch.bfloat16)
    return w, q, k, v


def run_varlen(q, k, v, seqlens, scale=None):
    cu = torch.tensor(np.concatenate([[0], np.cumsum(seqlens)]).astype(np.int32), device="cuda")
    o = ts.ts_attn_fwd_varlen(q.cuda(), k.cuda(), v.cuda(), cu, max(seqlens) if seqlens else 0,
                              scale=scale)
    torch.cuda.synchronize()
    return o.cpu()


def oracle_full(q, k, v, seqlens, scale):
    cu = np.concatenate([[0], np.cumsum(seqlens)]).astype(np.int32)
    return ts_ref.attn_full(W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v), cu, scale)


def as_f64(o):
    return o.float().numpy().astype(np.float64)


# ---------------------------------------------------------------------------------- full tensors

def test_tiny_full_dense_and_varlen():
    w = W.WORKLOADS["tiny"]
    q, k, v = W.make_inputs(w)
    say("tiny full", w.seqlens, w.H, w.d)
    ref = oracle_full(q, k, v, list(w.seqlens), w.scale)
    o_dense = ts.ts_attn_fwd(q.cuda().view(1, w.T, w.H, w.d), k.cuda().view(1, w.T, w.H, w.d),
                             v.cuda().view(1, w.T, w.H, w.d)).view(w.T, w.H, w.d)
    torch.cuda.synchronize()
    o_var = run_varlen(q, k, v, list(w.seqlens))
    e = assert_rows(as_f64(o_dense.cpu()), ref, "tiny dense", elementwise=False)
    say("tiny errors", e)
    assert torch.equal(o_dense.cpu().view(torch.int16), o_var.view(torch.int16))


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("L", [1, 2, 31, 63, 64, 65, 127, 255, 256, 257, 300, 777, 1000])
def test_ragged_lengths_full(L, d):
    w, q, k, v = draw([L], 3, d, seed=1000 + L + d)
    say("ragged", L, d)
    ref = oracle_full(q, k, v, [L], w.scale)
    o = run_varlen(q, k, v, [L])
    assert_rows(as_f64(o), ref, "L=%d d=%d" % (L, d), elementwise=False)


@pytest.mark.parametrize("d", [64, 128])
def test_dense_batch_full(d):
    B, L, H = 3, 333, 2
    w, q, k, v = draw([L] * B, H, d, seed=77 + d)
    say("dense batch", B, L, H, d)
    o = ts.ts_attn_fwd(q.cuda().view(B, L, H, d), k.cuda().view(B, L, H, d),
                       v.cuda().view(B, L, H, d))
    torch.cuda.synchronize()
    ref = oracle_full(q, k, v, [L] * B, w.scale)
    assert_rows(as_f64(o.cpu().view(B * L, H, d)), ref, "dense batch d=%d" % d,
                elementwise=False)
    o_var = run_varlen(q, k, v, [L] * B)
    assert torch.equal(o.cpu().view(B * L, H, d).view(torch.int16), o_var.view(torch.int16))


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("L", [1, 16, 17, 100, 224, 225, 256, 280, 480, 513, 544, 737])
def test_dense_ragged_lengths_full(L, d):
    """The dense call runs the ragged last query tile of every (sequence, head) after all full
    tiles when that tile leaves a wave without queries (L mod 256 in 1..224): every such order,
    and the plain one (225, 256, 480), against the oracle and bitwise against the packed call.
    A last tile of at most 32 queries (1, 16, 17, 280, 513, 544) takes the thin path, in which all
    eight waves share it."""
    B, H = 3, 2
    w, q, k, v = draw([L] * B, H, d, seed=3000 + L + d)
    say("dense ragged", B, L, H, d)
    o = ts.ts_attn_fwd(q.cuda().view(B, L, H, d), k.cuda().view(B, L, H, d),
                       v.cuda().view(B, L, H, d))
    torch.cuda.synchronize()
    o = o.cpu().view(B * L, H, d)
    assert_rows(as_f64(o), oracle_full(q, k, v, [L] * B, w.scale), "dense L=%d d=%d" % (L, d),
                elementwise=False)
    assert torch.equal(o.view(torch.int16), run_varlen(q, k, v, [L] * B).view(torch.int16))


@pytest.mark.parametrize("d", [64, 128])
def test_varlen_with_empty_and_tiny_segments_full(d):
    seqlens = [0, 5, 0, 300, 1, 0, 129, 64, 2, 513, 0]
    w, q, k, v = draw(seqlens, 2, d, seed=5 + d)
    say("varlen empty segments", seqlens, d)
    ref = oracle_full(q, k, v, seqlens, w.scale)
    o = run_varlen(q, k, v, seqlens)
    assert_rows(as_f64(o), ref, "varlen d=%d" % d, elementwise=False)


# lengths at and around the 64-key and 256-query tile edges, mixed with arbitrary ones
EDGE_LENGTHS = [0, 1, 2, 31, 32, 33, 63, 64, 65, 127, 128, 129, 255, 256, 257, 511, 512, 513]


def random_case(rng, max_len=1400):
    nseq = int(rng.integers(1, 10))
    lens = [int(rng.choice(EDGE_LENGTHS)) if rng.random() < 0.5 else int(rng.integers(1, max_len))
            for _ in range(nseq)]
    if sum(lens) == 0:
        lens[int(rng.integers(0, nseq))] = int(rng.integers(1, max_len))
    H = int(rng.choice([1, 2, 3, 5]))
    d = int(rng.choice([64, 128]))
    scale = None if rng.random() < 0.5 else float(np.float32(rng.uniform(-1.0, 1.5)))
    return lens, H, d, scale


@pytest.mark.parametrize("seed", range(10))
def test_random_packed_batches_full(seed):
    # seeded random batches: segment count, lengths, heads, head dim and scale all drawn, so that
    # tile edges, empty segments and the planner's ordering meet in combinations no listed case has
    rng = np.random.default_rng(4200 + seed)
    lens, H, d, scale = random_case(rng)
    w, q, k, v = draw(lens, H, d, seed=4300 + seed)
    sc = w.scale if scale is None else scale
    say("random packed", seed, lens, H, d, scale)
    ref = oracle_full(q, k, v, lens, sc)
    o = run_varlen(q, k, v, lens, scale=scale)
    assert_rows(as_f64(o), ref, "random packed seed=%d %r H=%d d=%d scale=%r" % (seed, lens, H, d, scale),
                elementwise=False)


def test_many_segments_beyond_sort_limit():
    rng = np.random.default_rng(9)
    seqlens = rng.integers(0, 6, size=5000).tolist()  # more segments than the plan sorts
    seqlens[1234] = 700
    w, q, k, v = draw(seqlens, 1, 128, seed=9)
    say("many segments", len(seqlens), sum(seqlens))
    ref = oracle_full(q, k, v, seqlens, w.scale)
    o = run_varlen(q, k, v, seqlens)
    assert_rows(as_f64(o), ref, "5000 segments", elementwise=False)


# Each of the special-input tests below also runs on segments whose last query tile holds at most
# 32 queries (24, 280 = 256 + 24, 536 = 512 + 24, 1044 = 4 * 256 + 20, 1560 = 6 * 256 + 24), which
# take the thin path: there each wave keeps its own running maximum over a quarter of every key
# tile, and the four waves of a query block combine their partials at the end.
@pytest.mark.parametrize("seqlens", [[200, 457], [24, 280]])
@pytest.mark.parametrize("scale", [0.0, -0.2, 0.9])
def test_other_scales_full(scale, seqlens):
    w, q, k, v = draw(seqlens, 2, 128, seed=31)
    scale = float(np.float32(scale))
    say("scale", scale)
    ref = oracle_full(q, k, v, seqlens, scale)
    o = run_varlen(q, k, v, seqlens, scale=scale)
    assert_rows(as_f64(o), ref, "scale=%g %r" % (scale, seqlens), elementwise=False)


@pytest.mark.parametrize("seqlens", [[1500, 700], [1560, 280]])
def test_peaked_scores_full(seqlens):
    # scores 8x larger than N(0,1) inputs give: softmax rows dominated by a few keys, and the
    # running max moves often (exercises the rescale path)
    w, q, k, v = draw(seqlens, 2, 128, seed=44, scale_q=8.0)
    say("peaked", seqlens)
    ref = oracle_full(q, k, v, seqlens, w.scale)
    o = run_varlen(q, k, v, seqlens)
    assert_rows(as_f64(o), ref, "peaked %r" % seqlens, elementwise=False)


@pytest.mark.parametrize("L", [1024, 1044])
def test_increasing_scores_force_rescale(L):
    # K rows grow along the sequence, so every tile raises the row max (by about 6 log2 units)
    # and every seventh or so passes the 2^40 headroom of the lazy maximum: the slow path then
    # rescales O and l in the middle of the sequence, several times
    H, d = 1, 128
    g = torch.Generator().manual_seed(3)
    q = torch.ones((L, H, d)).to(torch.bfloat16)
    ramp = torch.linspace(0.0, 6.0, L).view(L, 1, 1)
    k = (ramp + 0.01 * torch.randn((L, H, d), generator=g)).to(torch.bfloat16)
    v = torch.randn((L, H, d), generator=g).to(torch.bfloat16)
    scale = W.Workload("x", (L,), H, d, 0).scale
    say("forced rescale", L)
    ref = oracle_full(q, k, v, [L], scale)
    o = run_varlen(q, k, v, [L])
    assert_rows(as_f64(o), ref, "forced rescale L=%d" % L, elementwise=False)



@pytest.mark.parametrize("seqlens", [[640, 300], [536, 300]])
@pytest.mark.parametrize("gap", [5.0, 38.0, 45.0, 200.0, 1000.0])
def test_score_jump_mid_sequence(gap, seqlens):
    # One key in the middle of a segment (key 400, tile 6) scores `gap` log2 units above every
    # other key of every query row.  Below 40 the lazy maximum stays and the weights are up to
    # 2^gap times the earlier ones; above it the slow path must take the tile's maximum and
    # rescale O and l (without it, gap >= 167 overflows the fp32 weights).  In the thin tile of
    # the 536-query segment the key lies in the second 16-key block of its tile, so only the two
    # waves holding that block see the jump and their maxima differ from the other six waves'.
    H, d = 2, 128
    g = torch.Generator().manual_seed(57)
    T = sum(seqlens)
    q = torch.randn((T, H, d), generator=g)
    q[:, :, 0] = 4.0
    k = 0.3 * torch.randn((T, H, d), generator=g)
    k[:, :, 0] = 0.0
    v = torch.randn((T, H, d), generator=g)
    scale = W.Workload("x", tuple(seqlens), H, d, 0).scale
    c = float(np.float32(scale)) * 1.4426950408889634
    k[400, :, 0] = gap / (4.0 * c)
    q, k, v = q.to(torch.bfloat16), k.to(torch.bfloat16), v.to(torch.bfloat16)
    say("score jump", gap, seqlens)
    ref = oracle_full(q, k, v, seqlens, scale)
    o = run_varlen(q, k, v, seqlens)
    got = as_f64(o)
    assert np.all(np.isfinite(got))
    assert_rows(got, ref, "score jump %g %r" % (gap, seqlens), elementwise=False)

# ------------------------------------------------------------------------- full-size workloads

@pytest.mark.parametrize("name", ["dit_small", "dit_large", "highres", "varlen_serving",
                                  "dit_small_d64"])
def test_workload_sampled(name):
    w = W.WORKLOADS[name]
    say("workload", name, "T=%d H=%d d=%d" % (w.T, w.H, w.d))
    q, k, v = W.make_inputs(w)
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    if len(w.seqlens) == 1:
        o = ts.ts_attn_fwd(qd.view(1, w.T, w.H, w.d), kd.view(1, w.T, w.H, w.d),
                           vd.view(1, w.T, w.H, w.d)).view(w.T, w.H, w.d)
    else:
        cu = torch.tensor(w.cu_seqlens, device="cuda")
        o = ts.ts_attn_fwd_varlen(qd, kd, vd, cu, w.max_seqlen)
    torch.cuda.synchronize()
    assert torch.isfinite(o.float()).all()
    row_t, row_h = W.sample_rows(w)
    got = o[torch.from_numpy(row_t).cuda(), torch.from_numpy(row_h).long().cuda()].cpu()
    del qd, kd, vd, o
    say("oracle rows", row_t.size)
    ref = ts_ref.attn_rows(W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v), w.cu_seqlens,
                           w.scale, row_t, row_h)
    e = assert_rows(as_f64(got), ref, name)
    trivial = errors(np.zeros_like(ref), ref)
    say(name, "errors", e, "zero-output errors", trivial)
    assert e["mean_abs"] < 0.1 * trivial["mean_abs"]


# ---------------------------------------------------------------------------- bitwise properties

def test_segment_independence_bitwise():
    seqlens = [300, 1000, 77]
    w, q, k, v = draw(seqlens, 2, 128, seed=12)
    say("segment independence")
    o1 = run_varlen(q, k, v, seqlens)
    q2, k2, v2 = q.clone(), k.clone(), v.clone()
    q2[:300] = -q2[:300]
    k2[:300] = k2[:300] * 2
    v2[:300] = 0
    o2 = run_varlen(q2, k2, v2, seqlens)
    assert torch.equal(o1[300:].view(torch.int16), o2[300:].view(torch.int16))
    # packed result == each segment alone, bit for bit
    start = 0
    for L in seqlens:
        alone = run_varlen(q[start:start + L], k[start:start + L], v[start:start + L], [L])
        assert torch.equal(alone.view(torch.int16), o1[start:start + L].view(torch.int16))
        start += L


def test_deterministic_bitwise():
    w = W.WORKLOADS["varlen_serving"]
    seqlens = [s // 10 for s in w.seqlens]
    _, q, k, v = draw(seqlens, 4, 128, seed=8)
    say("determinism")
    a = run_varlen(q, k, v, seqlens)
    b = run_varlen(q, k, v, seqlens)
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


# ------------------------------------------------------------------------ exact-answer invariants

def test_identical_keys_give_mean_of_v():
    L, H, d = 700, 2, 128
    g = torch.Generator().manual_seed(21)
    q = torch.randn((L, H, d), generator=g).to(torch.bfloat16)
    k = torch.randn((1, H, d), generator=g).expand(L, H, d).contiguous().to(torch.bfloat16)
    v = torch.randn((L, H, d), generator=g).to(torch.bfloat16)
    say("identical keys")
    o = run_varlen(q, k, v, [L])
    mean_v = v.double().mean(dim=0, keepdim=True).expand(L, H, d).numpy()
    assert_rows(as_f64(o), mean_v, "identical keys", elementwise=False)


def test_dominant_key_returns_its_value_row():
    L, H, d = 513, 1, 128
    g = torch.Generator().manual_seed(22)
    k = torch.randn((L, H, d), generator=g).to(torch.bfloat16)
    v = torch.randn((L, H, d), generator=g).to(torch.bfloat16)
    jstar = 400
    q = (k[jstar:jstar + 1].float() * 4.0).expand(L, H, d).contiguous().to(torch.bfloat16)
    scale = 1.0
    say("dominant key")
    ref = oracle_full(q, k, v, [L], scale)
    gap = 30.0
    # the oracle confirms the gap premise, then the GPU must return V[j*]
    z = (q[0, 0].double() @ k[:, 0].double().T) * scale
    assert float(z[jstar] - torch.cat([z[:jstar], z[jstar + 1:]]).max()) > gap
    o = run_varlen(q, k, v, [L], scale=scale)
    target = v[jstar:jstar + 1].double().expand(L, H, d).numpy()
    assert_rows(as_f64(o), target, "dominant key", elementwise=False)
    assert_rows(as_f64(o), ref, "dominant key vs oracle", elementwise=False)


def test_constant_v_gives_constant():
    L, H, d = 900, 2, 64
    g = torch.Generator().manual_seed(23)
    q = torch.randn((L, H, d), generator=g).to(torch.bfloat16)
    k = torch.randn((L, H, d), generator=g).to(torch.bfloat16)
    v = torch.full((L, H, d), 0.71875).to(torch.bfloat16)
    say("constant V")
    o = run_varlen(q, k, v, [L])
    assert_rows(as_f64(o), np.full((L, H, d), 0.71875), "constant V", elementwise=False)


# ---------------------------------------------------------------------------------- error paths

def test_bad_cu_seqlens_is_a_noop_and_validate_mode_reports_it():
    T, H, d = 300, 1, 128
    q = torch.randn((T, H, d)).to(torch.bfloat16).cuda()
    bad = torch.tensor([0, 200, 100, 300], dtype=torch.int32, device="cuda")  # decreasing
    o = torch.full((T, H, d), 7.0, dtype=torch.bfloat16, device="cuda")
    say("bad cu_seqlens")
    ts.ts_attn_fwd_varlen(q, q, q, bad, 300, out=o)
    torch.cuda.synchronize()
    assert bool((o == 7.0).all())
    os.environ["TS_ATTN_VALIDATE"] = "1"
    try:
        with pytest.raises(ts.TsAttnError) as ei:
            ts.ts_attn_fwd_varlen(q, q, q, bad, 300, out=o)
        assert ei.value.status == 10
        # a segment longer than max_seqlen is rejected the same way
        cu = torch.tensor([0, 300], dtype=torch.int32, device="cuda")
        with pytest.raises(ts.TsAttnError):
            ts.ts_attn_fwd_varlen(q, q, q, cu, 100, out=o)
        # one segment whose end is not the tensors' row count (checked by the attention kernel
        # itself outside validation mode, below)
        short = torch.tensor([0, 200], dtype=torch.int32, device="cuda")
        with pytest.raises(ts.TsAttnError):
            ts.ts_attn_fwd_varlen(q, q, q, short, 300, out=o)
        # and a valid batch passes
        ts.ts_attn_fwd_varlen(q, q, q, cu, 300, out=o)
    finally:
        del os.environ["TS_ATTN_VALIDATE"]
    torch.cuda.synchronize()
    # outside validation mode a batch of one segment runs without the planning kernel; bad
    # offsets (not ending at the row count, or not starting at 0) or a total beyond max_seqlen
    # still leave o untouched
    for cu_l, max_len in (([0, 200], 300), ([100, 300], 300), ([0, 300], 100)):
        o = torch.full((T, H, d), 7.0, dtype=torch.bfloat16, device="cuda")
        ts.ts_attn_fwd_varlen(q, q, q, torch.tensor(cu_l, dtype=torch.int32, device="cuda"),
                              max_len, out=o)
        torch.cuda.synchronize()
        assert bool((o == 7.0).all()), (cu_l, max_len)


def wrapping_offsets(T, nseq, max_len):
    """Offsets whose int32 differences all lie in [0, max_len] and that start at 0 and end at T,
    while the offsets in between wrap far outside [0, T] (nseq * max_len >= 2^32)."""
    diffs = [max_len] * 256 + [(1 << 32) + T - 256 * max_len] + [0] * (nseq - 257)
    cu = [0]
    for x in diffs:
        cu.append(((cu[-1] + x + (1 << 31)) % (1 << 32)) - (1 << 31))
    assert cu[-1] == T and min(cu) < 0 and max(cu) > T
    return cu


def test_offsets_that_wrap_int32_are_rejected():
    # regression: the plan once checked only the (wrapping) differences of the offsets, which
    # these pass; every offset must now lie in [0, T], and the call is a device-side no-op
    T, H, d, nseq, max_len = 1024, 1, 64, 512, (1 << 24) - 512
    cu = torch.tensor(wrapping_offsets(T, nseq, max_len), dtype=torch.int32, device="cuda")
    q = torch.randn((T, H, d)).to(torch.bfloat16).cuda()
    o = torch.full((T, H, d), 7.0, dtype=torch.bfloat16, device="cuda")
    say("wrapping offsets", nseq, max_len)
    ts.ts_attn_fwd_varlen(q, q, q, cu, max_len, out=o)
    torch.cuda.synchronize()
    assert bool((o == 7.0).all())
    os.environ["TS_ATTN_VALIDATE"] = "1"
    try:
        with pytest.raises(ts.TsAttnError) as ei:
            ts.ts_attn_fwd_varlen(q, q, q, cu, max_len, out=o)
        assert ei.value.status == 10
    finally:
        del os.environ["TS_ATTN_VALIDATE"]
    torch.cuda.synchronize()


def test_sizes_beyond_int32_are_refused_by_the_binding():
    w, q, k, v = draw([64], 1, 64, seed=3)
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    cu = torch.tensor(w.cu_seqlens, device="cuda")
    with pytest.raises(ValueError):
        ts.ts_attn_fwd_varlen(qd, kd, vd, cu, (1 << 32) + 64)  # would reach the ABI as 64
    with pytest.raises(ValueError):
        ts.ts_attn_fwd_kvcache(qd, kd, vd, cu, cu, 64, (1 << 32) + 64)


def test_runs_on_a_side_stream():
    seqlens = [400, 123]
    w, q, k, v = draw(seqlens, 2, 128, seed=61)
    say("side stream")
    ref = oracle_full(q, k, v, seqlens, w.scale)
    s = torch.cuda.Stream()
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    cu = torch.tensor(w.cu_seqlens, device="cuda")
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        o = ts.ts_attn_fwd_varlen(qd, kd, vd, cu, w.max_seqlen)
    s.synchronize()
    assert_rows(as_f64(o.cpu()), ref, "side stream", elementwise=False)


def test_concurrent_calls_from_threads_on_separate_streams():
    """Four host threads, each on its own stream, call the packed attention (split and unsplit
    chunk calls included) 10 times each; every result equals the single-threaded one bitwise."""
    import threading
    seqlens = [700, 0, 333]
    w, q, k, v = draw(seqlens, 4, 128, seed=67)
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    cu = torch.tensor(w.cu_seqlens, device="cuda")
    ref_o = ts.ts_attn_fwd_varlen(qd, kd, vd, cu, w.max_seqlen)
    ref_kv, ref_lse = ts.ts_attn_fwd_kvcache(qd, kd, vd, cu, cu, w.max_seqlen, w.max_seqlen,
                                            return_lse=True, num_splits=3)
    torch.cuda.synchronize()
    say("threads")
    errors_seen = []

    def worker(n):
        try:
            st = torch.cuda.Stream()
            with torch.cuda.stream(st):
                for _ in range(10):
                    if n % 2:
                        o = ts.ts_attn_fwd_varlen(qd, kd, vd, cu, w.max_seqlen)
                        lse = None
                    else:
                        o, lse = ts.ts_attn_fwd_kvcache(qd, kd, vd, cu, cu, w.max_seqlen, w.max_seqlen,
                                                        return_lse=True, num_splits=3)
                    st.synchronize()
                    if not torch.equal(o, ref_o if n % 2 else ref_kv):
                        errors_seen.append("output of thread %d" % n)
                    if lse is not None and not torch.equal(lse, ref_lse):
                        errors_seen.append("lse of thread %d" % n)
        except Exception as e:  # reported below
            errors_seen.append(repr(e))

    threads = [threading.Thread(target=worker, args=(n,)) for n in range(4)]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads)
    assert not errors_seen, errors_seen[:3]


# ------------------------------------------------------------------------- closed-form fixtures

def test_closed_form_golden_cases():
    import json
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "closed_forms.json")
    for c in json.load(open(path))["cases"]:
        say("golden", c["name"])
        q, k, v = (torch.tensor(c[x], dtype=torch.float64).to(torch.bfloat16) for x in ("q", "k", "v"))
        d = c["d"]
        pad = 64 - d  # the kernel takes d = 64: zero channels change no score and no output
        q, k, v = (torch.nn.functional.pad(x, (0, pad)) for x in (q, k, v))
        exp = np.array([[[float(x) for x in row] for row in tok] for tok in c["expected"]])
        o = run_varlen(q, k, v, c["seqlens"], scale=c["scale"])
        got = as_f64(o)[:, :, :d]
        assert np.all(np.abs(got - exp) <= 2e-2), c["name"]
        assert np.abs(got - exp).mean() <= 2e-3, c["name"]
        assert np.all(as_f64(o)[:, :, d:] == 0.0)  # zero V channels stay zero


# --------------------------------------------------------------------------- the size limit

@pytest.mark.parametrize("d", [128, 64])
def test_segments_at_the_byte_limit_sampled(d):
    """A segment at the largest size the ABI accepts, (L + 256) * H * d * 2 < 2^31 bytes, in a
    packed batch whose second segment starts beyond 2 GiB: exercises the 32-bit in-segment
    offsets at their limit (also those of the K/V fetches that run ahead past the segment's end:
    up to three 128-key tiles at d = 64) and the 64-bit segment bases (H = 128 keeps the
    attention cheap)."""
    H = 128
    row_bytes = H * d * 2
    L = (1 << 31) // row_bytes - 256 - 1          # 65279 at d = 128, 130815 at d = 64
    seqlens = [L, 40000]
    T = sum(seqlens)
    assert (L + 256) * row_bytes < (1 << 31) <= (L + 257) * row_bytes
    assert L * row_bytes < (1 << 31) < T * row_bytes
    say("byte limit", "L=%d T=%d H=%d d=%d" % (L, T, H, d))
    q, k, v = W.make_device_inputs(T, H, d, seed=21, device=torch.device("cuda"))
    cu_np = np.array([0, L, T], dtype=np.int32)
    cu = torch.from_numpy(cu_np).cuda()
    scale = W.Workload("x", (T,), H, d, 0).scale
    o = ts.ts_attn_fwd_varlen(q, k, v, cu, L, scale=scale)
    o_dense = ts.ts_attn_fwd(q[:L].view(1, L, H, d), k[:L].view(1, L, H, d), v[:L].view(1, L, H, d),
                             scale=scale).view(L, H, d)
    torch.cuda.synchronize()
    # one past the limit is refused on the host, before any launch
    with pytest.raises(ts.TsAttnError):
        ts.ts_attn_fwd_varlen(q[:L + 1], k[:L + 1], v[:L + 1],
                              torch.tensor([0, L + 1], dtype=torch.int32, device="cuda"), L + 1)
    rng = np.random.default_rng(5)
    row_t = np.concatenate([[0, L - 1, L - 2, L - 255, L, T - 1, T - 300],
                            rng.integers(0, T, 57)]).astype(np.int64)
    row_h = np.concatenate([[0, H - 1, 77, H - 1, H - 1, H - 1, 3],
                            rng.integers(0, H, 57)]).astype(np.int32)
    tt, hh = torch.from_numpy(row_t).cuda(), torch.from_numpy(row_h).long().cuda()
    got = o[tt, hh].cpu()
    i0 = torch.from_numpy(np.nonzero(row_t < L)[0])  # rows of the first segment: dense == packed
    assert torch.equal(o_dense[tt[i0.cuda()], hh[i0.cuda()]].cpu(), got[i0])
    del o, o_dense
    hq, hk, hv = (W.bf16_bits(x.cpu()) for x in (q, k, v))
    del q, k, v
    torch.cuda.empty_cache()
    say("oracle rows", row_t.size)
    ref = ts_ref.attn_rows(hq, hk, hv, cu_np, scale, row_t, row_h)
    e = assert_rows(as_f64(got), ref, "byte limit d=%d" % d)
    trivial = errors(np.zeros_like(ref), ref)
    say("byte limit errors", e, "zero-output errors", trivial)
    assert e["mean_abs"] < 0.1 * trivial["mean_abs"]


def test_head_dim_64_long_segments_sampled():
    """d = 64 over long segments (hundreds of key tiles, the XCD remap of a large grid, the
    per-channel K offsets of the DiT workloads), sampled rows against the oracle."""
    w = W.Workload("d64_long", (20000, 7777), 6, 64, 64, k_offset=True)
    say("d64 long", w.seqlens, w.H, w.d)
    q, k, v = W.make_inputs(w)
    cu = torch.tensor(w.cu_seqlens, device="cuda")
    o = ts.ts_attn_fwd_varlen(q.cuda(), k.cuda(), v.cuda(), cu, w.max_seqlen)
    torch.cuda.synchronize()
    row_t, row_h = W.sample_rows(w)
    got = o[torch.from_numpy(row_t).cuda(), torch.from_numpy(row_h).long().cuda()].cpu()
    ref = ts_ref.attn_rows(W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v), w.cu_seqlens,
                           w.scale, row_t, row_h)
    e = assert_rows(as_f64(got), ref, "d64 long")
    say("d64 long errors", e)
    assert e["mean_abs"] < 0.1 * errors(np.zeros_like(ref), ref)["mean_abs"]


def test_q_k_v_may_be_one_tensor():
    """The ABI lets q, k and v alias one another (only o must be separate): self-similarity
    attention with q = k = v, packed and dense, against the oracle on the same array."""
    seqlens = [700, 129]
    w, q, _, _ = draw(seqlens, 2, 128, seed=91)
    say("aliased q = k = v")
    x = q.cuda()
    cu = torch.tensor(np.concatenate([[0], np.cumsum(seqlens)]).astype(np.int32), device="cuda")
    o = ts.ts_attn_fwd_varlen(x, x, x, cu, max(seqlens))
    o_dense = ts.ts_attn_fwd(x[:700].view(1, 700, 2, 128), x[:700].view(1, 700, 2, 128),
                             x[:700].view(1, 700, 2, 128)).view(700, 2, 128)
    torch.cuda.synchronize()
    ref = oracle_full(q, q, q, seqlens, w.scale)
    assert_rows(as_f64(o.cpu()), ref, "aliased", elementwise=False)
    assert torch.equal(o_dense.cpu(), o[:700].cpu())


def test_tiny_input_rounding_is_reported():
    """The tiny configuration specifies float32 q, k, v; the kernel reads them rounded once to
    bf16.  Reported, not gated beyond the usual bar on the bf16 inputs: the GPU output against
    the oracle on the bf16 inputs (the kernel's own error) and on the unrounded float32 draws
    (adding the effect of the input rounding)."""
    w = W.WORKLOADS["tiny"]
    q, k, v = W.make_inputs(w)
    o = ts.ts_attn_fwd(q.cuda().view(1, w.T, w.H, w.d), k.cuda().view(1, w.T, w.H, w.d),
                       v.cuda().view(1, w.T, w.H, w.d)).view(w.T, w.H, w.d)
    torch.cuda.synchronize()
    got = as_f64(o.cpu())
    ref_bf16 = ts_ref.attn_full(W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v), w.cu_seqlens,
                                w.scale)
    q32, k32, v32 = W.make_inputs_f32(w)
    ref_f32 = ts_ref.attn_full(q32.double().numpy(), k32.double().numpy(), v32.double().numpy(),
                               w.cu_seqlens, w.scale)
    e_bf16 = assert_parity(got, ref_bf16, "tiny")
    e_f32 = errors(got, ref_f32)
    say("tiny: oracle on bf16 inputs", e_bf16, "oracle on fp32 inputs", e_f32)
