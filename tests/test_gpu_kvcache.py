"""GPU parity of ts_attn_fwd_kvcache (chunk queries against per-session key/value ranges, with the
log-sum-exp output and the split-key path) against the fp64 oracle, through the C ABI.

Bars: the output O to the same bar as every other entry point (tests/metrics.py).  The lse to an
absolute 1e-2: the kernel's lse is (running max + log2 of the fp32 sum of the bf16-rounded
weights) * ln 2, and rounding each weight to bf16 changes that sum by at most 2^-9 relative,
i.e. the lse by at most 2e-3 (plus fp32 rounding); the bar leaves a factor of five.
"""
import os
import sys
import time

import numpy as np
import pytest
import torch

import workloads as W
from metrics import assert_parity, assert_rows
from oracle import ts_ref

pytestmark = pytest.mark.gpu

ts = pytest.importorskip("paper_2606_19271_amd")

LSE_ABS = 1e-2


def say(*a):
    print("[gpu-test]", *a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ts.load()
    return torch.device("cuda:0")


def draw(lq, lk, H, d, seed, k_offset=False):
    w = W.KvWorkload("custom", tuple(lq), tuple(lk), H, d, seed, k_offset)
    return (w,) + W.make_kv_inputs(w)


def run_kv(w, q, k, v, splits=0, scale=None, lse=True):
    cq = torch.tensor(w.cu_q, device="cuda")
    ck = torch.tensor(w.cu_k, device="cuda")
    r = ts.ts_attn_fwd_kvcache(q.cuda(), k.cuda(), v.cuda(), cq, ck, w.max_q, w.max_k,
                               scale=scale, return_lse=lse, num_splits=splits)
    torch.cuda.synchronize()
    if lse:
        return r[0].cpu(), r[1].cpu()
    return r.cpu(), None


def oracle(w, q, k, v, scale):
    return ts_ref.attn_kv_full(W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v), w.cu_q, w.cu_k, scale)


def check_lse(got, ref, what):
    got = got.double().numpy()
    fin = np.isfinite(ref)
    assert np.array_equal(np.isfinite(got), fin), what + ": -inf pattern differs"
    assert np.all(got[~fin] == -np.inf), what
    err = float(np.max(np.abs(got[fin] - ref[fin]))) if fin.any() else 0.0
    assert err <= LSE_ABS, "%s: lse max-abs %.3g" % (what, err)
    return err


def as_f64(o):
    return o.float().numpy().astype(np.float64)


# segments: several query and key tiles, ragged tails, a segment without keys, one without queries,
# a one-query segment and a one-key segment
LQ = [100, 0, 300, 257, 1, 40]
LK = [700, 50, 0, 1000, 64, 1]


@pytest.mark.parametrize("d", [64, 128])
def test_kv_full(d):
    w, q, k, v = draw(LQ, LK, 3, d, 31, k_offset=True)
    say("kv full", d, LQ, LK)
    o, lse = run_kv(w, q, k, v, splits=1)
    ro, rlse = oracle(w, q, k, v, w.scale)
    e = assert_rows(as_f64(o), ro, "kv full d=%d" % d, elementwise=False)
    le = check_lse(lse, rlse, "kv full d=%d" % d)
    say("errors", e, "lse", le)
    nokeys = slice(int(w.cu_q[2]), int(w.cu_q[3]))  # queries of the segment without keys
    assert torch.all(o[nokeys].float() == 0.0)


@pytest.mark.parametrize("splits", [2, 3, 7, 16])
@pytest.mark.parametrize("d", [64, 128])
def test_kv_forced_splits_full(splits, d):
    w, q, k, v = draw(LQ, LK, 2, d, 41)
    say("kv splits", splits, d)
    o, lse = run_kv(w, q, k, v, splits=splits)
    ro, rlse = oracle(w, q, k, v, w.scale)
    assert_rows(as_f64(o), ro, "kv splits=%d d=%d" % (splits, d), elementwise=False)
    check_lse(lse, rlse, "kv splits=%d d=%d" % (splits, d))
    # the split result differs from the unsplit one only by the rounding of the partials
    o1, _ = run_kv(w, q, k, v, splits=1)
    assert float((o.float() - o1.float()).abs().max()) <= 2e-2


# Query tiles of at most 32 queries take the thin path: the eight waves share the tile, each with
# 16 of its queries and a quarter of every key tile, and combine their partial results at the end.
# Query tails on both sides of 16 and 32, against key counts on both sides of the 16-key blocks,
# of a wave's quarter and of the key tile (a wave may see no key at all in the masked last tile).
THIN_LQ = [1, 8, 16, 17, 24, 31, 32, 33, 256 + 24, 512 + 32]
THIN_LK = [1, 15, 17, 40, 64, 129, 300, 700, 2000, 5000]


@pytest.mark.parametrize("splits", [1, 3, 0])
@pytest.mark.parametrize("d", [64, 128])
def test_kv_thin_query_tiles_full(splits, d):
    w, q, k, v = draw(THIN_LQ, THIN_LK, 3, d, 111 + d, k_offset=True)
    what = "kv thin d=%d splits=%d" % (d, splits)
    say(what)
    o, lse = run_kv(w, q, k, v, splits=splits)
    ro, rlse = oracle(w, q, k, v, w.scale)
    e = assert_rows(as_f64(o), ro, what, elementwise=False)
    le = check_lse(lse, rlse, what)
    say("errors", e, "lse", le)


@pytest.mark.parametrize("seed", range(10))
def test_kv_random_batches_full(seed):
    # seeded random chunk batches: per segment a query count and a key count drawn independently
    # (either may be zero or sit on a tile edge), random heads, head dim, scale and split count
    # (0 = the library's choice), with and without a per-channel offset on K (which shifts the
    # scores and so the running maximum)
    rng = np.random.default_rng(5200 + seed)
    edge = [0, 1, 63, 64, 65, 255, 256, 257]
    nseq = int(rng.integers(1, 8))
    lq = [int(rng.choice(edge)) if rng.random() < 0.4 else int(rng.integers(1, 600)) for _ in range(nseq)]
    lk = [int(rng.choice(edge)) if rng.random() < 0.4 else int(rng.integers(1, 2000)) for _ in range(nseq)]
    if sum(lq) == 0:
        lq[0] = 1
    if sum(lk) == 0:
        lk[0] = 1
    H = int(rng.choice([1, 2, 4]))
    d = int(rng.choice([64, 128]))
    scale = None if rng.random() < 0.5 else float(np.float32(rng.uniform(-1.0, 1.5)))
    splits = int(rng.choice([0, 0, 1, 2, 5]))
    k_offset = bool(rng.random() < 0.5)
    w, q, k, v = draw(lq, lk, H, d, 5300 + seed, k_offset=k_offset)
    sc = w.scale if scale is None else scale
    what = "kv random seed=%d lq=%r lk=%r H=%d d=%d scale=%r splits=%d" % (seed, lq, lk, H, d, scale, splits)
    say(what)
    o, lse = run_kv(w, q, k, v, splits=splits, scale=scale)
    ro, rlse = oracle(w, q, k, v, sc)
    assert_rows(as_f64(o), ro, what, elementwise=False)
    check_lse(lse, rlse, what)


def test_kv_equal_offsets_is_varlen_bitwise():
    lens = [300, 0, 1000, 65, 1]
    w, q, k, v = draw(lens, lens, 2, 128, 51)
    q = W.make_kv_inputs(w, seed=52)[0][: w.Tq]
    say("kv == varlen", lens)
    o_kv, lse = run_kv(w, q, k, v, splits=1)
    cu = torch.tensor(w.cu_q, device="cuda")
    o_var = ts.ts_attn_fwd_varlen(q.cuda(), k.cuda(), v.cuda(), cu, w.max_q)
    torch.cuda.synchronize()
    assert torch.equal(o_kv.view(torch.int16), o_var.cpu().view(torch.int16))
    _, rlse = oracle(w, q, k, v, w.scale)
    check_lse(lse, rlse, "kv == varlen")


def test_kv_without_lse_matches_with_lse():
    w, q, k, v = draw(LQ, LK, 2, 128, 61)
    a, _ = run_kv(w, q, k, v, splits=1, lse=False)
    b, _ = run_kv(w, q, k, v, splits=1, lse=True)
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    c, _ = run_kv(w, q, k, v, splits=4, lse=False)
    d, _ = run_kv(w, q, k, v, splits=4, lse=True)
    assert torch.equal(c.view(torch.int16), d.view(torch.int16))


@pytest.mark.parametrize("scale", [0.0, -0.3, 0.9])
def test_kv_other_scales(scale):
    w, q, k, v = draw([70, 200], [500, 129], 2, 64, 71)
    for splits in (1, 3):
        o, lse = run_kv(w, q, k, v, splits=splits, scale=scale)
        ro, rlse = oracle(w, q, k, v, scale)
        assert_rows(as_f64(o), ro, "kv scale=%g splits=%d" % (scale, splits),
                    elementwise=False)
        check_lse(lse, rlse, "kv scale=%g splits=%d" % (scale, splits))


def test_kv_deterministic_bitwise():
    w, q, k, v = draw(LQ, LK, 2, 128, 81)
    for splits in (1, 5):
        a, la = run_kv(w, q, k, v, splits=splits)
        b, lb = run_kv(w, q, k, v, splits=splits)
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))
        assert torch.equal(la.view(torch.int32), lb.view(torch.int32))


@pytest.mark.parametrize("name,n_random", [("kv_chunk", 12), ("kv_chunk_1s", 48)])
def test_kv_workload_sampled(name, n_random):
    """The full chunk-vs-cache workloads in the configuration the benchmark times (automatic
    splits), checked on sampled query rows of every head."""
    w = W.KV_WORKLOADS[name]
    q, k, v = W.make_kv_inputs(w)
    say("kv workload", name, w.Tq, w.Tk, w.H)
    o, lse = run_kv(w, q, k, v, splits=0)
    row_t, row_h = W.sample_kv_rows(w, n_random=n_random)
    ro, rlse = ts_ref.attn_kv_rows(W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v), w.cu_q, w.cu_k,
                                   w.scale, row_t, row_h)
    got = as_f64(o[torch.from_numpy(row_t), torch.from_numpy(row_h.astype(np.int64))])
    e = assert_rows(got, ro, name)
    le = check_lse(lse[torch.from_numpy(row_t), torch.from_numpy(row_h.astype(np.int64))], rlse, name)
    say(name, "errors", e, "lse", le)
    assert float(np.abs(got).mean()) > 1e-3  # not an all-zero output


def test_kv_rejected_offsets_leave_outputs_untouched():
    # a rejected plan is a no-op on every path: also with split key ranges, where the merge
    # kernel must not write O or lse from partials that were never computed
    w, q, k, v = draw([64, 64], [128, 128], 1, 64, 92)
    cq = torch.tensor(w.cu_q, device="cuda")
    bad_k = torch.tensor([0, 200, 256], dtype=torch.int32, device="cuda")  # segment longer than max_k
    for splits in (1, 3):
        o = torch.full((w.Tq, 1, 64), 7.0, dtype=torch.bfloat16, device="cuda")
        lse = torch.full((w.Tq, 1), 123.0, dtype=torch.float32, device="cuda")
        say("kv rejected offsets, splits", splits)
        ts.ts_attn_fwd_kvcache(q.cuda(), k.cuda(), v.cuda(), cq, bad_k, w.max_q, 128, out=o, lse=lse,
                               num_splits=splits)
        torch.cuda.synchronize()
        assert bool((o == 7.0).all()) and bool((lse == 123.0).all()), "splits=%d" % splits


@pytest.mark.parametrize("splits", [1, 3])
def test_kv_one_segment_bad_offsets_are_noops(splits):
    # A call of one segment runs without the planning kernel: the attention and merge kernels
    # check its offsets against {0, total} themselves.  Offsets that do not start at 0 or do not
    # end at the tensors' rows leave O and lse untouched; so do totals beyond max_seqlen, which
    # the host turns away before any device work; and validation mode still reports them.
    w, q, k, v = draw([64], [128], 1, 64, 93)
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    bad = [([0, 64], [0, 100], 64, 128), ([0, 64], [28, 128], 64, 128), ([5, 64], [0, 128], 64, 128),
           ([0, 64], [0, 128], 32, 128), ([0, 64], [0, 128], 64, 100)]
    for cq_l, ck_l, max_q, max_k in bad:
        o = torch.full((64, 1, 64), 7.0, dtype=torch.bfloat16, device="cuda")
        lse = torch.full((64, 1), 123.0, dtype=torch.float32, device="cuda")
        what = "one segment cu_q=%r cu_k=%r max=%d,%d splits=%d" % (cq_l, ck_l, max_q, max_k, splits)
        say(what)
        cq = torch.tensor(cq_l, dtype=torch.int32, device="cuda")
        ck = torch.tensor(ck_l, dtype=torch.int32, device="cuda")
        ts.ts_attn_fwd_kvcache(qd, kd, vd, cq, ck, max_q, max_k, out=o, lse=lse, num_splits=splits)
        torch.cuda.synchronize()
        assert bool((o == 7.0).all()) and bool((lse == 123.0).all()), what
        os.environ["TS_ATTN_VALIDATE"] = "1"
        try:
            with pytest.raises(ts.TsAttnError) as ei:
                ts.ts_attn_fwd_kvcache(qd, kd, vd, cq, ck, max_q, max_k, out=o, num_splits=splits)
            assert ei.value.status == 10, what
        finally:
            del os.environ["TS_ATTN_VALIDATE"]
    # the same tensors with their true offsets give the oracle's result
    o, l = run_kv(w, q, k, v, splits=splits)
    ro, rl = oracle(w, q, k, v, w.scale)
    assert_rows(as_f64(o), ro, "one segment splits=%d" % splits, elementwise=False)
    check_lse(l, rl, "one segment splits=%d" % splits)


def test_split_calls_share_the_workspace_across_streams_without_blocking_the_host():
    """Split chunk calls take their plan and partials from the device's cached workspace, which
    successive calls take in turn through an event waited for on the GPU.  Two streams enqueue
    alternating calls on different inputs with no synchronization in between: every result
    equals the one computed alone, bit for bit.  And the host does not wait for the GPU: 20
    calls of about 0.3 ms each are enqueued in well under half the time they take to run."""
    w = W.KV_WORKLOADS["kv_chunk_1s"]
    sets = []
    for seed in (101, 102):
        q, k, v = W.make_kv_inputs(w, seed=seed)
        sets.append((q.cuda(), k.cuda(), v.cuda()))
    cq = torch.tensor(w.cu_q, device="cuda")
    ck = torch.tensor(w.cu_k, device="cuda")
    refs = []
    for qd, kd, vd in sets:
        refs.append(ts.ts_attn_fwd_kvcache(qd, kd, vd, cq, ck, w.max_q, w.max_k, return_lse=True,
                                           num_splits=3))
        torch.cuda.synchronize()
    outs = [[(torch.empty_like(sets[j][0]), torch.empty((w.Tq, w.H), dtype=torch.float32,
                                                        device="cuda")) for _ in range(6)]
            for j in range(2)]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    say("two streams, shared workspace")
    for i in range(6):
        for j in range(2):
            with torch.cuda.stream(streams[j]):
                qd, kd, vd = sets[j]
                ts.ts_attn_fwd_kvcache(qd, kd, vd, cq, ck, w.max_q, w.max_k, out=outs[j][i][0],
                                       lse=outs[j][i][1], num_splits=3)
    torch.cuda.synchronize()
    for j in range(2):
        for i in range(6):
            assert torch.equal(outs[j][i][0].view(torch.int16), refs[j][0].view(torch.int16)), (j, i)
            assert torch.equal(outs[j][i][1].view(torch.int32), refs[j][1].view(torch.int32)), (j, i)
    qd, kd, vd = sets[0]
    o, lse = outs[0][0]
    t0 = time.perf_counter()
    for _ in range(20):
        ts.ts_attn_fwd_kvcache(qd, kd, vd, cq, ck, w.max_q, w.max_k, out=o, lse=lse, num_splits=3)
    t1 = time.perf_counter()
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    say("enqueue %.2f ms, run %.2f ms" % ((t1 - t0) * 1e3, (t2 - t0) * 1e3))
    assert t1 - t0 < 0.5 * (t2 - t0), (t1 - t0, t2 - t0)


def test_kv_offsets_that_wrap_int32_are_rejected():
    # key offsets whose wrapping differences pass a differences-only check (see the packed test)
    Tk, nseq, max_k = 1024, 512, (1 << 24) - 512
    diffs = [max_k] * 256 + [(1 << 32) + Tk - 256 * max_k] + [0] * (nseq - 257)
    ck = [0]
    for x in diffs:
        ck.append(((ck[-1] + x + (1 << 31)) % (1 << 32)) - (1 << 31))
    assert ck[-1] == Tk and min(ck) < 0
    cq = [0] + [1] * nseq  # one query in the first segment
    q = torch.randn((1, 1, 64)).to(torch.bfloat16).cuda()
    kv = torch.randn((Tk, 1, 64)).to(torch.bfloat16).cuda()
    o = torch.full((1, 1, 64), 7.0, dtype=torch.bfloat16, device="cuda")
    say("kv wrapping offsets")
    for splits in (1, 3):
        ts.ts_attn_fwd_kvcache(q, kv, kv, torch.tensor(cq, dtype=torch.int32, device="cuda"),
                               torch.tensor(ck, dtype=torch.int32, device="cuda"), 1, max_k, out=o,
                               num_splits=splits)
        torch.cuda.synchronize()
        assert bool((o == 7.0).all()), "splits=%d" % splits


def test_kv_bad_offsets_validate_mode():
    w, q, k, v = draw([64, 64], [128, 128], 1, 64, 91)
    cq = torch.tensor(w.cu_q, device="cuda")
    bad_k = torch.tensor([0, 200, 256], dtype=torch.int32, device="cuda")  # segment longer than max_k
    os.environ["TS_ATTN_VALIDATE"] = "1"
    try:
        with pytest.raises(ts.TsAttnError) as ei:
            ts.ts_attn_fwd_kvcache(q.cuda(), k.cuda(), v.cuda(), cq, bad_k, w.max_q, 128)
        assert ei.value.status == 10
    finally:
        del os.environ["TS_ATTN_VALIDATE"]


@pytest.mark.parametrize("splits", [0, 1, 3])
def test_kv_no_keys_at_all(splits):
    # queries but no keys anywhere: k and v are empty tensors (NULL data pointers), and every
    # row is the empty sum: O = 0, lse = -inf
    H, d, Tq = 2, 128, 300
    g = torch.Generator().manual_seed(8)
    q = torch.randn((Tq, H, d), generator=g).to(torch.bfloat16).cuda()
    k = torch.empty((0, H, d), dtype=torch.bfloat16, device="cuda")
    v = torch.empty((0, H, d), dtype=torch.bfloat16, device="cuda")
    cq = torch.tensor([0, 100, 300], dtype=torch.int32, device="cuda")
    ck = torch.tensor([0, 0, 0], dtype=torch.int32, device="cuda")
    say("no keys", splits)
    o, lse = ts.ts_attn_fwd_kvcache(q, k, v, cq, ck, 200, 0, return_lse=True, num_splits=splits)
    torch.cuda.synchronize()
    assert torch.count_nonzero(o.float()).item() == 0
    assert bool(torch.all(torch.isneginf(lse)).item())


def test_empty_batches_are_no_ops():
    # a coalesced batch without tokens: empty tensors (NULL data pointers) are accepted
    H, d = 2, 128
    e = torch.empty((0, H, d), dtype=torch.bfloat16, device="cuda")
    cu = torch.tensor([0, 0, 0], dtype=torch.int32, device="cuda")
    say("empty batches")
    o = ts.ts_attn_fwd_varlen(e, e, e, cu, 0)
    assert o.shape == (0, H, d)
    o = ts.ts_attn_fwd(e.view(0, 1, H, d), e.view(0, 1, H, d), e.view(0, 1, H, d))
    assert o.numel() == 0
    o, lse = ts.ts_attn_fwd_kvcache(e, e, e, cu, cu, 0, 0, return_lse=True)
    assert o.shape == (0, H, d) and lse.shape == (0, H)
    torch.cuda.synchronize()


@pytest.mark.parametrize("splits", [1, 3])
def test_kv_split_call_at_the_byte_limit_sampled(splits):
    """A query segment at the largest size the ABI accepts, (max_seqlen_q + 256) * H * d * 2 <
    2^31 bytes, with the key range split three ways: the float32 partial results of such a
    segment span up to 2^32 bytes, so their in-segment offsets use the whole unsigned 32-bit
    range of the buffer stores (rows near the segment's end, last head).  Sampled rows of O and
    lse against the oracle; one query more is refused on the host."""
    H, d = 128, 128
    row_bytes = H * d * 2
    Lq = (1 << 31) // row_bytes - 256 - 1          # 65279
    lq, lk = [Lq, 500], [2000, 3000]
    Tq, Tk = sum(lq), sum(lk)
    assert (Lq + 256) * row_bytes < (1 << 31) and (Lq + 256) * H * d * 4 >= (1 << 31)
    say("kv byte limit", "Lq=%d Tq=%d Tk=%d H=%d splits=%d" % (Lq, Tq, Tk, H, splits))
    q = W.make_device_inputs(Tq, H, d, seed=31, device=torch.device("cuda"))[0]
    torch.cuda.empty_cache()
    k, v = W.make_device_inputs(Tk, H, d, seed=32, device=torch.device("cuda"))[1:]
    cq_np = np.array([0, Lq, Tq], dtype=np.int32)
    ck_np = np.array([0, lk[0], Tk], dtype=np.int32)
    cq, ck = torch.from_numpy(cq_np).cuda(), torch.from_numpy(ck_np).cuda()
    scale = W.Workload("x", (1,), H, d, 0).scale
    o, lse = ts.ts_attn_fwd_kvcache(q, k, v, cq, ck, Lq, max(lk), return_lse=True,
                                    num_splits=splits)
    torch.cuda.synchronize()
    with pytest.raises(ts.TsAttnError):
        ts.ts_attn_fwd_kvcache(q, k, v, torch.tensor([0, Lq + 1, Tq], dtype=torch.int32,
                                                     device="cuda"), ck, Lq + 1, max(lk),
                               num_splits=splits)
    rng = np.random.default_rng(6)
    row_t = np.concatenate([[0, Lq - 1, Lq - 2, Lq - 255, Lq - 256, Lq, Tq - 1],
                            rng.integers(Lq - 3000, Lq, 40), rng.integers(0, Tq, 20)]).astype(np.int64)
    row_h = np.concatenate([[0, H - 1, H - 2, H - 1, H - 1, H - 1, H - 1],
                            rng.integers(H - 8, H, 40), rng.integers(0, H, 20)]).astype(np.int64)
    tt, hh = torch.from_numpy(row_t).cuda(), torch.from_numpy(row_h).cuda()
    got, got_lse = o[tt, hh].cpu(), lse[tt, hh].cpu()
    del o, lse
    hq, hk, hv = (W.bf16_bits(x.cpu()) for x in (q, k, v))
    del q, k, v
    torch.cuda.empty_cache()
    ro, rlse = ts_ref.attn_kv_rows(hq, hk, hv, cq_np, ck_np, scale, row_t, row_h.astype(np.int32))
    e = assert_rows(as_f64(got), ro, "kv byte limit")
    le = check_lse(got_lse, rlse, "kv byte limit")
    say("kv byte limit errors", e, "lse", le)
