"""The allocation-free chunk call ts_attn_fwd_kvcache_noalloc, through the C ABI, against the
allocating ts_attn_fwd_kvcache (bit for bit at the same split count) and the fp64 oracle: two
calls in a row, the second on a smaller input; a call whose automatic split count is lowered to
fit the static scratch; and replays of the call recorded into a HIP graph."""
import sys

import numpy as np
import pytest
import torch

import workloads as W
from metrics import assert_parity
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


def bits(t):
    return t.contiguous().view(torch.int32 if t.dtype == torch.float32 else torch.int16)


def inputs(w):
    q, k, v = W.make_kv_inputs(w)
    cq = torch.tensor(w.cu_q, device="cuda")
    ck = torch.tensor(w.cu_k, device="cuda")
    return (q, k, v), (q.cuda(), k.cuda(), v.cuda(), cq, ck, w.max_q, w.max_k)


def both(dev_args, splits):
    """(o, lse) of the allocation-free call, then of the allocating one, same arguments."""
    a = ts.ts_attn_fwd_kvcache_noalloc(*dev_args, return_lse=True, num_splits=splits)
    torch.cuda.synchronize()
    b = ts.ts_attn_fwd_kvcache(*dev_args, return_lse=True, num_splits=splits)
    torch.cuda.synchronize()
    return a, b


def check_oracle(w, host, o, lse, rows=None):
    hq, hk, hv = (W.bf16_bits(x) for x in host)
    if rows is None:
        ro, rl = ts_ref.attn_kv_full(hq, hk, hv, w.cu_q, w.cu_k, w.scale)
        got, gl = o.cpu(), lse.cpu()
    else:
        ro, rl = ts_ref.attn_kv_rows(hq, hk, hv, w.cu_q, w.cu_k, w.scale, *rows)
        tt, hh = torch.from_numpy(rows[0]), torch.from_numpy(rows[1].astype(np.int64))
        got, gl = o.cpu()[tt, hh], lse.cpu()[tt, hh]
    e = assert_parity(got.float().numpy().astype(np.float64), ro, w.name)
    gl = gl.double().numpy()
    fin = np.isfinite(rl)
    assert np.array_equal(np.isfinite(gl), fin) and np.all(gl[~fin] == -np.inf)
    le = float(np.max(np.abs(gl[fin] - rl[fin]))) if fin.any() else 0.0
    assert le <= LSE_ABS, (w.name, le)
    return e, le


def test_noalloc_matches_the_allocating_call_on_two_calls():
    # call 1: a one-frame chunk against a 21-frame cache, automatic split count (three key ranges,
    # 29 MB of partial results: they fit the 32 MiB scratch, so both calls choose the same n)
    w1 = W.KvWorkload("noalloc_1", (1560,), (32760,), 12, 128, 41, True)
    host1, dev1 = inputs(w1)
    say("noalloc call 1", w1.q_seqlens, w1.k_seqlens, w1.H, w1.d)
    (o1, l1), (r1, rl1) = both(dev1, 0)
    assert torch.equal(bits(o1), bits(r1)) and torch.equal(bits(l1), bits(rl1))
    e = check_oracle(w1, host1, o1, l1, W.sample_kv_rows(w1, n_random=24))
    say("call 1 errors", e)
    # call 2, smaller: ragged segments, a segment without keys and one without queries, d = 64,
    # two key ranges; the scratch still holds call 1's contents
    w2 = W.KvWorkload("noalloc_2", (100, 0, 300, 257, 1, 40), (700, 50, 0, 1000, 64, 1), 3, 64,
                      42)
    host2, dev2 = inputs(w2)
    say("noalloc call 2", w2.q_seqlens, w2.k_seqlens, w2.H, w2.d)
    (o2, l2), (r2, rl2) = both(dev2, 2)
    assert torch.equal(bits(o2), bits(r2)) and torch.equal(bits(l2), bits(rl2))
    e = check_oracle(w2, host2, o2, l2)
    say("call 2 errors", e)


def test_noalloc_lowers_the_automatic_split_count_to_fit():
    # 4000 queries x 12 heads against 32760 keys: the library's choice is four key ranges, whose
    # 98 MB of partials do not fit, nor do three or two ranges: one range, bit-identical to the
    # allocating call with num_splits = 1
    w = W.KvWorkload("noalloc_3", (4000,), (32760,), 12, 128, 43, True)
    host, dev = inputs(w)
    say("noalloc lowered splits", w.q_seqlens, w.k_seqlens)
    o, lse = ts.ts_attn_fwd_kvcache_noalloc(*dev, return_lse=True, num_splits=0)
    torch.cuda.synchronize()
    r, rl = ts.ts_attn_fwd_kvcache(*dev, return_lse=True, num_splits=1)
    torch.cuda.synchronize()
    assert torch.equal(bits(o), bits(r)) and torch.equal(bits(lse), bits(rl))
    with pytest.raises(ts.TsAttnError) as ei:
        ts.ts_attn_fwd_kvcache_noalloc(*dev, num_splits=2)
    assert ei.value.status == ts._lib.TS_ERR_SCRATCH
    check_oracle(w, host, o, lse, W.sample_kv_rows(w, n_random=8))


def test_noalloc_call_replays_from_a_graph():
    sets = []
    w = W.KvWorkload("noalloc_g", (300, 129), (900, 130), 2, 128, 44, True)
    for seed in (45, 46):
        sets.append(inputs(W.KvWorkload("noalloc_g", w.q_seqlens, w.k_seqlens, w.H, w.d, seed,
                                        True))[1])
    refs = [ts.ts_attn_fwd_kvcache(*s, return_lse=True, num_splits=2) for s in sets]
    torch.cuda.synchronize()
    q, k, v = (t.clone() for t in sets[0][:3])
    cq, ck = sets[0][3], sets[0][4]
    out = torch.empty_like(q)
    lse = torch.empty((q.shape[0], q.shape[1]), dtype=torch.float32, device="cuda")
    g = torch.cuda.CUDAGraph()
    say("capture noalloc")
    with torch.cuda.graph(g):
        ts.ts_attn_fwd_kvcache_noalloc(q, k, v, cq, ck, w.max_q, w.max_k, out=out, lse=lse,
                                       num_splits=2)
    for rep in range(5):
        src = sets[rep % 2]
        for dst, s in zip((q, k, v), src[:3]):  # eager work between replays: new inputs in place
            dst.copy_(s)
        out.fill_(0)
        lse.fill_(0)
        g.replay()
        torch.cuda.synchronize()
        say("replay", rep)
        ro, rl = refs[rep % 2]
        assert torch.equal(bits(out), bits(ro)) and torch.equal(bits(lse), bits(rl)), rep
