"""HIP graph capture of the C ABI on the GPU: dense, packed and chunk calls recorded by stream
capture replay with the inputs as they are at replay time, bit-identical to eager calls, over
several replays with eager work in between (on a capturing stream the packed and chunk calls run
on the static scratch array of the allocation-free call); the copy call refuses capture with
TS_ERR_CAPTURE and leaves the capture usable."""
import sys

import numpy as np
import pytest
import torch

import workloads as W

pytestmark = pytest.mark.gpu

ts = pytest.importorskip("paper_2606_19271_amd")
from paper_2606_19271_amd import _lib  # noqa: E402

TS_ERR_CAPTURE = _lib.STATUS_NAMES.index("TS_ERR_CAPTURE")


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
    return t.contiguous().view(torch.int16)


@pytest.mark.parametrize("d", [64, 128])
def test_dense_call_replays_from_a_graph(d):
    B, L, H = 2, 700, 3
    sets = []
    for seed in (901, 902):
        w = W.Workload("graph", (L,) * B, H, d, seed + d)
        q, k, v = W.make_inputs(w)
        sets.append(tuple(t.cuda().view(B, L, H, d) for t in (q, k, v)))
    # eager references (this also makes the device's first call outside capture)
    refs = [ts.ts_attn_fwd(*s) for s in sets]
    torch.cuda.synchronize()
    q, k, v = (t.clone() for t in sets[0])
    out = torch.empty_like(q)
    g = torch.cuda.CUDAGraph()
    say("capture dense", B, L, H, d)
    with torch.cuda.graph(g):
        ts.ts_attn_fwd(q, k, v, out=out)
    for rep in range(5):
        src = sets[rep % 2]
        for dst, s in zip((q, k, v), src):  # eager work between replays: new inputs in place
            dst.copy_(s)
        out.fill_(0)
        g.replay()
        torch.cuda.synchronize()
        say("replay", rep)
        assert torch.equal(bits(out), bits(refs[rep % 2])), "replay %d differs from the eager call" % rep
    # the eager entry point still works after the capture
    again = ts.ts_attn_fwd(*sets[1])
    torch.cuda.synchronize()
    assert torch.equal(bits(again), bits(refs[1]))


# (segments of queries, segments of keys, H, d, num_splits): several segments (planning kernel),
# one segment (no planning kernel), split key ranges (merge kernel), the library's split choice
GRAPH_CASES = [
    ((300, 0, 129), None, 2, 128, 1),
    ((1000,), None, 2, 64, 1),
    ((300, 129), (900, 130), 2, 128, 2),
    ((700,), (2600,), 3, 128, 0),
]


@pytest.mark.parametrize("lq,lk,H,d,splits", GRAPH_CASES)
def test_packed_and_chunk_calls_replay_from_a_graph(lq, lk, H, d, splits):
    kv = lk is not None
    sets = []
    for seed in (904, 905):
        if kv:
            w = W.KvWorkload("graph", lq, lk, H, d, seed, True)
            q, k, v = W.make_kv_inputs(w)
            cq, ck = torch.tensor(w.cu_q, device="cuda"), torch.tensor(w.cu_k, device="cuda")
            mq, mk = w.max_q, w.max_k
        else:
            w = W.Workload("graph", lq, H, d, seed)
            q, k, v = W.make_inputs(w)
            cq = ck = torch.tensor(w.cu_seqlens, device="cuda")
            mq = mk = w.max_seqlen
        sets.append((q.cuda(), k.cuda(), v.cuda()))

    def call(q, k, v, out=None, lse=None):
        if kv:
            return ts.ts_attn_fwd_kvcache(q, k, v, cq, ck, mq, mk, out=out, lse=lse,
                                          return_lse=True, num_splits=splits)
        return ts.ts_attn_fwd_varlen(q, k, v, cq, mq, out=out), None

    refs = [call(*s) for s in sets]  # eager references (allocating calls, outside capture)
    torch.cuda.synchronize()
    q, k, v = (t.clone() for t in sets[0])
    out = torch.empty_like(q)
    lse = torch.empty((q.shape[0], H), dtype=torch.float32, device="cuda") if kv else None
    g = torch.cuda.CUDAGraph()
    say("capture", "kv" if kv else "packed", lq, lk, H, d, splits)
    with torch.cuda.graph(g):
        call(q, k, v, out=out, lse=lse)
    for rep in range(5):
        src = sets[rep % 2]
        for dst, s in zip((q, k, v), src):  # eager work between replays: new inputs in place
            dst.copy_(s)
        out.fill_(0)
        if kv:
            lse.fill_(0)
        g.replay()
        torch.cuda.synchronize()
        say("replay", rep)
        ro, rl = refs[rep % 2]
        assert torch.equal(bits(out), bits(ro)), "replay %d differs from the eager call" % rep
        if kv:
            assert torch.equal(lse.view(torch.int32), rl.view(torch.int32)), rep


def test_copy_call_refuses_capture():
    q = torch.zeros((64, 2, 128), dtype=torch.bfloat16, device="cuda")
    src = torch.zeros(4096, dtype=torch.uint8, device="cuda")
    dst = torch.zeros_like(src)
    g = torch.cuda.CUDAGraph()
    say("capture with a refused copy")
    with torch.cuda.graph(g):
        y = q * 2  # the graph records something of its own
        with pytest.raises(ts.TsAttnError) as e:
            ts.ts_state_copy(src, dst, [(0, 0, 4096)])
    assert e.value.status == TS_ERR_CAPTURE, e.value
    g.replay()
