"""HIP graph capture of the C ABI on the GPU: a dense call recorded by stream capture replays
with the inputs as they are at replay time, bit-identical to eager calls, over several replays
with eager work in between; packed, chunk and copy calls refuse capture with TS_ERR_CAPTURE and
leave the capture usable."""
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


def test_packed_chunk_and_copy_calls_refuse_capture():
    w = W.Workload("graph", (300, 0, 129), 2, 128, 903)
    q, k, v = (t.cuda() for t in W.make_inputs(w))
    cu = torch.tensor(w.cu_seqlens, device="cuda")
    ref = ts.ts_attn_fwd_varlen(q, k, v, cu, w.max_seqlen)  # eager, before the capture
    torch.cuda.synchronize()
    src = torch.zeros(4096, dtype=torch.uint8, device="cuda")
    dst = torch.zeros_like(src)
    g = torch.cuda.CUDAGraph()
    say("capture with refused calls")
    with torch.cuda.graph(g):
        y = q * 2  # the graph records something of its own
        with pytest.raises(ts.TsAttnError) as e1:
            ts.ts_attn_fwd_varlen(q, k, v, cu, w.max_seqlen)
        with pytest.raises(ts.TsAttnError) as e2:
            ts.ts_attn_fwd_kvcache(q, k, v, cu, cu, w.max_seqlen, w.max_seqlen)
        with pytest.raises(ts.TsAttnError) as e3:
            ts.ts_state_copy(src, dst, [(0, 0, 4096)])
    for e in (e1, e2, e3):
        assert e.value.status == TS_ERR_CAPTURE, e.value
    g.replay()
    torch.cuda.synchronize()
    assert torch.equal(y, q * 2)
    # and the same calls work eagerly afterwards
    o = ts.ts_attn_fwd_varlen(q, k, v, cu, w.max_seqlen)
    torch.cuda.synchronize()
    assert torch.equal(bits(o), bits(ref))
