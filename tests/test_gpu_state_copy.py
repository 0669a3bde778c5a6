"""GPU tests of ts_state_copy (session suspend / resume / compaction copies) against the oracle
(oracle/state_copy.py), bit for bit, in every direction: device -> pinned host, pinned host ->
device, device -> device and pinned host -> pinned host; more ranges than one launch holds;
ranges of zero bytes; a full offload -> resume round trip of sessions of a packed KV batch; and
the refusal of pageable host memory.
"""
import sys

import numpy as np
import pytest
import torch

import workloads as W
from oracle import state_copy as SC

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


def rand_u8(n, seed):
    return torch.from_numpy(np.random.default_rng(seed).integers(0, 256, n, dtype=np.uint8))


def buffer(data, where):
    if where == "dev":
        return data.cuda()
    t = torch.empty(data.numel(), dtype=torch.uint8, pin_memory=True)
    t.copy_(data)
    return t


def rand_ranges(n, src_bytes, dst_bytes, seed, max_len=1 << 16):
    """n non-overlapping destination ranges (multiples of 16) in random order."""
    rng = np.random.default_rng(seed)
    lens = rng.integers(0, max_len // 16, n) * 16
    lens[rng.random(n) < 0.1] = 0
    gaps = rng.integers(0, 64, n) * 16
    dst_off = np.cumsum(np.concatenate([[0], (lens + gaps)[:-1]]))
    assert dst_off[-1] + lens[-1] <= dst_bytes
    src_off = np.array([rng.integers(0, (src_bytes - l) // 16 + 1) * 16 for l in lens])
    perm = rng.permutation(n)
    return [(int(src_off[i]), int(dst_off[i]), int(lens[i])) for i in perm]


@pytest.mark.parametrize("src_where,dst_where", [("dev", "host"), ("host", "dev"), ("dev", "dev"),
                                                 ("host", "host")])
def test_copy_directions_bitwise(src_where, dst_where):
    sb, db = 3 << 20, 4 << 20
    src0, dst0 = rand_u8(sb, 1), rand_u8(db, 2)
    ranges = rand_ranges(40, sb, db, 3)
    say("copy", src_where, "->", dst_where, len(ranges))
    src, dst = buffer(src0, src_where), buffer(dst0, dst_where)
    ts.ts_state_copy(src, dst, ranges)
    torch.cuda.synchronize()
    ref = SC.copy_ranges(src0.numpy(), dst0.numpy(), ranges)
    assert np.array_equal(dst.cpu().numpy(), ref)


def test_more_ranges_than_one_launch_and_one_large_range():
    sb, db = 8 << 20, 16 << 20
    src0, dst0 = rand_u8(sb, 4), rand_u8(db, 5)
    ranges = rand_ranges(150, sb, db // 2, 6, max_len=1 << 15)  # 150 > 64 ranges per launch
    ranges.append((16, db // 2, sb - 32))                       # ~8 MB, not a chunk multiple
    src, dst = buffer(src0, "dev"), buffer(dst0, "host")
    ts.ts_state_copy(src, dst, ranges)
    torch.cuda.synchronize()
    assert np.array_equal(dst.numpy(), SC.copy_ranges(src0.numpy(), dst0.numpy(), ranges))


def test_offload_and_resume_sessions_round_trip():
    """Suspend sessions 3 and 1 of a packed KV batch to pinned host memory, clear their rows on the
    device, resume them into a fresh batch, and compact the remaining sessions into a new packed
    batch: every byte must come back exactly (paper Sec. 3.1 suspension and resumption)."""
    w = W.KvWorkload("t", (10, 0, 30, 25, 5), (700, 64, 0, 1000, 333), 3, 64, 9)
    _, k, v = W.make_kv_inputs(w)
    row = w.H * w.d * 2
    kd, vd = k.cuda(), v.cuda()
    sessions = [3, 1]
    rk, end_k = ts.pack_ranges(w.cu_k, sessions, row)
    rv, end_v = ts.pack_ranges(w.cu_k, sessions, row, dst_start=end_k)
    host = torch.empty(end_v, dtype=torch.uint8, pin_memory=True)
    ts.ts_state_copy(kd.view(torch.uint8).view(-1), host, rk)
    ts.ts_state_copy(vd.view(torch.uint8).view(-1), host, rv)
    torch.cuda.synchronize()
    # the host image equals the oracle's
    ref_ranges_k, e1 = SC.session_ranges(w.cu_k, sessions, row)
    ref_ranges_v, e2 = SC.session_ranges(w.cu_k, sessions, row, dst_start=e1)
    assert (ref_ranges_k, e1, ref_ranges_v, e2) == (rk, end_k, rv, end_v)
    ref = SC.copy_ranges(W.bf16_bits(k).view(np.uint8).ravel(), np.zeros(end_v, np.uint8), ref_ranges_k)
    ref = SC.copy_ranges(W.bf16_bits(v).view(np.uint8).ravel(), ref, ref_ranges_v)
    assert np.array_equal(host.numpy(), ref)
    # resume into cleared device tensors at the original places
    k2, v2 = torch.zeros_like(kd), torch.zeros_like(vd)
    ts.ts_state_copy(host, k2.view(torch.uint8).view(-1), [(d, s, n) for s, d, n in rk])
    ts.ts_state_copy(host, v2.view(torch.uint8).view(-1), [(d, s, n) for s, d, n in rv])
    torch.cuda.synchronize()
    for s in sessions:
        a, b = int(w.cu_k[s]), int(w.cu_k[s + 1])
        assert torch.equal(k2[a:b].cpu().view(torch.int16), k[a:b].view(torch.int16))
        assert torch.equal(v2[a:b].cpu().view(torch.int16), v[a:b].view(torch.int16))
    # compact the sessions that stay (0, 2, 4) into a new packed batch on the device
    stay = [0, 2, 4]
    rc, end = ts.pack_ranges(w.cu_k, stay, row)
    kc = torch.empty(end, dtype=torch.uint8, device="cuda")
    ts.ts_state_copy(kd.view(torch.uint8).view(-1), kc, rc)
    torch.cuda.synchronize()
    expect = torch.cat([k[int(w.cu_k[s]):int(w.cu_k[s + 1])] for s in stay])
    assert torch.equal(kc.cpu().view(torch.int16).view(-1), expect.view(torch.int16).view(-1))


def test_pageable_host_memory_is_refused():
    # zero-byte ranges: nothing would be launched even if the check were to pass
    dev = torch.zeros(4096, dtype=torch.uint8, device="cuda")
    pageable = torch.zeros(4096, dtype=torch.uint8)
    assert not pageable.is_pinned()
    lib = ts.load()
    import ctypes
    r = np.zeros((1, 3), np.int64)
    rc = lib.ts_state_copy(ctypes.c_void_p(dev.data_ptr()), 4096, ctypes.c_void_p(pageable.data_ptr()),
                           4096, ctypes.c_void_p(r.ctypes.data), 1, ctypes.c_void_p(None))
    assert rc == 11  # TS_ERR_MEMORY
    with pytest.raises(ValueError):
        ts.ts_state_copy(dev, pageable, [(0, 0, 0)])
