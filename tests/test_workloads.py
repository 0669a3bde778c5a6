"""The seeded workload generator: reproducible draws, shapes, and the metric's per-call counts."""
import numpy as np
import pytest
import torch

import workloads as W


def test_draws_are_reproducible_and_bf16():
    w = W.Workload("x", (100, 28), 3, 64, 7, k_offset=True)
    a, b = W.make_inputs(w), W.make_inputs(w)
    for x, y in zip(a, b):
        assert x.dtype == torch.bfloat16 and x.shape == (128, 3, 64)
        assert torch.equal(x.view(torch.int16), y.view(torch.int16))
    assert W.sha256(a[0]) == W.sha256(b[0])
    c = W.make_inputs(w, seed=8)
    assert not torch.equal(a[0], c[0])


def test_k_offset_is_per_head_channel():
    w0 = W.Workload("x", (4000,), 2, 64, 3, k_offset=False)
    w1 = W.Workload("x", (4000,), 2, 64, 3, k_offset=True)
    k0, k1 = W.make_inputs(w0)[1].float(), W.make_inputs(w1)[1].float()
    shift = (k1 - k0).mean(dim=0)  # ~ the offset, one value per (head, channel)
    assert shift.shape == (2, 64)
    assert 0.8 < float(shift.std()) < 2.0  # std sqrt(2) ~ 1.41
    assert float(k0.mean(dim=0).abs().max()) < 0.1


def test_workload_table():
    t = {n: W.WORKLOADS[n] for n in W.ORDER}
    assert t["tiny"].T == 1024 and t["tiny"].H == 2 and t["tiny"].d == 64
    assert t["dit_large"].T == 32760 == 21 * 30 * 52
    assert t["highres"].T == 75600 == 21 * 45 * 80
    assert t["varlen_serving"].T == 101010
    assert list(t["varlen_serving"].cu_seqlens) == [0, 8190, 16380, 32760, 65520, 98280, 101010]
    # Sum_s 4 L_s^2 d H
    assert t["tiny"].flops == 4 * 1024 ** 2 * 64 * 2
    assert abs(t["dit_large"].flops - 2.198e13) / 2.198e13 < 1e-3
    assert abs(t["highres"].flops - 1.1705e14) / 1.1705e14 < 1e-3
    assert abs(t["varlen_serving"].flops - 1.5706e13) / 1.5706e13 < 1e-3
    assert t["dit_large"].hbm_bytes == 4 * 32760 * 40 * 128 * 2
    assert t["tiny"].scale == 0.125
    assert np.float32(t["dit_large"].scale) == np.float32(1) / np.sqrt(np.float32(128))


def test_sample_rows_cover_segment_ends_for_every_head():
    w = W.WORKLOADS["varlen_serving"]
    rt, rh = W.sample_rows(w, full_tiles=False)
    assert rt.size == rh.size == w.H * 6 * 66
    cu = w.cu_seqlens
    for h in range(w.H):
        ts = set(rt[rh == h].tolist())
        for s in range(6):
            assert cu[s] in ts and cu[s + 1] - 1 in ts
    assert rt.min() >= 0 and rt.max() < w.T
    rt2, _ = W.sample_rows(w, full_tiles=False)
    assert np.array_equal(rt, rt2)


@pytest.mark.parametrize("name", ["dit_small", "dit_large", "highres", "varlen_serving"])
def test_sample_rows_reach_every_tile_slot_and_differ_per_head(name):
    """Every (wave, lane) slot of a 256-query tile is sampled in every segment that has it, the
    random rows differ between heads, and one complete tile plus the ragged last tile of every
    segment are included whole."""
    w = W.WORKLOADS[name]
    rt, rh = W.sample_rows(w)
    cu = w.cu_seqlens
    seg = np.searchsorted(cu, rt, side="right") - 1
    for s in range(len(w.seqlens)):
        lo, hi = int(cu[s]), int(cu[s + 1])
        sel = seg == s
        assert set(((rt[sel] - lo) % 256).tolist()) == set(range(min(256, hi - lo)))
        assert set(range(256 * ((hi - lo) // 256) + lo, hi)) <= set(rt[sel].tolist())
        t0 = [t for t in range(lo, hi - 255, 256) if set(range(t, t + 256)) <= set(rt[sel].tolist())]
        assert t0, (name, s)
    a, b = set(rt[rh == 0].tolist()), set(rt[rh == 1].tolist())
    assert len(a ^ b) > 100
    assert rt.min() >= 0 and rt.max() < w.T and rh.max() < w.H


def test_kv_workloads_shapes_and_draws():
    for w in W.KV_WORKLOADS.values():
        assert len(w.q_seqlens) == len(w.k_seqlens)
        assert w.cu_q[-1] == w.Tq and w.cu_k[-1] == w.Tk
        assert all(b >= a for a, b in zip(w.q_seqlens, w.k_seqlens))  # keys include the chunk
        assert w.flops == sum(4 * a * b * w.d * w.H for a, b in zip(w.q_seqlens, w.k_seqlens))
    w = W.KvWorkload("t", (5, 0, 9), (20, 3, 9), 2, 64, 3, True)
    q, k, v = W.make_kv_inputs(w)
    assert q.shape == (14, 2, 64) and k.shape == v.shape == (32, 2, 64)
    assert q.dtype == k.dtype == v.dtype == torch.bfloat16
    q2, k2, v2 = W.make_kv_inputs(w)
    assert torch.equal(q, q2) and torch.equal(k, k2) and torch.equal(v, v2)
    row_t, row_h = W.sample_kv_rows(w, n_random=4)
    assert set(row_t.tolist()) >= {0, 4, 5, 13} and row_t.max() < w.Tq
    assert row_h.max() == 1
