"""Seeded random sweep of every attention entry point against the fp64 oracle, through the C ABI.

Each case is a dense batch, a packed batch, or a chunk-vs-cache batch (allocating, or allocating
and allocation-free on the same arguments), with segment lengths drawn around the 256-query
tile, the 32-query thin tile, the 16-key blocks and the key tiles (64 keys at d = 128, 128 at
d = 64), one segment half of the time (the call then runs without the planning kernel), and
random heads, head width, scale (zero and negative included), score peaking (q x 1, 4, 8) and
split count.  Bars: those of every other parity test (tests/metrics.py, per-row relative bar
included; the element bar is left to the long-segment tests, see metrics.assert_rows), lse within
1e-2 with exact -inf for rows without keys, the dense call bit-identical to the packed one, and
the allocation-free call bit-identical to the allocating one at the same split count."""
import sys

import numpy as np
import pytest
import torch

import workloads as W
from metrics import assert_rows
from oracle import ts_ref

pytestmark = pytest.mark.gpu

ts = pytest.importorskip("paper_2606_19271_amd")

EDGES = [1, 2, 15, 16, 17, 24, 31, 32, 33, 63, 64, 65, 127, 128, 129, 255, 256, 257, 280, 288,
         289, 511, 512, 513, 536, 544, 545]


def say(*a):
    print("[gpu-test]", *a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ts.load()


def one_case(rng):
    d = int(rng.choice([64, 128]))
    H = int(rng.integers(1, 5))
    nseq = 1 if rng.random() < 0.5 else int(rng.integers(2, 6))

    def length(lo=1):
        return int(rng.choice(EDGES)) if rng.random() < 0.6 else int(rng.integers(lo, 1800))

    scale = float(np.float32(rng.choice([1 / np.sqrt(d), 1 / np.sqrt(d), 0.0, -0.3, 0.9])))
    peak = float(rng.choice([1.0, 1.0, 4.0, 8.0]))
    kind = str(rng.choice(["dense", "packed", "kv", "kv_noalloc"]))
    g = torch.Generator().manual_seed(int(rng.integers(1 << 30)))
    if kind in ("dense", "packed"):
        if kind == "dense":
            B, L = int(rng.integers(1, 4)), length()
            ls = [L] * B
        else:
            ls = [length() for _ in range(nseq)]
        T = sum(ls)
        q = (torch.randn((T, H, d), generator=g) * peak).to(torch.bfloat16)
        k = torch.randn((T, H, d), generator=g).to(torch.bfloat16)
        v = torch.randn((T, H, d), generator=g).to(torch.bfloat16)
        cu = np.concatenate([[0], np.cumsum(ls)]).astype(np.int32)
        desc = "%s ls=%s H=%d d=%d scale=%g peak=%g" % (kind, ls, H, d, scale, peak)
        say(desc)
        qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
        o = ts.ts_attn_fwd_varlen(qd, kd, vd, torch.tensor(cu, device="cuda"), max(ls), scale=scale)
        if kind == "dense":
            od = ts.ts_attn_fwd(qd.view(B, L, H, d), kd.view(B, L, H, d), vd.view(B, L, H, d),
                                scale=scale)
            torch.cuda.synchronize()
            assert torch.equal(od.view(T, H, d).view(torch.int16), o.view(torch.int16)), desc
        torch.cuda.synchronize()
        ref = ts_ref.attn_full(W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v), cu, scale)
    else:
        lq = [length() for _ in range(nseq)]
        lk = [length(0) for _ in range(nseq)]
        Tq, Tk = sum(lq), sum(lk)
        q = (torch.randn((Tq, H, d), generator=g) * peak).to(torch.bfloat16)
        k = torch.randn((Tk, H, d), generator=g).to(torch.bfloat16)
        v = torch.randn((Tk, H, d), generator=g).to(torch.bfloat16)
        cq = np.concatenate([[0], np.cumsum(lq)]).astype(np.int32)
        ck = np.concatenate([[0], np.cumsum(lk)]).astype(np.int32)
        splits = int(rng.choice([0, 0, 1, 2, 3, 7]))
        desc = "%s lq=%s lk=%s H=%d d=%d scale=%g peak=%g splits=%d" % (kind, lq, lk, H, d, scale,
                                                                        peak, splits)
        say(desc)
        args = (q.cuda(), k.cuda(), v.cuda(), torch.tensor(cq, device="cuda"),
                torch.tensor(ck, device="cuda"), max(lq), max(lk))
        o, lse = ts.ts_attn_fwd_kvcache(*args, scale=scale, return_lse=True, num_splits=splits)
        torch.cuda.synchronize()
        if kind == "kv_noalloc":
            try:
                o2, l2 = ts.ts_attn_fwd_kvcache_noalloc(*args, scale=scale, return_lse=True,
                                                        num_splits=splits)
                torch.cuda.synchronize()
                if splits != 0:  # the library's own choice may differ when the scratch is small
                    assert torch.equal(o2.view(torch.int16), o.view(torch.int16)), desc
                    assert torch.equal(l2.view(torch.int32), lse.view(torch.int32)), desc
            except ts.TsAttnError as e:
                assert e.status == ts._lib.TS_ERR_SCRATCH, desc
        ref, ref_lse = ts_ref.attn_kv_full(W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v), cq, ck,
                                           scale)
        gl = lse.cpu().numpy().astype(np.float64)
        fin = np.isfinite(ref_lse)
        assert np.array_equal(np.isfinite(gl), fin) and np.all(gl[~fin] == -np.inf), desc
        if fin.any():
            assert float(np.abs(gl[fin] - ref_lse[fin]).max()) <= 1e-2, desc
    got = o.float().cpu().numpy().astype(np.float64)
    if got.size:
        assert_rows(got, ref, desc, elementwise=False)
    return kind


@pytest.mark.parametrize("seed", [7001, 7002])
def test_random_calls_of_every_entry_point(seed):
    rng = np.random.default_rng(seed)
    kinds = [one_case(rng) for _ in range(60)]
    assert {"dense", "packed", "kv", "kv_noalloc"} <= set(kinds)
