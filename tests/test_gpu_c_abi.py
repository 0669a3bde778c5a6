"""The C ABI from a plain C program (tests/c_abi/caller.c: HIP runtime calls and include/ts_attn.h,
no C++ and no PyTorch), on the GPU: its results against the fp64 oracle, and bitwise equal to the
same call made through the Python binding (which only marshals arguments)."""
import importlib.util
import os
import subprocess
import sys

import numpy as np
import pytest
import torch

import workloads as W
from metrics import assert_parity
from oracle import ts_ref

pytestmark = pytest.mark.gpu

ts = pytest.importorskip("paper_2606_19271_amd")

HERE = os.path.dirname(os.path.abspath(__file__))
_spec = importlib.util.spec_from_file_location("c_abi_build", os.path.join(HERE, "c_abi", "build.py"))
c_abi_build = importlib.util.module_from_spec(_spec)
_spec.loader.exec_module(c_abi_build)

LSE_ABS = 1e-2  # as in test_gpu_kvcache.py


def say(*a):
    print("[gpu-test]", *a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def caller():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ts.load()
    if not os.path.exists(c_abi_build.EXE):
        c_abi_build.build()
    return c_abi_build.EXE


def run_caller(path, tmp_path, mode, cu_q, cu_k, H, d, q, k, v, scale, num_splits=0):
    nseq = len(cu_q) - 1
    lq = np.diff(cu_q)
    lk = np.diff(cu_k)
    hdr = np.array([mode, nseq, H, d, int(cu_q[-1]), int(cu_k[-1]), int(lq.max()), int(lk.max()),
                    num_splits], dtype="<i4")
    fin, fout = str(tmp_path / "in.bin"), str(tmp_path / "out.bin")
    with open(fin, "wb") as f:
        f.write(hdr.tobytes())
        f.write(np.array([scale], dtype="<f4").tobytes())
        f.write(np.asarray(cu_q, dtype="<i4").tobytes())
        f.write(np.asarray(cu_k, dtype="<i4").tobytes())
        for t in (q, k, v):
            f.write(W.bf16_bits(t).astype("<u2").tobytes())
    say("c caller mode", mode, "nseq", nseq, "H", H, "d", d, "splits", num_splits)
    r = subprocess.run([path, fin, fout], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    raw = open(fout, "rb").read()
    n = int(cu_q[-1]) * H * d
    o_bits = np.frombuffer(raw[:2 * n], dtype="<u2").reshape(int(cu_q[-1]), H, d)
    lse = None
    if mode == 1:
        lse = np.frombuffer(raw[2 * n:], dtype="<f4").reshape(int(cu_q[-1]), H)
    return o_bits, lse


def bits_to_f64(bits):
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def torch_bits(t):
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def test_packed_call_from_c(caller, tmp_path):
    seqlens = [300, 0, 517, 64]
    w = W.Workload("c_abi", tuple(seqlens), 3, 128, 71)
    q, k, v = W.make_inputs(w)
    cu = w.cu_seqlens
    o_bits, _ = run_caller(caller, tmp_path, 0, cu, cu, 3, 128, q, k, v, w.scale)
    ref = ts_ref.attn_full(W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v), cu, w.scale)
    assert_parity(bits_to_f64(o_bits), ref, "packed call from C")
    o_py = ts.ts_attn_fwd_varlen(q.cuda(), k.cuda(), v.cuda(), torch.tensor(cu, device="cuda"),
                                 max(seqlens))
    torch.cuda.synchronize()
    assert np.array_equal(o_bits, torch_bits(o_py)), "C and Python callers differ"


def test_dense_call_from_c(caller, tmp_path):
    B, L, H, d = 2, 333, 2, 64
    w = W.Workload("c_abi", (L,) * B, H, d, 72)
    q, k, v = W.make_inputs(w)
    scale = float(np.float32(0.7))
    o_bits, _ = run_caller(caller, tmp_path, 2, w.cu_seqlens, w.cu_seqlens, H, d, q, k, v, scale)
    ref = ts_ref.attn_full(W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v), w.cu_seqlens, scale)
    assert_parity(bits_to_f64(o_bits), ref, "dense call from C")
    o_py = ts.ts_attn_fwd(q.cuda().view(B, L, H, d), k.cuda().view(B, L, H, d),
                          v.cuda().view(B, L, H, d), scale=scale)
    torch.cuda.synchronize()
    assert np.array_equal(o_bits, torch_bits(o_py).reshape(B * L, H, d)), "C and Python callers differ"


@pytest.mark.parametrize("splits", [0, 3])
def test_kvcache_call_from_c(caller, tmp_path, splits):
    lq, lk = [100, 0, 257, 1], [700, 50, 1000, 1]
    w = W.KvWorkload("c_abi", tuple(lq), tuple(lk), 2, 64, 73, True)
    q, k, v = W.make_kv_inputs(w)
    o_bits, lse = run_caller(caller, tmp_path, 1, w.cu_q, w.cu_k, 2, 64, q, k, v, w.scale, splits)
    ro, rlse = ts_ref.attn_kv_full(W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v), w.cu_q, w.cu_k,
                                   w.scale)
    assert_parity(bits_to_f64(o_bits), ro, "kv call from C, splits=%d" % splits)
    fin = np.isfinite(rlse)
    assert np.array_equal(np.isfinite(lse), fin)
    assert float(np.max(np.abs(lse[fin] - rlse[fin]))) <= LSE_ABS
    o_py, lse_py = ts.ts_attn_fwd_kvcache(q.cuda(), k.cuda(), v.cuda(), torch.tensor(w.cu_q, device="cuda"),
                                          torch.tensor(w.cu_k, device="cuda"), w.max_q, w.max_k,
                                          return_lse=True, num_splits=splits)
    torch.cuda.synchronize()
    assert np.array_equal(o_bits, torch_bits(o_py)), "C and Python callers differ"
    assert np.array_equal(lse.view(np.uint32), lse_py.cpu().numpy().view(np.uint32))
