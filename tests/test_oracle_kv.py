"""Pins of the oracle's chunk-vs-cache attention (ts_ref_attn_kv_rows_*) with its log-sum-exp.

Segment s has its queries at rows cu_q[s]:cu_q[s+1] of q and its keys and values at rows
cu_k[s]:cu_k[s+1] of k and v; every query attends to every key of its segment (the chunk step of
a chunk-autoregressive model against the session's cached state, paper Sec. 2 and Sec. 6.1).
Nothing here compares the oracle with itself: the pins are a 50-digit mpmath brute force, torch's
CPU float64 scaled_dot_product_attention (which accepts Lq != Lk), scipy's logsumexp over numpy
scores, closed forms (one key, no key), and the merge identity -- attention over keys A followed
by keys B equals the lse-weighted combination of attention over A and over B -- which is what the
split-key path of the GPU library relies on.  The planted-mistake check at the end runs the same
pins on textual mutants of the C source.
"""
import ctypes

import numpy as np
import pytest
import scipy.special
import torch

from oracle import brute, ts_ref
from oracle import build as obuild


def rnd(shape, seed, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


def cu_of(lens):
    return np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)


def make(lq, lk, H, d, seed, qscale=1.0):
    q = rnd((sum(lq), H, d), seed, qscale)
    k = rnd((sum(lk), H, d), seed + 1)
    v = rnd((sum(lk), H, d), seed + 2)
    return q, k, v, cu_of(lq), cu_of(lk)


# ------------------------------------------------------------------------------ brute force

@pytest.mark.parametrize("lq,lk,H,d,scale", [
    ([1], [1], 1, 1, 0.7),
    ([2, 3], [5, 1], 2, 4, 0.5),
    ([3, 0, 2], [0, 4, 6], 2, 4, 1.3),   # a segment with queries but no keys, one with no queries
    ([4, 1], [9, 2], 1, 8, -0.8),
])
def test_kv_brute_force_mpmath(lq, lk, H, d, scale):
    q, k, v, cq, ck = make(lq, lk, H, d, 11)
    out, lse = ts_ref.attn_kv_full(q, k, v, cq, ck, scale)
    rout, rlse = brute.attn_kv_brute(q.tolist(), k.tolist(), v.tolist(), cq, ck, scale)
    rout = np.array(rout, dtype=np.float64)
    rlse = np.array(rlse, dtype=np.float64)
    assert np.max(np.abs(out - rout) / np.maximum(np.abs(rout), 1e-3)) <= 1e-13
    fin = np.isfinite(rlse)
    assert np.array_equal(fin, np.isfinite(lse))
    assert np.all(lse[~fin] == -np.inf)
    assert np.max(np.abs(lse[fin] - rlse[fin])) <= 1e-13 * max(1.0, np.max(np.abs(rlse[fin])))


def test_kv_brute_force_large_scores():
    # scores near 1500: only a max-subtracted evaluation stays finite in double
    q, k, v, cq, ck = make([3], [7], 1, 4, 21, qscale=10.0)
    k *= 10.0
    out, lse = ts_ref.attn_kv_full(q, k, v, cq, ck, 5.0)
    rout, rlse = brute.attn_kv_brute(q.tolist(), k.tolist(), v.tolist(), cq, ck, 5.0)
    assert np.all(np.isfinite(out)) and np.all(np.isfinite(lse))
    assert np.max(np.abs(out - np.array(rout, dtype=np.float64))) <= 1e-12
    # scores reach ~1.4e3, so their double rounding alone is ~1e-13 absolute
    assert np.max(np.abs(lse - np.array(rlse, dtype=np.float64))) <= 1e-12


# ------------------------------------------------------------------------ library routines

def test_kv_matches_torch_sdpa_float64():
    lq, lk, H, d, scale = [40, 7, 64], [300, 129, 64], 3, 32, 0.2
    q, k, v, cq, ck = make(lq, lk, H, d, 31)
    out, _ = ts_ref.attn_kv_full(q, k, v, cq, ck, scale)
    for s in range(len(lq)):
        qs = torch.from_numpy(q[cq[s]:cq[s + 1]]).permute(1, 0, 2).contiguous()
        ks = torch.from_numpy(k[ck[s]:ck[s + 1]]).permute(1, 0, 2).contiguous()
        vs = torch.from_numpy(v[ck[s]:ck[s + 1]]).permute(1, 0, 2).contiguous()
        ref = torch.nn.functional.scaled_dot_product_attention(qs, ks, vs, scale=scale)
        assert np.max(np.abs(out[cq[s]:cq[s + 1]] - ref.permute(1, 0, 2).numpy())) <= 1e-12


def test_kv_lse_matches_scipy_logsumexp():
    lq, lk, H, d, scale = [17, 33], [250, 90], 2, 16, 0.35
    q, k, v, cq, ck = make(lq, lk, H, d, 41)
    _, lse = ts_ref.attn_kv_full(q, k, v, cq, ck, scale)
    for s in range(len(lq)):
        for h in range(H):
            z = scale * (q[cq[s]:cq[s + 1], h] @ k[ck[s]:ck[s + 1], h].T)
            ref = scipy.special.logsumexp(z, axis=1)
            assert np.max(np.abs(lse[cq[s]:cq[s + 1], h] - ref)) <= 1e-12


# -------------------------------------------------------------------------------- closed forms

def test_kv_one_key_and_no_key():
    q, k, v, cq, ck = make([3, 2, 4], [1, 0, 1], 2, 8, 51)
    out, lse = ts_ref.attn_kv_full(q, k, v, cq, ck, 0.9)
    # one key: O is that key's V row, lse its scaled score
    for t in range(3):
        assert np.array_equal(out[t], v[0])
        assert np.allclose(lse[t], 0.9 * np.einsum("hd,hd->h", q[t], k[0]), rtol=0, atol=1e-14)
    # no key: the empty sum
    assert np.all(out[3:5] == 0.0) and np.all(lse[3:5] == -np.inf)
    for t in range(5, 9):
        assert np.array_equal(out[t], v[1])


def test_kv_equal_segments_is_self_attention():
    lens, H, d, scale = [5, 0, 70, 33], 2, 16, 0.25
    q, k, v, cq, ck = make(lens, lens, H, d, 61)
    q = rnd(k.shape, 62)
    out, _ = ts_ref.attn_kv_full(q, k, v, cq, ck, scale)
    ref = ts_ref.attn_full(q, k, v, cq, scale)
    assert np.max(np.abs(out - ref)) <= 1e-14


def test_kv_bf16_inputs_widen_exactly():
    q, k, v, cq, ck = make([20, 11], [70, 5], 2, 64, 71)
    tq, tk, tv = (torch.from_numpy(x).to(torch.bfloat16) for x in (q, k, v))
    bits = [t.view(torch.int16).numpy().view(np.uint16) for t in (tq, tk, tv)]
    wide = [t.double().numpy() for t in (tq, tk, tv)]
    a = ts_ref.attn_kv_full(*bits, cq, ck, 0.125)
    b = ts_ref.attn_kv_full(*wide, cq, ck, 0.125)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


# ---------------------------------------------------------------------------------- merge identity

def merge(parts):
    """Combine (out, lse) of disjoint key ranges of the same queries into the whole range."""
    lses = np.stack([p[1] for p in parts])
    lse = np.logaddexp.reduce(lses, axis=0)
    out = sum(np.exp(p[1] - lse)[..., None] * p[0] for p in parts)
    return out, lse


def test_kv_merge_of_two_key_ranges():
    # each segment's keys split at an arbitrary point (empty parts included) reproduce the whole
    lq, lk, H, d, scale = [9, 4, 6], [40, 3, 25], 2, 8, 0.6
    q, k, v, cq, ck = make(lq, lk, H, d, 81)
    whole = ts_ref.attn_kv_full(q, k, v, cq, ck, scale)
    cut = [17, 0, 25]  # keys [0, cut) of segment s in part A, the rest in part B
    ia = np.concatenate([np.arange(ck[s], ck[s] + cut[s]) for s in range(3)])
    ib = np.concatenate([np.arange(ck[s] + cut[s], ck[s + 1]) for s in range(3)])
    ca = cu_of(cut)
    cb = cu_of([lk[s] - cut[s] for s in range(3)])
    pa = ts_ref.attn_kv_full(q, k[ia], v[ia], cq, ca, scale)
    pb = ts_ref.attn_kv_full(q, k[ib], v[ib], cq, cb, scale)
    out, lse = merge([pa, pb])
    assert np.max(np.abs(out - whole[0])) <= 1e-13
    assert np.max(np.abs(lse - whole[1])) <= 1e-13


# --------------------------------------------------------------------------- planted mistakes

SRC = open(obuild.SRC).read()

KV_MUTANTS = {
    "keys_from_query_offsets": ("int64_t kb = cu_k[s], ke = cu_k[s + 1];",
                                "int64_t kb = cu_q[s], ke = cu_q[s + 1];"),
    "segment_of_query_from_key_offsets": ("int32_t s = find_segment(cu_q, nseq, t);",
                                          "int32_t s = find_segment(cu_k, nseq, t);"),
    "lse_without_max": ("*lse = m + log(den);", "*lse = log(den);"),
    "lse_base_two": ("*lse = m + log(den);", "*lse = m + log2(den);"),
    "no_max_subtraction": ("double w = exp(z[j - kb] - m);", "double w = exp(z[j - kb]);"),
    "scale_dropped": ("z[j - kb] = scale * dot;", "z[j - kb] = dot;"),
    "empty_lse_zero": ("*lse = -INFINITY;", "*lse = 0.0;"),
    "v_rows_from_tensor_start": ("int64_t vrow = j * row_stride + (int64_t)h * d;",
                                 "int64_t vrow = (j - kb) * row_stride + (int64_t)h * d;"),
    "query_head_ignored": ("int64_t qrow = t * row_stride + (int64_t)h * d;",
                           "int64_t qrow = t * row_stride;"),
    "no_normalisation": ("for (int32_t c = 0; c < d; c++) out[c] = out[c] / den;", ""),
}


def compile_variant(tmp_path, name, text):
    c = tmp_path / (name + ".c")
    so = tmp_path / (name + ".so")
    c.write_text(text)
    obuild.build(str(c), str(so))
    lib = ctypes.CDLL(str(so))
    p, i32, i64, f64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double
    lib.ts_ref_attn_kv_rows_f64.argtypes = [p, p, p, p, p, i32, i32, i32, f64, p, p, i64, p, p]
    lib.ts_ref_attn_kv_rows_f64.restype = ctypes.c_int
    return lib


def run(lib, q, k, v, cq, ck, scale):
    Tq, H, d = q.shape
    tt, hh = np.meshgrid(np.arange(Tq, dtype=np.int64), np.arange(H, dtype=np.int32), indexing="ij")
    tt, hh = tt.ravel().copy(), hh.ravel().copy()
    out, lse = np.empty((Tq * H, d)), np.empty(Tq * H)
    P = lambda a: ctypes.c_void_p(a.ctypes.data)  # noqa: E731
    rc = lib.ts_ref_attn_kv_rows_f64(P(q), P(k), P(v), P(cq), P(ck), cq.size - 1, H, d,
                                     float(scale), P(tt), P(hh), tt.size, P(out), P(lse))
    return None if rc else (out.reshape(Tq, H, d), lse.reshape(Tq, H))


def pins_pass(lib):
    """The pins above, condensed; True only if every one holds."""
    # brute force with separate offsets, a segment without keys and two heads
    q, k, v, cq, ck = make([3, 2, 2], [5, 0, 3], 2, 4, 91)
    got = run(lib, q, k, v, cq, ck, 0.7)
    rout, rlse = brute.attn_kv_brute(q.tolist(), k.tolist(), v.tolist(), cq, ck, 0.7)
    rout, rlse = np.array(rout, dtype=np.float64), np.array(rlse, dtype=np.float64)
    if got is None or not np.all(np.isfinite(got[0])):
        return False
    fin = np.isfinite(rlse)
    if np.max(np.abs(got[0] - rout)) > 1e-12 or not np.array_equal(np.isfinite(got[1]), fin):
        return False
    if np.any(got[1][~fin] != -np.inf) or np.max(np.abs(got[1][fin] - rlse[fin])) > 1e-12:
        return False
    # large scores: finite only with the max subtracted
    q, k, v, cq, ck = make([2], [6], 1, 4, 92, qscale=10.0)
    k *= 10.0
    got = run(lib, q, k, v, cq, ck, 5.0)
    rout, rlse = brute.attn_kv_brute(q.tolist(), k.tolist(), v.tolist(), cq, ck, 5.0)
    if got is None or not np.all(np.isfinite(got[0])) or not np.all(np.isfinite(got[1])):
        return False
    if np.max(np.abs(got[0] - np.array(rout, dtype=np.float64))) > 1e-12:
        return False
    if np.max(np.abs(got[1] - np.array(rlse, dtype=np.float64))) > 1e-9:
        return False
    return True


def test_unmodified_kv_oracle_passes(tmp_path):
    assert pins_pass(compile_variant(tmp_path, "orig", SRC))


@pytest.mark.parametrize("name", sorted(KV_MUTANTS))
def test_kv_mutant_is_caught(tmp_path, name):
    old, new = KV_MUTANTS[name]
    assert SRC.count(old) == 1, "mutation anchor not found once: %s" % name
    lib = compile_variant(tmp_path, name, SRC.replace(old, new))
    assert not pins_pass(lib), "pins missed mutant %s" % name
