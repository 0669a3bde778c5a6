"""Pins of the fp64 oracle against things other than itself.

The paper prints no attention values, so every pin comes from mathematics or an independent
implementation: a 50-digit mpmath brute force on tiny inputs, torch's CPU float64
scaled_dot_product_attention (a library routine the single-segment case reduces to), scipy's
softmax / logistic functions for the weights and the two-key closed form, and exact invariants
(identical keys, dominant key, one key, constant V, shift, permutation, segment independence,
convex hull, linearity).  tests/test_oracle_mutants.py plants mistakes in a copy of the oracle and
checks that these pins catch each one.
"""
import numpy as np
import pytest
import scipy.special
import torch

import workloads as W
from oracle import brute, ts_ref


def rnd(shape, seed, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


def full(q, k, v, cu, scale):
    return ts_ref.attn_full(q, k, v, np.asarray(cu, dtype=np.int32), scale)


# ------------------------------------------------------------------------------- P1 brute force

@pytest.mark.parametrize("H,d,seqlens,scale", [
    (1, 1, [1], 0.7),
    (2, 4, [3, 0, 7], 0.5),
    (2, 8, [16, 2, 1], 1.3),
    (1, 4, [0, 5, 0], -0.8),
])
def test_brute_force_mpmath(H, d, seqlens, scale):
    T = sum(seqlens)
    q, k, v = (rnd((T, H, d), s) for s in (1, 2, 3))
    cu = np.concatenate([[0], np.cumsum(seqlens)])
    got = full(q, k, v, cu, scale)
    ref = np.array(brute.attn_brute(q.tolist(), k.tolist(), v.tolist(), cu, scale), dtype=np.float64)
    assert np.max(np.abs(got - ref) / np.maximum(np.abs(ref), 1e-3)) <= 1e-13


def test_brute_force_large_scores_needs_max_subtraction():
    # scores near 2000: exp() of them overflows double, so only a max-subtracted evaluation is
    # finite; the 50-digit brute force needs no subtraction
    T, H, d = 6, 1, 4
    q, k, v = rnd((T, H, d), 4, 10.0), rnd((T, H, d), 5, 10.0), rnd((T, H, d), 6)
    scale = 5.0
    got = full(q, k, v, [0, T], scale)
    ref = np.array(brute.attn_brute(q.tolist(), k.tolist(), v.tolist(), [0, T], scale), dtype=np.float64)
    assert np.all(np.isfinite(got))
    assert np.max(np.abs(got - ref)) <= 1e-12


def test_bf16_inputs_widen_exactly():
    w = W.Workload("x", (37, 90), 2, 64, 3)
    q, k, v = W.make_inputs(w)
    a = ts_ref.attn_full(W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v), w.cu_seqlens, w.scale)
    b = ts_ref.attn_full(q.double().numpy(), k.double().numpy(), v.double().numpy(), w.cu_seqlens,
                         w.scale)
    assert np.array_equal(a, b)
    # brute force on a few bf16 rows too
    ref = brute.attn_brute(q.double()[:37].tolist(), k.double()[:37].tolist(),
                           v.double()[:37].tolist(), [0, 37], w.scale)
    assert np.max(np.abs(a[:37] - np.array(ref, dtype=np.float64))) <= 1e-13


# ------------------------------------------------------------------ P2 library routine (SDPA)

def sdpa_segments(q, k, v, seqlens, scale):
    out, start = [], 0
    for L in seqlens:
        if L == 0:
            continue
        # [T, H, d] -> [H, L, d]
        qs, ks, vs = (torch.from_numpy(x[start:start + L]).permute(1, 0, 2).contiguous() for x in (q, k, v))
        o = torch.nn.functional.scaled_dot_product_attention(qs, ks, vs, scale=scale)
        out.append(o.permute(1, 0, 2).numpy())
        start += L
    return np.concatenate(out, axis=0)


@pytest.mark.parametrize("seqlens,H,d", [([1024], 2, 64), ([300, 0, 700, 48], 3, 128), ([2048], 1, 32)])
def test_matches_torch_sdpa_float64(seqlens, H, d):
    T = sum(seqlens)
    q, k, v = rnd((T, H, d), 11), rnd((T, H, d), 12), rnd((T, H, d), 13)
    scale = 1.0 / np.sqrt(d)
    got = full(q, k, v, np.concatenate([[0], np.cumsum(seqlens)]), scale)
    ref = sdpa_segments(q, k, v, seqlens, scale)
    assert np.max(np.abs(got - ref)) <= 1e-12


def test_tiny_workload_matches_sdpa_on_bf16_values():
    w = W.WORKLOADS["tiny"]
    q, k, v = W.make_inputs(w)
    got = ts_ref.attn_full(W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v), w.cu_seqlens, w.scale)
    ref = sdpa_segments(q.double().numpy(), k.double().numpy(), v.double().numpy(), [w.T], w.scale)
    assert np.max(np.abs(got - ref)) <= 1e-12


# -------------------------------------------------------------------------- P3 weights (softmax)

def test_weights_are_softmax_and_sum_to_one():
    T, H, d = 50, 2, 16
    q, k, v = rnd((T, H, d), 21), rnd((T, H, d), 22), rnd((T, H, d), 23)
    cu = np.array([0, 20, 50], dtype=np.int32)
    scale = 0.3
    for t, h in [(0, 0), (19, 1), (20, 0), (49, 1)]:
        w, out = ts_ref.attn_weights(q, k, v, cu, scale, t, h)
        lo, hi = (0, 20) if t < 20 else (20, 50)
        z = scale * (k[lo:hi, h] @ q[t, h])
        assert np.all(w >= 0)
        assert abs(w.sum() - 1.0) <= 1e-14
        assert np.max(np.abs(w - scipy.special.softmax(z))) <= 1e-15
        assert np.max(np.abs(out - w @ v[lo:hi, h])) <= 1e-14


# ------------------------------------------------------------------------- P4-P6 closed forms

def test_identical_keys_and_zero_scale_give_mean_of_v():
    T, H, d = 40, 2, 8
    q, v = rnd((T, H, d), 31), rnd((T, H, d), 32)
    k = np.broadcast_to(rnd((1, H, d), 33), (T, H, d)).copy()
    cu = [0, 15, 40]
    mean = np.concatenate([np.broadcast_to(v[:15].mean(0), (15, H, d)),
                           np.broadcast_to(v[15:].mean(0), (25, H, d))])
    assert np.max(np.abs(full(q, k, v, cu, 0.7) - mean)) <= 1e-14
    k2 = rnd((T, H, d), 34)
    assert np.max(np.abs(full(q, k2, v, cu, 0.0) - mean)) <= 1e-14


def test_dominant_key_returns_its_value_row():
    L, H, d = 64, 1, 16
    rng = np.random.default_rng(41)
    k = rng.standard_normal((L, H, d))
    v = rng.standard_normal((L, H, d))
    jstar = 17
    q = np.broadcast_to(k[jstar] * 6.0, (L, H, d)).copy()
    scale = 1.0
    z = scale * (k[:, 0] @ q[0, 0])
    gap = z[jstar] - np.max(np.delete(z, jstar))
    assert gap >= 30
    out = full(q, k, v, [0, L], scale)
    bound = L * np.exp(-gap) * np.abs(v).max() * 2
    assert np.max(np.abs(out - v[jstar][None])) <= bound


def test_single_key_two_keys_and_constant_v():
    H, d = 2, 8
    q, k, v = rnd((3, H, d), 51), rnd((3, H, d), 52), rnd((3, H, d), 53)
    cu = [0, 1, 3]  # a one-token segment and a two-token segment
    out = full(q, k, v, cu, 0.9)
    assert np.array_equal(out[0], v[0])  # one key: O = V exactly
    for t in (1, 2):
        for h in range(H):
            z1 = 0.9 * q[t, h] @ k[1, h]
            z2 = 0.9 * q[t, h] @ k[2, h]
            two = scipy.special.expit(z1 - z2) * v[1, h] + scipy.special.expit(z2 - z1) * v[2, h]
            assert np.max(np.abs(out[t, h] - two)) <= 1e-15
    vc = np.full((3, H, d), -1.25)
    assert np.max(np.abs(full(q, k, vc, cu, 0.9) + 1.25)) <= 1e-15


# ----------------------------------------------------------------------------- P7-P10 invariants

def test_shift_of_keys_by_a_per_channel_offset_is_invisible():
    T, H, d = 70, 2, 16
    q, k, v = rnd((T, H, d), 61), rnd((T, H, d), 62), rnd((T, H, d), 63)
    b = rnd((1, H, d), 64, 2.0)
    cu = [0, 30, 70]
    assert np.max(np.abs(full(q, k, v, cu, 0.4) - full(q, k + b, v, cu, 0.4))) <= 1e-12


def test_permutations():
    T, H, d = 45, 2, 8
    q, k, v = rnd((T, H, d), 71), rnd((T, H, d), 72), rnd((T, H, d), 73)
    cu = [0, 45]
    base = full(q, k, v, cu, 0.5)
    p = np.random.default_rng(74).permutation(T)
    assert np.max(np.abs(full(q[p], k, v, cu, 0.5) - base[p])) <= 1e-13
    assert np.max(np.abs(full(q, k[p], v[p], cu, 0.5) - base)) <= 1e-13


def test_segment_independence():
    seqlens = [13, 0, 29, 8]
    T, H, d = sum(seqlens), 2, 8
    q, k, v = rnd((T, H, d), 81), rnd((T, H, d), 82), rnd((T, H, d), 83)
    cu = np.concatenate([[0], np.cumsum(seqlens)])
    base = full(q, k, v, cu, 0.6)
    parts = [full(q[a:b], k[a:b], v[a:b], [0, b - a], 0.6) for a, b in zip(cu[:-1], cu[1:]) if b > a]
    assert np.array_equal(base, np.concatenate(parts))
    q2, k2, v2 = q.copy(), k.copy(), v.copy()
    q2[:13] *= -3
    k2[:13] += 1
    v2[:13] = 0
    other = full(q2, k2, v2, cu, 0.6)
    assert np.array_equal(other[13:], base[13:])


def test_convex_hull_and_linearity_in_v():
    T, H, d = 60, 3, 8
    q, k, v = rnd((T, H, d), 91), rnd((T, H, d), 92), rnd((T, H, d), 93)
    v2 = rnd((T, H, d), 94)
    cu = [0, 25, 60]
    out = full(q, k, v, cu, 0.5)
    for lo, hi in ((0, 25), (25, 60)):
        assert np.all(out[lo:hi] <= v[lo:hi].max(axis=0) + 1e-15)
        assert np.all(out[lo:hi] >= v[lo:hi].min(axis=0) - 1e-15)
    lin = full(q, k, 2.0 * v - 3.0 * v2, cu, 0.5)
    assert np.max(np.abs(lin - (2.0 * out - 3.0 * full(q, k, v2, cu, 0.5)))) <= 1e-13


# ------------------------------------------------------------------------------ argument checks

def test_rejects_bad_segments_and_rows():
    q = rnd((4, 1, 2), 1)
    with pytest.raises(RuntimeError):
        ts_ref.attn_full(q, q, q, np.array([0, 3, 2, 4], dtype=np.int32), 1.0)
    with pytest.raises(ValueError):
        ts_ref.attn_full(q, q, q, np.array([0, 3], dtype=np.int32), 1.0)
    with pytest.raises(RuntimeError):
        ts_ref.attn_rows(q, q, q, [0, 4], 1.0, [4], [0])
