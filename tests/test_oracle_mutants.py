"""Plants plausible mistakes in a copy of the oracle's C source and checks that the pins catch each.

Each mutant is one textual edit of oracle/ts_ref.c (a dropped term, a wrong sign or index, a
swapped operand, an off-by-one), compiled on the CPU into a temporary library.  The same checks the
pin suite uses -- mpmath brute force, torch float64 SDPA, closed forms -- must fail on every mutant
and pass on the unmodified source.  The product oracle itself carries no mutation hooks.
"""
import ctypes
import os
import subprocess

import numpy as np
import pytest
import torch

from oracle import brute
from oracle import build as obuild

SRC = open(obuild.SRC).read()

MUTANTS = {
    "no_max_subtraction": ("double w = exp(z[j - j0] - m);", "double w = exp(z[j - j0]);"),
    "max_added": ("double w = exp(z[j - j0] - m);", "double w = exp(z[j - j0] + m);"),
    "scale_dropped": ("double zj = scale * dot;", "double zj = dot;"),
    "k_head_ignored": ("int64_t koff = j * row_stride + (int64_t)h * d;", "int64_t koff = j * row_stride;"),
    "q_k_swapped_rows": ("dot += elem(q, qoff + c) * elem(k, koff + c);",
                         "dot += elem(q, koff + c) * elem(k, qoff + c);"),
    "last_key_dropped": ("int64_t j0 = cu[s], j1 = cu[s + 1];", "int64_t j0 = cu[s], j1 = cu[s + 1] - 1;"),
    "no_normalisation": ("for (int32_t c = 0; c < d; c++) out[c] /= den;", ""),
    "v_row_is_query": ("int64_t voff = j * row_stride + (int64_t)h * d;",
                       "int64_t voff = t * row_stride + (int64_t)h * d;"),
    "segment_search_strict": ("if ((int64_t)cu[mid] <= t) lo = mid; else hi = mid;",
                              "if ((int64_t)cu[mid] < t) lo = mid; else hi = mid;"),
    "first_key_skipped": ("for (int64_t j = j0; j < j1; j++) {\n    int64_t koff",
                          "for (int64_t j = j0 + 1; j < j1; j++) {\n    int64_t koff"),
}


def compile_variant(tmp_path, name, src_text):
    c = tmp_path / (name + ".c")
    so = tmp_path / (name + ".so")
    c.write_text(src_text)
    obuild.build(str(c), str(so))
    lib = ctypes.CDLL(str(so))
    p, i32, i64, f64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double
    lib.ts_ref_attn_rows_f64.argtypes = [p, p, p, p, i32, i32, i32, f64, p, p, i64, p]
    lib.ts_ref_attn_rows_f64.restype = ctypes.c_int
    return lib


def run(lib, q, k, v, cu, scale):
    T, H, d = q.shape
    tt, hh = np.meshgrid(np.arange(T, dtype=np.int64), np.arange(H, dtype=np.int32), indexing="ij")
    tt, hh = tt.ravel().copy(), hh.ravel().copy()
    out = np.empty((T * H, d))
    cu = np.asarray(cu, dtype=np.int32)
    P = lambda a: ctypes.c_void_p(a.ctypes.data)  # noqa: E731
    rc = lib.ts_ref_attn_rows_f64(P(q), P(k), P(v), P(cu), cu.size - 1, H, d, float(scale),
                                  P(tt), P(hh), tt.size, P(out))
    if rc:
        return None
    return out.reshape(T, H, d)


def pins_pass(lib):
    """The pin checks, condensed; True only if every one holds."""
    rng = np.random.default_rng(5)
    # brute force, three segments incl. an empty one, scale != 1, two heads
    seqlens, H, d = [3, 0, 7, 2], 2, 4
    T = sum(seqlens)
    q, k, v = (rng.standard_normal((T, H, d)) for _ in range(3))
    cu = np.concatenate([[0], np.cumsum(seqlens)])
    got = run(lib, q, k, v, cu, 0.7)
    ref = np.array(brute.attn_brute(q.tolist(), k.tolist(), v.tolist(), cu, 0.7), dtype=np.float64)
    if got is None or not np.all(np.isfinite(got)) or np.max(np.abs(got - ref)) > 1e-12:
        return False
    # large scores: only a max-subtracted evaluation stays finite
    qb, kb = rng.standard_normal((6, 1, 4)) * 10, rng.standard_normal((6, 1, 4)) * 10
    vb = rng.standard_normal((6, 1, 4))
    got = run(lib, qb, kb, vb, [0, 6], 5.0)
    ref = np.array(brute.attn_brute(qb.tolist(), kb.tolist(), vb.tolist(), [0, 6], 5.0), dtype=np.float64)
    if got is None or not np.all(np.isfinite(got)) or np.max(np.abs(got - ref)) > 1e-12:
        return False
    # library routine: torch float64 SDPA on one segment
    L, H, d = 200, 2, 16
    q, k, v = (rng.standard_normal((L, H, d)) for _ in range(3))
    got = run(lib, q, k, v, [0, L], 0.25)
    t = [torch.from_numpy(x).permute(1, 0, 2).contiguous() for x in (q, k, v)]
    ref = torch.nn.functional.scaled_dot_product_attention(*t, scale=0.25).permute(1, 0, 2).numpy()
    if got is None or np.max(np.abs(got - ref)) > 1e-12:
        return False
    return True


def test_unmodified_oracle_passes(tmp_path):
    assert pins_pass(compile_variant(tmp_path, "orig", SRC))


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(tmp_path, name):
    old, new = MUTANTS[name]
    assert SRC.count(old) == 1, "mutation anchor not found once: %s" % name
    lib = compile_variant(tmp_path, name, SRC.replace(old, new))
    assert not pins_pass(lib), "pins missed mutant %s" % name
