"""The parity bars themselves (tests/metrics.py), on the CPU: bf16 spacing and rounding against
their definitions, and that the per-row bars reject a wrong result confined to one row or one
element while the correctly rounded result passes them."""
import numpy as np
import torch

import metrics as M


def test_ulp_bf16_is_the_bf16_spacing():
    x = np.array([1.0, 1.5, 0.75, 3.9, -2.0, 1e-3, 0.0])
    # bf16 keeps 8 significant bits: spacing 2^(e - 7) in [2^e, 2^(e+1))
    want = np.array([2.0 ** -7, 2.0 ** -7, 2.0 ** -8, 2.0 ** -6, 2.0 ** -6, 2.0 ** -17, 0.0])
    assert np.array_equal(M.ulp_bf16(x), want)
    # the next bf16 above 1 + ulp / 2 (a tie, to even) and the largest below 2
    b = torch.tensor([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, 2.0 - 2.0 ** -7], dtype=torch.float64)
    assert np.array_equal(M.bf16_of(b.numpy()), [1.0, 1.0 + 2.0 ** -6, 2.0 - 2.0 ** -7])


def test_row_bars_accept_rounding_and_reject_a_wrong_row():
    rng = np.random.default_rng(0)
    ref = rng.standard_normal((200, 64)) * 0.01
    got = M.bf16_of(ref)
    r = M.row_errors(got, ref)
    assert r["frac_correctly_rounded"] == 1.0 and r["ulp_slack_max"] <= 0.5
    assert r["row_rel_max"] < 2.0 ** -8
    M.assert_rows(got, ref)
    bad = got.copy()
    bad[17] *= 1.05                      # one row 5 % off: under every absolute gate
    assert M.errors(bad, ref)["max_abs"] < M.MAX_ABS
    assert M.row_errors(bad, ref)["row_rel_max"] > M.ROW_REL
    bad = got.copy()
    bad[3, 5] += 8 * M.ulp_bf16(ref[3, 5]) + 0.02 * np.linalg.norm(ref[3]) / 8
    assert M.row_errors(bad, ref)["ulp_slack_max"] > 1.0


def test_row_bars_on_full_outputs_and_empty_rows():
    # a full output [T, H, d] is T * H rows; a row whose exact result is zero (a query without
    # keys) passes only when the output is exactly zero there
    rng = np.random.default_rng(1)
    ref = rng.standard_normal((5, 3, 16)) * 0.1
    ref[2, 1] = 0.0
    got = M.bf16_of(ref)
    r = M.row_errors(got, ref)
    assert r["rows"] == 15 and r["ulp_slack_max"] <= 0.5 and r["row_rel_max"] < 2.0 ** -8
    got[2, 1, 3] = 1e-30
    r = M.row_errors(got, ref)
    assert r["row_rel_max"] > M.ROW_REL and r["ulp_slack_max"] > 1.0
