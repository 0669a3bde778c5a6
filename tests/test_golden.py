"""The oracle against the closed-form fixtures of tests/golden/closed_forms.json (written by
tests/golden/make_golden.py from closed forms only)."""
import json
import os

import numpy as np
import pytest

from oracle import ts_ref

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "closed_forms.json")
CASES = json.load(open(GOLDEN))["cases"]


def case_arrays(c):
    q, k, v = (np.array(c[x], dtype=np.float64) for x in ("q", "k", "v"))
    exp = np.array([[[float(x) for x in row] for row in tok] for tok in c["expected"]])
    cu = np.concatenate([[0], np.cumsum(c["seqlens"])]).astype(np.int32)
    return q, k, v, cu, exp


@pytest.mark.parametrize("c", CASES, ids=[c["name"] for c in CASES])
def test_oracle_matches_closed_form(c):
    q, k, v, cu, exp = case_arrays(c)
    got = ts_ref.attn_full(q, k, v, cu, c["scale"])
    assert np.max(np.abs(got - exp)) <= 1e-15


@pytest.mark.parametrize("c", CASES, ids=[c["name"] for c in CASES])
def test_inputs_are_exact_in_bf16(c):
    import torch
    for x in ("q", "k", "v"):
        a = torch.tensor(c[x], dtype=torch.float64)
        assert torch.equal(a.to(torch.bfloat16).double(), a)
