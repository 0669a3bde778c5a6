"""Writes tests/golden/closed_forms.json: small attention cases whose exact answer follows from a
closed form, not from any implementation.

The paper prints no attention values to copy, so the fixtures are worked examples of the
definition (segment-local non-causal softmax attention of the coalesced chunk batch, Sec. 3.1 and
Sec. 6.1) in the special cases where the answer has a closed form:
  * all scores of a segment equal  -> O is the segment mean of V (exact rational, via fractions);
  * a one-token segment            -> O = V;
  * a two-key segment              -> O = sigmoid(z1 - z2) V1 + sigmoid(z2 - z1) V2, with the
                                      logistic function evaluated by mpmath at 40 digits.
Every input is a small dyadic number, exact in bfloat16, so the same values feed the oracle and
the GPU kernel.  Run: python tests/golden/make_golden.py
"""
import json
import os
from fractions import Fraction

import mpmath

HERE = os.path.dirname(os.path.abspath(__file__))


def mean_case():
    # two segments [2, 4], H=2, d=4.  In each (segment, head) every key is the same vector or
    # differs from it only in channels where q is zero, so all scores of the row are equal.
    seqlens, H, d = [2, 4], 2, 4
    T = sum(seqlens)
    q = [[[1.0, 0.0, -0.5, 0.0], [0.0, 2.0, 0.0, 0.25]] for _ in range(T)]
    q[3][0] = [0.5, 0.0, 1.5, 0.0]
    q[4][1] = [0.0, -1.0, 0.0, 3.0]
    k = []
    for t in range(T):
        # head 0: channels 1 and 3 vary (q is zero there); head 1: channels 0 and 2 vary
        a = (t % 3) * 0.5
        k.append([[0.75, a, 1.25, -a], [a - 1.0, -0.5, 2.0 * a, 0.125]])
    v = [[[float(t + h), float(-t) * 0.5, 0.25 * h, float(t * t) * 0.125] for h in range(H)]
         for t in range(T)]
    exp = [[[None] * d for _ in range(H)] for _ in range(T)]
    start = 0
    for L in seqlens:
        for h in range(H):
            for c in range(d):
                m = sum(Fraction(v[j][h][c]) for j in range(start, start + L)) / L
                assert Fraction(float(m)) == m  # dyadic mean: exact as a double
                for t in range(start, start + L):
                    exp[t][h][c] = str(float(m))
        start += L
    # q_t . k_j is the same for all j of a segment: head 0 uses channels 0 and 2 of k (constant);
    # for the rows edited above the product with the constant channels is still j-independent.
    return {"name": "equal_scores_mean_of_v", "seqlens": seqlens, "H": H, "d": d, "scale": 0.5,
            "closed_form": "all scores of a row equal -> O = mean of V over the segment",
            "q": q, "k": k, "v": v, "expected": exp}


def single_token_case():
    seqlens, H, d = [1, 1, 1], 1, 4
    q = [[[1.0, -2.0, 0.5, 4.0]], [[0.0, 0.0, 0.0, 0.0]], [[-8.0, 1.0, 2.0, 0.25]]]
    k = [[[3.0, 0.5, -1.0, 2.0]], [[1.0, 1.0, 1.0, 1.0]], [[0.125, 0.0, -4.0, 1.0]]]
    v = [[[0.5, -0.75, 1.0, 6.0]], [[-3.0, 2.0, 0.0, 0.5]], [[1.5, 1.5, -1.5, -0.125]]]
    exp = [[[str(x) for x in row[0]]] for row in v]
    return {"name": "one_token_segments", "seqlens": seqlens, "H": H, "d": d, "scale": 1.0,
            "closed_form": "a segment of one token attends only to itself -> O = V",
            "q": q, "k": k, "v": v, "expected": exp}


def two_key_case():
    seqlens, H, d = [2], 1, 4
    q = [[[1.0, 0.0, 0.5, 0.0]], [[0.0, 2.0, 0.0, -1.0]]]
    k = [[[0.5, 1.0, -0.25, 2.0]], [[-0.25, 0.5, 1.0, 0.0]]]
    v = [[[1.0, -2.0, 0.5, 3.0]], [[-1.0, 4.0, 2.0, 0.0]]]
    scale = 0.75
    mpmath.mp.dps = 40
    exp = []
    for t in range(2):
        z = [mpmath.mpf(scale) * mpmath.fsum(mpmath.mpf(q[t][0][c]) * mpmath.mpf(k[j][0][c])
                                             for c in range(d)) for j in range(2)]
        s1 = 1 / (1 + mpmath.exp(-(z[0] - z[1])))  # logistic(z1 - z2)
        s2 = 1 / (1 + mpmath.exp(-(z[1] - z[0])))
        exp.append([[mpmath.nstr(s1 * v[0][0][c] + s2 * v[1][0][c], 30) for c in range(d)]])
    return {"name": "two_keys_logistic", "seqlens": seqlens, "H": H, "d": d, "scale": scale,
            "closed_form": "two keys -> O = sigmoid(z1 - z2) V1 + sigmoid(z2 - z1) V2",
            "q": q, "k": k, "v": v, "expected": exp}


def main():
    cases = [mean_case(), single_token_case(), two_key_case()]
    doc = {"about": "Closed-form attention cases (see make_golden.py); inputs exact in bf16.",
           "cases": cases}
    with open(os.path.join(HERE, "closed_forms.json"), "w") as f:
        json.dump(doc, f, indent=1)


if __name__ == "__main__":
    main()
