"""Brute-force attention in 50-digit mpmath arithmetic, for tiny inputs only.

Test infrastructure only.  It evaluates the same definition as ts_ref.c -- segment-local,
non-causal softmax(scale * Q K^T) V, one (token, head) row at a time -- with no max subtraction
(exact high-precision exp needs none), so it pins the C oracle's rounding and its
max-subtraction step independently.
"""
import mpmath


def attn_brute(q, k, v, cu_seqlens, scale, dps=50):
    """q, k, v: nested sequences [T][H][d] of numbers; returns nested lists [T][H][d] of mpf."""
    with mpmath.workdps(dps):
        T, H, d = len(q), len(q[0]), len(q[0][0])
        sc = mpmath.mpf(scale)
        out = [[[None] * d for _ in range(H)] for _ in range(T)]
        cu = [int(c) for c in cu_seqlens]
        for s in range(len(cu) - 1):
            lo, hi = cu[s], cu[s + 1]
            for t in range(lo, hi):
                for h in range(H):
                    w = []
                    for j in range(lo, hi):
                        dot = mpmath.fsum(mpmath.mpf(q[t][h][c]) * mpmath.mpf(k[j][h][c]) for c in range(d))
                        w.append(mpmath.exp(sc * dot))
                    den = mpmath.fsum(w)
                    for c in range(d):
                        out[t][h][c] = mpmath.fsum(w[j - lo] * mpmath.mpf(v[j][h][c]) for j in range(lo, hi)) / den
        return out
