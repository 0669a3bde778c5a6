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


def attn_kv_brute(q, k, v, cu_q, cu_k, scale, dps=50):
    """Chunk queries against per-segment key ranges: q [Tq][H][d], k, v [Tk][H][d] nested
    sequences; segment s has queries cu_q[s]:cu_q[s+1] and keys cu_k[s]:cu_k[s+1].  Returns
    (out [Tq][H][d], lse [Tq][H]) as mpf, lse = log sum_j exp(scale * <q, k_j>) (-inf and a zero
    row for a segment without keys)."""
    with mpmath.workdps(dps):
        Tq, H, d = len(q), len(q[0]), len(q[0][0])
        sc = mpmath.mpf(scale)
        out = [[[mpmath.mpf(0)] * d for _ in range(H)] for _ in range(Tq)]
        lse = [[mpmath.mpf("-inf")] * H for _ in range(Tq)]
        cq, ck = [int(c) for c in cu_q], [int(c) for c in cu_k]
        for s in range(len(cq) - 1):
            for t in range(cq[s], cq[s + 1]):
                for h in range(H):
                    keys = range(ck[s], ck[s + 1])
                    if len(keys) == 0:
                        continue
                    w = [mpmath.exp(sc * mpmath.fsum(mpmath.mpf(q[t][h][c]) * mpmath.mpf(k[j][h][c])
                                                     for c in range(d))) for j in keys]
                    den = mpmath.fsum(w)
                    lse[t][h] = mpmath.log(den)
                    for c in range(d):
                        out[t][h][c] = mpmath.fsum(wj * mpmath.mpf(v[j][h][c]) for wj, j in zip(w, keys)) / den
        return out, lse
