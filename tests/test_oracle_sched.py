"""Pins of the scheduler oracle (oracle/sched_ref.py) to what the paper and arithmetic fix:

- the App. A volatility-to-parameter table (tests/golden/app_a_volatility_levels.json): every
  tabulated volatility maps to its own level, and any window maps to the row whose tabulated
  volatility is nearest (the midpoint boundaries are exactly the nearest-row rule);
- sigma(t) against numpy's population standard deviation of the last W epochs;
- M_tar against a brute force in exact decimal arithmetic (smallest M with M K rho >= N_req);
- placement: on tiny cases with free migration, the bottleneck after every epoch equals the
  optimum of the min-max placement problem found by enumerating every feasible placement;
- hand-derived traces of Sec. 5.2.1 (assignment ties, the gain Gamma with the alpha-beta
  migration cost) and of Alg. 1 (hysteresis, proportional scale-out and scale-in, re-placement of
  the sessions of removed GPUs, pending sessions when every GPU is full, the one-epoch delay of
  the App. A parameter replacement), every expected value worked out by hand in the comments;
- invariants of the constraints of Eq. (1) on seeded random traces;
- planted mistakes (a flipped sign, a dropped term, a wrong index...) in a copy of the oracle,
  each of which must fail one of the pins above.
"""
import itertools
import json
import math
import os
import types
from fractions import Fraction

import numpy as np
import pytest

from oracle import sched_ref as SR
import workloads as W

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                      "app_a_volatility_levels.json")
TABLE = json.load(open(GOLDEN))["levels"]
VOLS = [r["volatility"] for r in TABLE]
LAT4 = [0.0, 150.0, 200.0, 260.0, 330.0]   # per-chunk latency of a GPU hosting n = 0..4 sessions


def make(mod, K=4, m_min=1, m_max=8, m_init=1, lat=LAT4, eta=1.0, alpha=0.0, beta=0.0,
         delta=0.1, window=8, bounds=(), lams=(0.2,), rhos=(0.5,)):
    return mod.SchedRef(K, m_min, m_max, m_init, list(lat), eta, alpha, beta, delta, window,
                        list(bounds), list(lams), list(rhos))


def app_a(mod, **kw):
    return make(mod, bounds=mod.level_bounds_from_table(VOLS), lams=[r["lambda"] for r in TABLE],
                rhos=[r["rho"] for r in TABLE], **kw)


def arrive(*ids, nbytes=0):
    return [(SR.ARRIVE, i, nbytes) for i in ids]


def ev(kind, *ids):
    return [(kind, i, 0) for i in ids]


def groups(s):
    """{GPU id: sorted sessions} of the current placement."""
    out = {g: [] for g, _ in s.gpu_loads()}
    for i, g in s.placement():
        if g >= 0:
            out[g].append(i)
    return out


# ---- pins, each a function of the oracle module so that planted mistakes can be run through ----

def pin_app_a_table(mod):
    rhos = [r["rho"] for r in TABLE]
    assert all(a >= b for a, b in zip(rhos, rhos[1:]))  # rho* never rises with volatility (App. A)
    s = app_a(mod)
    for r in TABLE:
        assert s.quantise(r["volatility"]) == r["level"]
    # windows of zeros with a burst: the level is the nearest tabulated volatility's
    for W_, burst, nb in itertools.product((4, 8, 16), (1, 2, 3, 5, 8, 12, 20), (1, 2, 3)):
        a = [0] * (W_ - nb) + [burst] * nb
        sigma = float(np.std(a))
        near = min(TABLE, key=lambda r: abs(r["volatility"] - sigma))
        if abs(abs(near["volatility"] - sigma) - min(abs(r["volatility"] - sigma) for r in TABLE
                                                      if r is not near)) < 1e-9:
            continue  # equidistant: on a boundary
        s = app_a(mod, window=W_, m_max=10 ** 6)
        nid = 0
        for x in a:
            s.step(arrive(*range(nid, nid + x)))
            nid += x
        assert s.level == near["level"], (W_, burst, nb, sigma)
        assert s.rho_hat == near["rho"] and s.lam == near["lambda"]


def pin_volatility_numpy(mod):
    rng = np.random.default_rng(11)
    for W_ in (1, 3, 8, 20):
        s = make(mod, window=W_, m_max=10 ** 6, bounds=[0.5, 1.5], lams=[0.1, 0.2, 0.3],
                 rhos=[0.9, 0.6, 0.3])
        hist, nid = [], 0
        for t in range(40):
            x = int(rng.integers(0, 6)) if rng.random() < 0.6 else 0
            s.step(arrive(*range(nid, nid + x)))
            nid += x
            hist.append(x)
            ref = float(np.std(hist[-W_:]))
            assert abs(s.sigma - ref) <= 1e-12 * max(1.0, ref)
            assert s.level == 1 + (ref > 0.5) + (ref > 1.5)


def pin_activations_count(mod):
    """a_t counts arrivals and activations, not departures or idle transitions."""
    s = make(mod, window=3, m_max=100)
    s.step(arrive(1, 2, 3))
    s.step(ev(SR.IDLE, 1, 2) + ev(SR.DEPART, 3))
    s.step(ev(SR.ACTIVATE, 1) + arrive(4))
    assert s.history == [3, 0, 2]
    assert abs(s.sigma - float(np.std([3, 0, 2]))) < 1e-15


def pin_target_budget(mod):
    for rho in (0.25, 0.5, 0.55, 0.6, 0.65, 0.7, 0.8, 0.88, 0.95, 1.0):
        for K in (1, 2, 3, 4, 8, 10, 12):
            s = make(mod, K=K, lat=[0.0] * (K + 1), m_min=0, m_max=10 ** 6, rhos=(rho,))
            r = Fraction(str(rho))
            for n in range(0, 301):
                m = math.ceil(Fraction(n) / (K * r))   # exact: smallest M with M K rho >= N
                assert s.target(n) == m, (rho, K, n)
    s = make(mod, K=4, m_min=2, m_max=5, rhos=(0.5,))
    assert [s.target(n) for n in (0, 1, 4, 5, 10, 11, 40)] == [2, 2, 2, 3, 5, 5, 5]


def brute_min_bottleneck(n_sessions, n_gpus, K, lat):
    best = math.inf
    for assign in itertools.product(range(n_gpus), repeat=n_sessions):
        loads = [assign.count(g) for g in range(n_gpus)]
        if max(loads, default=0) <= K:
            best = min(best, max(lat[n] for n in loads))
    return best


def pin_placement_optimal(mod):
    """Free migration (kappa = 0), fixed budget: min-max placement reaches the optimum."""
    lat = [0.0, 100.0, 170.0, 250.0]
    rng = np.random.default_rng(5)
    for M in (1, 2, 3):
        s = make(mod, K=3, m_min=M, m_max=M, m_init=M, lat=lat)
        live, idle, nid = set(), set(), 0
        for t in range(60):
            ch = []
            r = rng.random()
            if r < 0.45 and len(live) + len(idle) < 7:
                ch = arrive(nid); live.add(nid); nid += 1
            elif r < 0.65 and live:
                i = int(rng.choice(sorted(live))); live.remove(i); ch = ev(SR.DEPART, i)
            elif r < 0.85 and live:
                i = int(rng.choice(sorted(live))); live.remove(i); idle.add(i); ch = ev(SR.IDLE, i)
            elif idle:
                i = int(rng.choice(sorted(idle))); idle.remove(i); live.add(i)
                ch = ev(SR.ACTIVATE, i)
            d = s.step(ch)
            n_on = min(len(live), 3 * M)
            assert d["pending"] == len(live) - n_on
            assert d["bottleneck_ms"] == brute_min_bottleneck(n_on, M, 3, lat), (M, t)


def pin_assignment_and_gain(mod):
    """Sec. 5.2.1 by hand: K = 4, two GPUs, l = (0, 150, 200, 260, 330) ms, eta = 1,
    kappa = 1e-3 ms per byte of state."""
    s = make(mod, m_min=2, m_max=2, m_init=2, beta=1e-3)
    # 1 -> g0 (both give L = 150, equal loads, lower id); 2 -> g1 (L 150 < 200);
    # 3 -> g0 (both give 200, equal loads, lower id); 4 -> g1 (200 < 260).
    # (2,2): moving any session gives L' = max(l(1), l(3)) = 260 > 200: no move.
    d = s.step([(SR.ARRIVE, 1, 80000), (SR.ARRIVE, 2, 10000), (SR.ARRIVE, 3, 30000),
                (SR.ARRIVE, 4, 20000)])
    assert groups(s) == {0: [1, 3], 1: [2, 4]}
    assert (d["placed"], d["migrations"], d["bottleneck_ms"]) == (4, 0, 200.0)
    # (2,0): Gamma = 200 - max(l(1), l(1)) - kappa = 50 - kappa: session 1 (kappa 80) -30,
    # session 3 (kappa 30) +20 -> move 3.  Then (1,1): L' = max(l(0), l(2)) = 200 > 150: stop.
    d = s.step(ev(SR.DEPART, 2, 4))
    assert groups(s) == {0: [1], 1: [3]}
    assert (d["placed"], d["migrations"], d["bottleneck_ms"]) == (0, 1, 150.0)
    # 5 -> g0 (both 200, equal loads, lower id); 6 -> g1 (200 < 260)
    d = s.step([(SR.ARRIVE, 5, 5000), (SR.ARRIVE, 6, 5000)])
    assert groups(s) == {0: [1, 5], 1: [3, 6]}
    # 3 idles: suspended, slot freed.  (2,1): Gamma = 200 - max(l(1), l(2)) - kappa < 0.
    d = s.step(ev(SR.IDLE, 3))
    assert groups(s) == {0: [1, 5], 1: [6]} and dict(s.placement())[3] == -1
    assert (d["migrations"], d["n_req"]) == (0, 3)
    # 3 comes back: g0 would give 260, g1 gives 200 -> g1
    d = s.step(ev(SR.ACTIVATE, 3))
    assert groups(s) == {0: [1, 5], 1: [3, 6]} and d["placed"] == 1


def pin_assignment_prefers_less_loaded(mod):
    """Ties of the resulting bottleneck go to the less-loaded GPU, then the lower id.  Three GPUs,
    K = 4, migration too costly to rebalance (kappa = 1000 ms > any latency gap)."""
    s = make(mod, m_min=3, m_max=3, m_init=3, alpha=1000.0)
    # round robin: g0 = {1,4,7}, g1 = {2,5,8}, g2 = {3,6,9}
    s.step(arrive(*range(1, 10)))
    assert groups(s) == {0: [1, 4, 7], 1: [2, 5, 8], 2: [3, 6, 9]}
    s.step(ev(SR.DEPART, 5, 8, 3, 6, 9))          # (3,1,0), nothing moves
    assert groups(s) == {0: [1, 4, 7], 1: [2], 2: []}
    # 10: g0 gives 330, g1 and g2 both 260 (g0 dominates) -> the less loaded, g2
    s.step(arrive(10))
    assert groups(s) == {0: [1, 4, 7], 1: [2], 2: [10]}
    # 11: g1 and g2 tie at 260 with equal loads -> the lower id, g1
    s.step(arrive(11))
    assert groups(s) == {0: [1, 4, 7], 1: [2, 11], 2: [10]}


def pin_hysteresis_band(mod):
    """No scaling while rho_max stays in (rho_hat - delta, rho_hat + delta], even when the
    proportional target differs from M.  K = 10, rho* = 0.5, delta = 0.15: band (0.35, 0.65]."""
    lat = [0.0] + [100.0 + 20.0 * n for n in range(1, 11)]
    s = make(mod, K=10, lat=lat, m_init=2, delta=0.15)
    d = s.step(arrive(*range(1, 13)))      # (6,6): rho 0.6 in the band, although ceil(12/5) = 3
    assert (d["m"], d["m_target"], d["rho_max"]) == (2, 2, 0.6)
    d = s.step(arrive(13))                 # (7,6): rho 0.7 > 0.65 -> M_tar = ceil(13/5) = 3
    assert (d["m"], d["m_target"]) == (3, 3)
    assert sorted(len(v) for v in groups(s).values()) == [4, 4, 5]   # free moves balance
    one_each = [v[0] for v in groups(s).values()]
    d = s.step(ev(SR.DEPART, *one_each))   # (4,3,3): rho 0.4 in the band, although ceil(10/5) = 2
    assert (d["m"], d["m_target"], d["rho_max"]) == (3, 3, 0.4)


def pin_migration_cost_blocks(mod):
    """(4,0) with kappa = 100 ms each: Gamma = 330 - max(l(3), l(1)) - 100 = -30: nothing moves;
    with kappa = 50 for session 5 only, Gamma = +20 for it: it moves, and then from (3,1)
    Gamma = 260 - 200 - 100 < 0."""
    for cheap, expect in ((None, {0: [1, 3, 5, 7], 1: []}), (5, {0: [1, 3, 7], 1: [5]})):
        s = make(mod, m_min=2, m_max=2, m_init=2, beta=1e-3)
        s.step([(SR.ARRIVE, i, 50000 if i == cheap else 100000) for i in range(1, 9)])
        assert groups(s) == {0: [1, 3, 5, 7], 1: [2, 4, 6, 8]}
        d = s.step(ev(SR.DEPART, 2, 4, 6, 8))
        assert groups(s) == expect
        assert d["migrations"] == (0 if cheap is None else 1)


def pin_closed_loop_trace(mod):
    """Alg. 1 by hand: K = 4, l = (0, 150, 200, 260, 330), rho* = 0.5, delta = 0.1 (band
    [0.4, 0.6]), budget 1..8, free migration (eta kappa = 0, so a move needs L' < L)."""
    s = make(mod)
    # E1: 1 -> g0; rho 0.25 < 0.4 but M_tar = max(1, ceil(1/2)) = 1: no change
    d = s.step(arrive(1))
    assert (d["m"], d["m_target"], groups(s)) == (1, 1, {0: [1]})
    # E2: (3) rho 0.75 > 0.6 -> M_tar = ceil(3/2) = 2: add g1, then rebalance: from g0,
    # L' = max(l(2), l(1)) = 200 < 260 for every session -> first (session 1); then (2,1) stops.
    d = s.step(arrive(2, 3))
    assert (d["m"], d["m_target"], d["migrations"]) == (2, 2, 1)
    assert groups(s) == {0: [2, 3], 1: [1]} and d["rho_max"] == 0.5
    # E3: 4 -> g1 (200 < 260); (2,2) rho 0.5 in the band: no scaling
    d = s.step(arrive(4))
    assert (d["m"], groups(s)) == (2, {0: [2, 3], 1: [1, 4]})
    # E4: 5 -> g0 (tie at 260, equal loads, lower id); rho 0.75 -> M_tar = ceil(5/2) = 3, add g2;
    # from g0 = {2,3,5}: to g1 L' = 260 (gain 0), to g2 L' = 200 (gain 60) -> session 2 -> g2;
    # then g0 = {3,5} vs g2 = {2}: L' = max(l(1), l(2)) = 200, gain 0: stop.
    d = s.step(arrive(5))
    assert (d["m"], d["m_target"], d["migrations"]) == (3, 3, 1)
    assert groups(s) == {0: [3, 5], 1: [1, 4], 2: [2]}
    # E5: 1, 3, 5 idle -> loads (0,1,1); rho 0.25 < 0.4 -> M_tar = max(1, ceil(2/2)) = 1:
    # remove the two least-loaded GPUs, g0 (empty) and then g2 (load 1, higher id than g1);
    # session 2 goes to g1.
    d = s.step(ev(SR.IDLE, 1, 3, 5))
    assert (d["m"], d["m_target"], d["placed"], d["migrations"]) == (1, 1, 0, 1)
    assert groups(s) == {1: [2, 4]} and d["rho_max"] == 0.5
    # E6: 1, 3, 5 return: 1 and 3 fill g1, 5 is pending (rho_max = inf) -> M_tar = ceil(5/2) = 3:
    # new GPUs g3, g4 (fresh ids); 5 -> g3 (tie with g4 at L = 330, lower id); rebalance from
    # g1 = {1,2,3,4}: to g3 (load 1) or g4 (load 0) L' = 260, gain 70 -> the less-loaded g4 takes
    # session 1; then from g1 = {2,3,4}: to g3 or g4 (both load 1) L' = 200, gain 60 -> the lower
    # id, g3, takes session 2; then (2,2,1) stops.
    d = s.step(ev(SR.ACTIVATE, 1, 3, 5))
    assert (d["m"], d["m_target"], d["placed"], d["migrations"], d["pending"]) == (3, 3, 3, 2, 0)
    assert groups(s) == {1: [3, 4], 3: [2, 5], 4: [1]}


def pin_scale_direction_bounds_target(mod):
    """Sec. 5.2.2: the hysteresis band decides the direction of a scaling step and the
    proportional rule M_tar = ceil(N_req / (K rho*)) its size.  A scale-out that would lower M,
    or a scale-in that would raise it, contradicts the direction the band chose, so the target is
    bounded by M(t-) on the side the band points away from.

    Reachable scale-out case by hand: K = 4, l = (0, 150, 200, 260, 330), rho* = 0.5, delta = 0.1
    (band [0.4, 0.6]), budget 1..3 starting at 3, kappa = 10^6 ms per session (no move can pay).
    E1: sessions 1..12 arrive round robin, (4,4,4), rho 1.0 > 0.6: M_tar = ceil(12/2) = 6,
    clamped to m_max = 3: no change.  E2: every session of g1 and g2 departs, (4,0,0): moving one
    gains 330 - max(l(3), l(1)) - 10^6 < 0, nothing moves; rho 1.0 > 0.6 is a scale-out, while
    ceil(4/2) = 2 < 3: M stays 3 and nothing is removed.

    Scale-in: with every active session placed, N_req <= M n_max, so rho_max < rho* - delta gives
    N_req / (K rho*) < M and ceil(...) <= M: the bound never binds on a reachable state.  It is
    pinned on the controller itself: rho_max = 0.1 (below the band) with a proportional target of
    ceil(100/2) = 50 GPUs for M = 2 is a scale-in, which removes no GPU and so adds none either."""
    s = make(mod, m_min=1, m_max=3, m_init=3, alpha=1e6)
    d = s.step(arrive(*range(1, 13)))
    assert groups(s) == {0: [1, 4, 7, 10], 1: [2, 5, 8, 11], 2: [3, 6, 9, 12]}
    assert (d["m"], d["m_target"]) == (3, 3)
    d = s.step(ev(SR.DEPART, 2, 5, 8, 11, 3, 6, 9, 12))
    assert (d["rho_max"], d["n_req"], d["migrations"]) == (1.0, 4, 0)
    assert (d["m"], d["m_target"]) == (3, 3)
    assert groups(s) == {0: [1, 4, 7, 10], 1: [], 2: []}
    s = make(mod, m_min=1, m_max=100, m_init=2)
    assert s.target(100) == 50
    assert s.scale(0.1, 2, 100) == 2          # scale-in: min(50, 2)
    assert s.scale(0.9, 60, 100) == 60        # scale-out: max(50, 60)
    assert s.scale(0.9, 2, 100) == 50 and s.scale(0.1, 60, 100) == 50
    assert s.scale(0.5, 2, 100) == 2          # inside the band: M unchanged


def pin_gmax_lowest_id_tie(mod):
    """Sec. 5.2.1 leaves g_max in argmax_j l(n_j); the reading takes the lowest-id GPU at the
    bottleneck.  By hand: K = 4, l = (0, 150, 200, 260, 330), budget fixed at three GPUs, free
    migration.  E1: sessions 1..9 round robin, (3,3,3).  E2: sessions 3 and 9 of g2 depart,
    (3,3,1): g0 and g1 share the bottleneck 260; g_max = g0, and moving its lowest session (1)
    to g2 gives L' = max(l(2), l(2)) = 200 < 260 (the move to g1 would give l(4)).  Then (2,3,2):
    g_max = g1, and its best move gives L' = max(l(2), l(3)) = 260, no gain: stop, with session 1
    on g2 (taking g1 first would have moved session 2 instead)."""
    s = make(mod, m_min=3, m_max=3, m_init=3)
    s.step(arrive(*range(1, 10)))
    assert groups(s) == {0: [1, 4, 7], 1: [2, 5, 8], 2: [3, 6, 9]}
    d = s.step(ev(SR.DEPART, 3, 9))
    assert d["migrations"] == 1 and d["bottleneck_ms"] == 260.0
    assert groups(s) == {0: [4, 7], 1: [2, 5, 8], 2: [1, 6]}


def pin_pending_when_full(mod):
    """K = 2, budget fixed at one GPU: the third active session has to wait."""
    s = make(mod, K=2, lat=[0.0, 100.0, 150.0], m_min=1, m_max=1)
    d = s.step(arrive(1, 2, 3))
    assert (d["pending"], d["rho_max"], d["m"], d["n_req"]) == (1, math.inf, 1, 3)
    assert dict(s.placement()) == {1: 0, 2: 0, 3: -1}
    d = s.step(ev(SR.DEPART, 1))
    assert (d["pending"], d["rho_max"], d["placed"]) == (0, 1.0, 1)
    assert dict(s.placement()) == {2: 0, 3: 0}


def pin_parameter_delay(mod):
    """The new (lambda, rho_hat) of epoch t applies from epoch t+1 (App. A, replace step).
    Two levels: rho* 0.8 up to sigma 0.1, 0.25 above; delta 0.05, K = 4."""
    s = make(mod, delta=0.05, window=2, m_max=10, bounds=[0.1], lams=[0.1, 0.3], rhos=[0.8, 0.25])
    d = s.step(arrive(1))              # a = [1]: sigma 0, level 1
    assert (d["m"], d["level"]) == (1, 1)
    # (3): rho 0.75 is inside [0.75, 0.85] of the level-1 band: no scaling in this epoch, although
    # the window [1, 2] (sigma 0.5) now selects level 2 (rho 0.25)
    d = s.step(arrive(2, 3))
    assert (d["m"], d["level"], d["rho_hat"], d["lambda"]) == (1, 2, 0.25, 0.3)
    # next epoch: 0.75 > 0.30 -> M_tar = ceil(3 / 1) = 3, sessions spread one per GPU
    d = s.step([])
    assert d["m"] == 3 and sorted(len(v) for v in groups(s).values()) == [1, 1, 1]


def pin_changes_within_one_epoch(mod):
    """Changes of one epoch take effect together: idle-and-back keeps the GPU, a session that
    departs and re-arrives under the same id is a new session, arrive-then-idle never holds a GPU."""
    s = make(mod, m_min=2, m_max=2, m_init=2, alpha=1000.0)
    s.step(arrive(1, 2, 3))                               # g0 = {1,3}, g1 = {2}
    d = s.step(ev(SR.IDLE, 1) + ev(SR.ACTIVATE, 1))
    assert groups(s) == {0: [1, 3], 1: [2]} and (d["placed"], s.history[-1]) == (0, 1)
    # the new session 3 is placed afresh: g0 and g1 both give 200 with equal loads -> g0
    d = s.step(ev(SR.DEPART, 3) + arrive(3))
    assert groups(s) == {0: [1, 3], 1: [2]} and d["placed"] == 1
    d = s.step(arrive(4) + ev(SR.IDLE, 4))
    assert dict(s.placement())[4] == -1 and d["placed"] == 0 and d["n_req"] == 3


def pin_invalid_changes(mod):
    s = make(mod)
    s.step(arrive(1, 2) + ev(SR.IDLE, 2))
    before = (s.placement(), s.gpu_loads(), list(s.history), dict(s.active))
    for bad in (arrive(3) + arrive(1), arrive(3) + ev(SR.IDLE, 2), ev(SR.ACTIVATE, 1),
                ev(SR.DEPART, 9), [(7, 1, 0)], [(SR.ARRIVE, 4, -1)]):
        with pytest.raises(mod.SchedError):
            s.step(bad)
        assert (s.placement(), s.gpu_loads(), list(s.history), dict(s.active)) == before


def pin_invariants(mod):
    for seed in (1, 2, 3):
        trace = W.session_trace(60, seed=seed, mean_arrivals=1.5, burst_every=9, burst=6,
                                p_idle=0.2, p_resume=0.3, p_depart=0.08)
        s = app_a(mod, K=4, m_min=1, m_max=6, m_init=1, lat=LAT4, beta=1e-4, window=6)
        for ch in trace:
            d = s.step(ch)
            loads = dict(s.gpu_loads())
            assert len(loads) == d["m"] and 1 <= d["m"] <= 6
            assert all(n <= 4 for n in loads.values())
            place = dict(s.placement())
            for i, g in place.items():
                if not s.active[i]:
                    assert g == -1
                else:
                    assert g == -1 or g in loads
            waiting = sum(1 for i, g in place.items() if s.active[i] and g == -1)
            assert waiting == d["pending"]
            if waiting:
                assert d["m"] == 6 and all(n == 4 for n in loads.values())
            assert d["bottleneck_ms"] == max((LAT4[n] for n in loads.values()), default=0.0)


PINS = [pin_app_a_table, pin_volatility_numpy, pin_activations_count, pin_target_budget,
        pin_placement_optimal, pin_assignment_and_gain, pin_assignment_prefers_less_loaded,
        pin_hysteresis_band, pin_migration_cost_blocks, pin_scale_direction_bounds_target,
        pin_gmax_lowest_id_tie, pin_closed_loop_trace, pin_pending_when_full, pin_parameter_delay,
        pin_changes_within_one_epoch, pin_invalid_changes,
        pin_invariants]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_oracle_pin(pin):
    pin(SR)


# ---- planted mistakes ---------------------------------------------------------------------
MUTANTS = {
    "gain_sign": ("gain = (L - Lp) - self.eta", "gain = (Lp - L) - self.eta"),
    "no_migration_cost": ("gain = (L - Lp) - self.eta * self.kappa(i)", "gain = (L - Lp)"),
    "kappa_no_beta": ("return self.alpha + self.beta * float(self.bytes[i])", "return self.alpha"),
    "lprime_target_only": ("Lp = max(self.lat[self.load(moved, gmax)], self.lat[self.load(moved, j)])",
                           "Lp = self.lat[self.load(moved, j)]"),
    "lprime_source_only": ("Lp = max(self.lat[self.load(moved, gmax)], self.lat[self.load(moved, j)])",
                           "Lp = self.lat[self.load(moved, gmax)]"),
    "rebalance_tie_ignores_load": ("tie = (self.load(phi, j), j, i)", "tie = (j, i)"),
    "gmax_min": ("key=lambda g: (-lat_of[g], g)", "key=lambda g: (lat_of[g], g)"),
    "gmax_highest_id_tie": ("key=lambda g: (-lat_of[g], g)", "key=lambda g: (-lat_of[g], -g)"),
    "scale_out_may_shrink": ("return max(self.target(n_req), m_prev)", "return self.target(n_req)"),
    "scale_in_may_grow": ("return min(self.target(n_req), m_prev)", "return self.target(n_req)"),
    "assign_tie_more_loaded": ("key = (self.bottleneck(trial, gpus), n, g)",
                               "key = (self.bottleneck(trial, gpus), -n, g)"),
    "assign_ignores_latency": ("key = (self.bottleneck(trial, gpus), n, g)", "key = (n, g)"),
    "capacity_off_by_one": ("if n >= self.K:", "if n > self.K:"),
    "target_capacity_off_by_one": ("if j == gmax or self.load(phi, j) >= self.K:",
                                   "if j == gmax or self.load(phi, j) > self.K:"),
    "hysteresis_out_sign": ("rho_max > self.rho_hat + self.delta", "rho_max > self.rho_hat - self.delta"),
    "hysteresis_in_sign": ("rho_max < self.rho_hat - self.delta", "rho_max < self.rho_hat + self.delta"),
    "target_no_rho": ("n_req / (self.K * self.rho_hat)", "n_req / self.K"),
    "target_floor": ("m = math.ceil(", "m = math.floor("),
    "target_no_clamp_max": ("return min(max(m, self.m_min), self.m_max)", "return max(m, self.m_min)"),
    "scale_in_most_loaded": ("key=lambda g: (self.load(self.phi, g), -g)",
                             "key=lambda g: (-self.load(self.phi, g), -g)"),
    "scale_in_lower_id": ("key=lambda g: (self.load(self.phi, g), -g)",
                          "key=lambda g: (self.load(self.phi, g), g)"),
    "quantise_flip": ("if sigma > b:", "if sigma < b:"),
    "window_head": ("window = self.history[-self.W:]", "window = self.history[:self.W]"),
    "sample_std": ("statistics.pstdev(window)", "statistics.stdev(window)"),
    "rho_level_index": ("self.rho_tab[self.level - 1]", "self.rho_tab[min(self.level, len(self.rho_tab) - 1)]"),
    "activate_not_counted": ("active[i] = True\n                a_t += 1", "active[i] = True"),
    "idle_not_suspended": ("(self.phi.get(i) if active[i] and i not in fresh else None)",
                           "(self.phi.get(i) if i not in fresh else None)"),
    "update_before_scale": [("        a_t = self.apply_changes(changes)\n",
                             "        a_t = self.apply_changes(changes)\n        self.update_parameters(a_t)\n"),
                            ("        self.update_parameters(a_t)\n        return {", "        return {")],
    "n_req_placed_only": ("n_req = sum(1 for i in self.active if self.active[i])",
                          "n_req = sum(1 for i in self.active if self.phi[i] is not None)"),
    "pending_rho_finite": ("if self.pending() > 0:\n            return math.inf", "if False:\n            pass"),
    "no_rebalance_after_scale_out": ("            self.next_gpu += m_tar - m_prev\n            self.place(self.gpus, stats)",
                                     "            self.next_gpu += m_tar - m_prev"),
    "gpu_ids_reused": ("list(range(self.next_gpu, self.next_gpu + m_tar - m_prev))",
                       "[max(self.gpus, default=-1) + 1 + r for r in range(m_tar - m_prev)]"),
}


def mutant_module(name):
    edits = MUTANTS[name]
    src = open(SR.__file__).read()
    for old, new in (edits if isinstance(edits, list) else [edits]):
        assert src.count(old) == 1, name
        src = src.replace(old, new)
    mod = types.ModuleType("sched_mutant_" + name)
    mod.__dict__["__file__"] = SR.__file__
    exec(compile(src, "sched_mutant_" + name, "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name):
    mod = mutant_module(name)
    for pin in PINS:
        try:
            pin(mod)
        except Exception:  # an assertion or a crash both count as caught
            return
    raise AssertionError(f"mutant {name} passes every pin")
