"""Plain reference of the paper's closed-loop session scheduler (Sec. 5, Alg. 1, App. A).

TEST INFRASTRUCTURE: only tests/, the smoke check and bench.py's cpu_baseline leg use this module;
the product scheduler is the C++ library behind include/ts_sched.h and shares no code with it.

Everything here is recomputed from scratch at every use (GPU loads by counting the placement,
the bottleneck as a maximum over all GPUs, every candidate placement built as a new dict), in
the order the paper gives the steps, so each step can be checked against the text by eye:

  one decision epoch t (Alg. 1):
    apply the epoch's session changes                            (Sec. 5.1, sessions and states)
    (phi, rho_max) <- PLACE(S, phi(t-), M(t-))                   (Sec. 5.2.1)
        initialise from phi(t-) (departed and suspended sessions hold no GPU)
        session assignment over U(t) = {active and unplaced}
        migration-aware min-max rebalancing while the best gain Gamma is positive
    M_tar <- SCALE(rho_max, M(t-))                               (Sec. 5.2.2)
        hysteresis: out if rho_max > rho_hat + delta, in if rho_max < rho_hat - delta
        proportional target M_tar = ceil(N_req / (K rho_hat))
    scale-in: PLACE onto the reduced set, then M <- M_tar; scale-out: M <- M_tar, then PLACE
    measure - quantise - look up - replace of (lambda, rho_hat)  (App. A)

Readings where the paper leaves a choice open:
  R1 idle sessions are suspended (their GPU slot released) as soon as they go idle;
  R2 U(t) is handled in increasing session id; assignment ties go to the less-loaded GPU, then
     to the lower GPU id;
  R3 rebalancing: g_max is the lowest-id GPU of maximum latency; a move (i, j') has
     L = l(n_gmax) and L' = max(l(n_gmax - 1), l(n_j' + 1)), the latencies of the two GPUs it
     changes; among equal gains the move to the less-loaded target is taken (the tie rule of
     assignment), then the lower target id, then the lower session id;
  R4 kappa_i = alpha + beta * (state bytes of s_i);
  R5 N_req counts every active session, placed or not; rho_max is +infinity while an active
     session has no GPU (all GPUs full), so the autoscaler scales out for it;
  R6 M_tar = ceil(N_req / (K rho_hat) - 1e-9), clamped to [m_min, m_max]; the 1e-9 absorbs the
     binary rounding of decimal rho values such as 0.95;
  R7 scale-in removes the least-loaded GPUs (the highest id first among equal loads); their
     sessions join U(t) and the second PLACE puts them on the remaining GPUs; scale-out adds
     empty GPUs with fresh ids (never reused);
  R8 a_t = number of arrivals plus activations in epoch t; sigma(t) = population standard
     deviation over the last W epochs (fewer at the start); level l holds sigma in
     (bound_{l-1}, bound_l]; the new (lambda, rho_hat) applies from the next epoch; before the
     first epoch the level-1 parameters hold.
"""
import math
import statistics

ARRIVE, DEPART, ACTIVATE, IDLE = 0, 1, 2, 3


class SchedError(ValueError):
    """An invalid session change: the scheduler state is left unchanged."""


class SchedRef:
    def __init__(self, K, m_min, m_max, m_init, chunk_latency, eta, alpha, beta, delta, window,
                 level_bound, level_lambda, level_rho):
        assert len(chunk_latency) == K + 1
        # latency grows with co-location (Sec. 5.1); rebalancing terminates because of it
        assert all(a <= b for a, b in zip(chunk_latency, chunk_latency[1:]))
        assert len(level_bound) == len(level_rho) - 1 and len(level_lambda) == len(level_rho)
        self.K, self.m_min, self.m_max = K, m_min, m_max
        self.lat = [float(x) for x in chunk_latency]
        self.eta, self.alpha, self.beta, self.delta = float(eta), float(alpha), float(beta), float(delta)
        self.W = window
        self.bound, self.lam_tab, self.rho_tab = list(level_bound), list(level_lambda), list(level_rho)
        self.active = {}       # session id -> bool (alpha_i)
        self.bytes = {}        # session id -> state bytes
        self.phi = {}          # session id -> GPU id or None
        self.gpus = list(range(m_init))
        self.next_gpu = m_init
        self.history = []      # a_tau of past epochs
        self.level, self.lam, self.rho_hat, self.sigma = 1, self.lam_tab[0], self.rho_tab[0], 0.0

    # ---- quantities of Sec. 5.1 / 5.2 ------------------------------------------------------
    def load(self, phi, g):
        """n_j: sessions placed on GPU g."""
        return sum(1 for x in phi.values() if x == g)

    def bottleneck(self, phi, gpus):
        """L: the largest per-chunk latency over the provisioned GPUs (0 with none)."""
        return max((self.lat[self.load(phi, g)] for g in gpus), default=0.0)

    def kappa(self, i):
        """Migration cost of session i in the alpha-beta model (R4)."""
        return self.alpha + self.beta * float(self.bytes[i])

    # ---- placement controller, Sec. 5.2.1 -------------------------------------------------
    def place(self, gpus, stats):
        phi = self.phi
        # session assignment over U(t), increasing id (R2)
        U = sorted(i for i in self.active if self.active[i] and phi[i] is None)
        for i in U:
            best = None
            for g in gpus:
                n = self.load(phi, g)
                if n >= self.K:
                    continue
                trial = dict(phi)
                trial[i] = g
                key = (self.bottleneck(trial, gpus), n, g)
                if best is None or key < best:
                    best = key
            if best is not None:
                phi[i] = best[2]
                stats["placed"] += 1
        # migration-aware min-max rebalancing (R3).  With l non-decreasing, a move of positive
        # gain has n_j' + 1 < n_gmax, so the sum of squared loads drops by at least 2 per move:
        # more than N K / 2 moves would mean the loop does not terminate.
        limit = len(phi) * self.K // 2 + 1
        moves = 0
        while len(gpus) >= 2:
            moves += 1
            if moves > limit:
                raise RuntimeError("rebalancing exceeded its move bound")
            lat_of = {g: self.lat[self.load(phi, g)] for g in gpus}
            gmax = min(gpus, key=lambda g: (-lat_of[g], g))
            L = lat_of[gmax]
            best = None
            for i in sorted(s for s in phi if phi[s] == gmax):
                for j in gpus:
                    if j == gmax or self.load(phi, j) >= self.K:
                        continue
                    moved = dict(phi)
                    moved[i] = j
                    Lp = max(self.lat[self.load(moved, gmax)], self.lat[self.load(moved, j)])
                    gain = (L - Lp) - self.eta * self.kappa(i)
                    tie = (self.load(phi, j), j, i)   # R3: less-loaded target, lower ids
                    if best is None or gain > best[0] or (gain == best[0] and tie < best[1]):
                        best = (gain, tie)
            if best is None or not best[0] > 0.0:
                break
            _, (_, j, i) = best
            phi[i] = j
            stats["migrations"] += 1

    def pending(self):
        return sum(1 for i in self.active if self.active[i] and self.phi[i] is None)

    def rho_max(self):
        """max_j n_j / K after placement; +inf while an active session has no GPU (R5)."""
        if self.pending() > 0:
            return math.inf
        return max((self.load(self.phi, g) for g in self.gpus), default=0) / self.K

    # ---- autoscaling controller, Sec. 5.2.2 -----------------------------------------------
    def target(self, n_req):
        m = math.ceil(n_req / (self.K * self.rho_hat) - 1e-9)  # R6
        return min(max(m, self.m_min), self.m_max)

    def scale(self, rho_max, m_prev, n_req):
        if rho_max > self.rho_hat + self.delta:
            return max(self.target(n_req), m_prev)
        if rho_max < self.rho_hat - self.delta:
            return min(self.target(n_req), m_prev)
        return m_prev

    # ---- App. A -----------------------------------------------------------------------------
    def quantise(self, sigma):
        level = 1
        for b in self.bound:
            if sigma > b:
                level += 1
        return level

    def update_parameters(self, a_t):
        self.history.append(a_t)
        window = self.history[-self.W:]
        self.sigma = statistics.pstdev(window) if len(window) > 1 else 0.0
        self.level = self.quantise(self.sigma)
        self.lam, self.rho_hat = self.lam_tab[self.level - 1], self.rho_tab[self.level - 1]

    # ---- one decision epoch, Alg. 1 ---------------------------------------------------------
    def apply_changes(self, changes):
        """Validates all changes against a copy first, so an invalid epoch changes nothing."""
        active, byts = dict(self.active), dict(self.bytes)
        fresh = set()          # sessions that arrived in this epoch: they hold no GPU yet
        a_t = 0
        for kind, i, nbytes in changes:
            if kind == ARRIVE:
                if i in active or nbytes < 0:
                    raise SchedError(f"bad arrival of session {i}")
                active[i], byts[i] = True, nbytes
                fresh.add(i)
                a_t += 1
            elif kind == DEPART:
                if i not in active:
                    raise SchedError(f"departure of unknown session {i}")
                del active[i], byts[i]
            elif kind == ACTIVATE:
                if i not in active or active[i]:
                    raise SchedError(f"activation of session {i} that is not idle")
                active[i] = True
                a_t += 1
            elif kind == IDLE:
                if i not in active or not active[i]:
                    raise SchedError(f"idle event of session {i} that is not active")
                active[i] = False
            else:
                raise SchedError(f"unknown event kind {kind}")
        # initialise from phi(t-): departed sessions vanish, idle ones are suspended (R1); a
        # session that went idle and came back within the epoch keeps its GPU
        self.phi = {i: (self.phi.get(i) if active[i] and i not in fresh else None) for i in active}
        self.active, self.bytes = active, byts
        return a_t

    def step(self, changes):
        a_t = self.apply_changes(changes)
        stats = {"placed": 0, "migrations": 0}
        self.place(self.gpus, stats)
        m_prev = len(self.gpus)
        n_req = sum(1 for i in self.active if self.active[i])
        m_tar = self.scale(self.rho_max(), m_prev, n_req)
        if m_tar < m_prev:
            # R7: the least-loaded GPUs go; their sessions are re-placed before the removal
            order = sorted(self.gpus, key=lambda g: (self.load(self.phi, g), -g))
            removed = set(order[:m_prev - m_tar])
            kept = [g for g in self.gpus if g not in removed]
            displaced = sorted(i for i in self.phi if self.phi[i] in removed)
            for i in displaced:
                self.phi[i] = None
            sub = {"placed": 0, "migrations": 0}
            self.place(kept, sub)
            stats["placed"] += sub["placed"] - len(displaced)
            stats["migrations"] += sub["migrations"] + len(displaced)
            self.gpus = kept
        elif m_tar > m_prev:
            self.gpus = self.gpus + list(range(self.next_gpu, self.next_gpu + m_tar - m_prev))
            self.next_gpu += m_tar - m_prev
            self.place(self.gpus, stats)
        self.update_parameters(a_t)
        return {
            "m": len(self.gpus), "m_target": m_tar, "placed": stats["placed"],
            "migrations": stats["migrations"], "pending": self.pending(), "n_req": n_req,
            "level": self.level, "bottleneck_ms": self.bottleneck(self.phi, self.gpus),
            "rho_max": self.rho_max(), "rho_hat": self.rho_hat, "lambda": self.lam,
            "volatility": self.sigma,
        }

    def placement(self):
        return [(i, -1 if self.phi[i] is None else self.phi[i]) for i in sorted(self.phi)]

    def gpu_loads(self):
        return [(g, self.load(self.phi, g)) for g in self.gpus]


def level_bounds_from_table(volatilities):
    """Level boundaries as the midpoints between consecutive tabulated level volatilities."""
    return [(a + b) / 2.0 for a, b in zip(volatilities[:-1], volatilities[1:])]
