// sched.cpp -- the paper's closed-loop session scheduler (Sec. 5, Alg. 1, App. A) on the CPU,
// behind the C ABI of include/ts_sched.h.
//
// One call of ts_sched_step is one decision epoch t:
//   0. apply the epoch's session changes to the session table, then initialise the placement
//      from phi(t-): departed sessions are gone, sessions that ended the epoch idle are suspended
//      (their slot is released), sessions that arrived in the epoch hold no GPU;
//   1. PLACE (Sec. 5.2.1): assign U(t) = {active, unplaced} in increasing session id, each to the
//      feasible GPU (fewer than K sessions) with the smallest resulting bottleneck latency, ties
//      to the less-loaded GPU, then the lower GPU id; then migration-aware min-max rebalancing:
//      g_max is the lowest-id GPU of maximum latency, a move (i, j') gains
//      Gamma = (L - L') - eta * kappa_i with L = l(n_gmax), L' = max(l(n_gmax - 1), l(n_j' + 1))
//      and kappa_i = alpha + beta * bytes_i; the best move is applied while its gain is positive,
//      equal gains going to the less-loaded target (the assignment's tie rule), then the lower
//      target id, then the lower session id;
//   2. SCALE (Sec. 5.2.2): rho_max = max_j n_j / K (+infinity while an active session has no
//      GPU); above rho_hat + delta the budget may grow, below rho_hat - delta shrink, to
//      M_tar = ceil(N_req / (K rho_hat)) clamped to [m_min, m_max], N_req = active sessions;
//   3. Alg. 1: scale-in removes the least-loaded GPUs (the highest id first among equal loads) and
//      re-places their sessions with PLACE on the remaining GPUs; scale-out adds empty GPUs with
//      fresh ids, then runs PLACE;
//   4. App. A: a_t = arrivals + activations of the epoch; sigma(t) = population standard
//      deviation of the last W values of a; the level l with sigma in (bound_{l-1}, bound_l]
//      gives the (lambda, rho_hat) used from the next epoch on.
//
// Data structures: GPUs are grouped by load (by_load[n] = ids of the GPUs hosting n sessions).
// With l non-decreasing in n (validated at creation), every quantity the controller compares
// depends on a GPU only through its load class, so a placement choice looks at the lowest id of
// each non-empty class: O(K) per assigned session and O(K^2) per rebalancing move, independent
// of the number of GPUs.  A positive-gain move needs n_j' + 1 < n_gmax, which lowers the sum of
// squared loads by at least 2, so one PLACE makes at most N K / 2 moves.
#include "ts_sched.h"

#include <math.h>
#include <stdint.h>

#include <algorithm>
#include <map>
#include <new>
#include <set>
#include <vector>

namespace {

struct Session {
  bool active;
  int32_t gpu;    // -1: no GPU
  int64_t bytes;  // state size, for the migration cost
};

}  // namespace

struct ts_sched {
  ts_sched_params p;
  std::map<int64_t, Session> sessions;           // by id
  std::set<int64_t> waiting;                     // U(t): active sessions without a GPU
  int32_t n_active = 0;
  std::map<int32_t, std::set<int64_t>> gpus;     // GPU id -> its sessions
  std::vector<std::set<int32_t>> by_load;        // by_load[n] = GPUs hosting n sessions
  int32_t next_gpu = 0;
  std::vector<int32_t> window;                   // ring of the last W activation counts
  int32_t window_fill = 0, window_head = 0;
  int32_t level = 1;
  double rho_hat = 0.0, lambda = 0.0, sigma = 0.0;
};

namespace {

struct Stats {
  int32_t placed = 0, migrations = 0;
};

double lat(const ts_sched& s, int32_t n) { return s.p.chunk_latency[n]; }

// L: the largest latency over the provisioned GPUs (0 with none).
double bottleneck(const ts_sched& s) {
  double L = 0.0;
  bool any = false;
  for (int32_t n = 0; n <= s.p.K; ++n)
    if (!s.by_load[n].empty() && (!any || lat(s, n) > L)) {
      L = lat(s, n);
      any = true;
    }
  return L;
}

void put(ts_sched& s, int64_t id, int32_t g) {
  auto& on = s.gpus[g];
  const int32_t n = (int32_t)on.size();
  s.by_load[n].erase(g);
  s.by_load[n + 1].insert(g);
  on.insert(id);
  s.sessions[id].gpu = g;
}

void take(ts_sched& s, int64_t id) {
  Session& ss = s.sessions[id];
  if (ss.gpu < 0) return;
  auto& on = s.gpus[ss.gpu];
  const int32_t n = (int32_t)on.size();
  s.by_load[n].erase(ss.gpu);
  s.by_load[n - 1].insert(ss.gpu);
  on.erase(id);
  ss.gpu = -1;
}

// Lowest GPU id of load class n other than `except`; -1 if there is none.
int32_t first_of_class(const ts_sched& s, int32_t n, int32_t except) {
  for (int32_t g : s.by_load[n])
    if (g != except) return g;
  return -1;
}

// Session assignment of U(t), in increasing session id.
void assign(ts_sched& s, Stats& st) {
  std::vector<int64_t> placed_now;
  for (int64_t i : s.waiting) {
    const double L = bottleneck(s);
    int32_t best_g = -1;
    double best_L = 0.0;
    for (int32_t n = 0; n < s.p.K; ++n) {
      const int32_t g = first_of_class(s, n, -1);
      if (g < 0) continue;
      // l is non-decreasing, so the bottleneck after the placement is l(n + 1) or the old one
      const double Lg = lat(s, n + 1) > L ? lat(s, n + 1) : L;
      if (best_g < 0 || Lg < best_L) {  // classes come in increasing n: ties keep the less loaded
        best_g = g;
        best_L = Lg;
      }
    }
    if (best_g < 0) break;  // every GPU is full: this and the remaining sessions wait
    put(s, i, best_g);
    placed_now.push_back(i);
    ++st.placed;
  }
  for (int64_t i : placed_now) s.waiting.erase(i);
}

// Migration-aware min-max rebalancing from the bottleneck GPU.
void rebalance(ts_sched& s, Stats& st) {
  while (s.gpus.size() >= 2) {
    const double L = bottleneck(s);
    int32_t gmax = -1, nmax = 0;
    for (int32_t n = 0; n <= s.p.K; ++n)
      if (!s.by_load[n].empty() && lat(s, n) == L) {
        const int32_t g = *s.by_load[n].begin();
        if (gmax < 0 || g < gmax) {
          gmax = g;
          nmax = n;
        }
      }
    if (nmax == 0) break;
    // the first target of each load class below K, and the L' of a move there
    int32_t tgt[TS_SCHED_MAX_K];
    double lp[TS_SCHED_MAX_K];
    for (int32_t n = 0; n < s.p.K; ++n) {
      tgt[n] = first_of_class(s, n, gmax);
      const double a = lat(s, nmax - 1), b = lat(s, n + 1);
      lp[n] = a >= b ? a : b;
    }
    // the best move maximises the gain; equal gains go to the less-loaded target, then the
    // lower target id, then the lower session id
    bool have = false;
    double best_gain = 0.0;
    int64_t best_i = -1;
    int32_t best_j = -1, best_n = 0;
    for (int64_t i : s.gpus[gmax]) {
      const double kappa = s.p.mig_alpha_ms + s.p.mig_beta_ms_per_byte * (double)s.sessions[i].bytes;
      const double cost = s.p.eta * kappa;
      // this session's best target (classes come in increasing load)
      bool have_i = false;
      double gi = 0.0;
      int32_t ji = -1, ni = 0;
      for (int32_t n = 0; n < s.p.K; ++n) {
        if (tgt[n] < 0) continue;
        const double gain = (L - lp[n]) - cost;
        if (!have_i || gain > gi) {
          have_i = true;
          gi = gain;
          ji = tgt[n];
          ni = n;
        }
      }
      if (have_i && (!have || gi > best_gain ||
                     (gi == best_gain && (ni < best_n || (ni == best_n && ji < best_j))))) {
        have = true;  // sessions come in increasing id: a full tie keeps the earlier one
        best_gain = gi;
        best_i = i;
        best_j = ji;
        best_n = ni;
      }
    }
    if (!have || !(best_gain > 0.0)) break;
    take(s, best_i);
    put(s, best_i, best_j);
    ++st.migrations;
  }
}

void place(ts_sched& s, Stats& st) {
  assign(s, st);
  rebalance(s, st);
}

int32_t target_budget(const ts_sched& s, int32_t n_req) {
  // the 1e-9 keeps the binary rounding of a decimal rho (0.95, say) from adding a GPU
  double m = ceil((double)n_req / ((double)s.p.K * s.rho_hat) - 1e-9);
  if (m < (double)s.p.m_min) m = (double)s.p.m_min;
  if (m > (double)s.p.m_max) m = (double)s.p.m_max;
  return (int32_t)m;
}

void add_gpu(ts_sched& s) {
  const int32_t g = s.next_gpu++;
  s.gpus[g];
  s.by_load[0].insert(g);
}

double rho_max_now(const ts_sched& s) {
  if (!s.waiting.empty()) return INFINITY;
  int32_t top = 0;
  for (int32_t n = 0; n <= s.p.K; ++n)
    if (!s.by_load[n].empty()) top = n;
  return (double)top / (double)s.p.K;
}

void update_parameters(ts_sched& s, int32_t a_t) {
  const int32_t W = s.p.window;
  s.window[s.window_head] = a_t;
  s.window_head = (s.window_head + 1) % W;
  if (s.window_fill < W) ++s.window_fill;
  // population variance from exact integer sums, (n sum a^2 - (sum a)^2) / n^2: with the
  // numerator below 2^53 (any realistic trace) one rounding in the quotient and one in the root
  __int128 s1 = 0, s2 = 0;
  for (int32_t k = 0; k < s.window_fill; ++k) {
    const __int128 a = s.window[k];
    s1 += a;
    s2 += a * a;
  }
  const __int128 n = s.window_fill;
  s.sigma = n > 1 ? sqrt((double)(n * s2 - s1 * s1) / (double)(n * n)) : 0.0;
  int32_t lv = 1;
  for (int32_t b = 0; b + 1 < s.p.levels; ++b)
    if (s.sigma > s.p.level_bound[b]) ++lv;
  s.level = lv;
  s.rho_hat = s.p.level_rho[lv - 1];
  s.lambda = s.p.level_lambda[lv - 1];
}

bool finite_nonneg(double x) { return isfinite(x) && x >= 0.0; }

bool params_ok(const ts_sched_params* p) {
  if (p->K < 1 || p->K > TS_SCHED_MAX_K) return false;
  if (p->m_min < 0 || p->m_max < p->m_min || p->m_init < p->m_min || p->m_init > p->m_max ||
      p->m_max > TS_SCHED_MAX_GPUS)
    return false;
  if (!(finite_nonneg(p->eta) && p->eta > 0.0) || !finite_nonneg(p->delta)) return false;
  if (!finite_nonneg(p->mig_alpha_ms) || !finite_nonneg(p->mig_beta_ms_per_byte)) return false;
  if (p->window < 1 || p->window > TS_SCHED_MAX_WINDOW) return false;
  if (p->levels < 1 || p->levels > TS_SCHED_MAX_LEVELS) return false;
  for (int32_t i = 0; i < p->levels; ++i)
    if (!(p->level_rho[i] > 0.0 && p->level_rho[i] <= 1.0) || !isfinite(p->level_lambda[i]))
      return false;
  for (int32_t i = 0; i + 1 < p->levels; ++i) {
    if (!isfinite(p->level_bound[i])) return false;
    if (i > 0 && !(p->level_bound[i] > p->level_bound[i - 1])) return false;
  }
  for (int32_t n = 0; n <= p->K; ++n) {
    if (!isfinite(p->chunk_latency[n])) return false;
    if (n > 0 && p->chunk_latency[n] < p->chunk_latency[n - 1]) return false;
  }
  return true;
}

// state of a session while a batch of changes is checked: 0 absent, 1 active, 2 idle
int state_of(const ts_sched& s, const std::map<int64_t, int>& overlay, int64_t id) {
  auto o = overlay.find(id);
  if (o != overlay.end()) return o->second;
  auto it = s.sessions.find(id);
  if (it == s.sessions.end()) return 0;
  return it->second.active ? 1 : 2;
}

int check_changes(const ts_sched& s, int32_t n, const int32_t* kinds, const int64_t* ids,
                  const int64_t* state_bytes) {
  std::map<int64_t, int> overlay;
  for (int32_t c = 0; c < n; ++c) {
    const int st = state_of(s, overlay, ids[c]);
    switch (kinds[c]) {
      case TS_EV_ARRIVE:
        if (st != 0 || (state_bytes && state_bytes[c] < 0)) return TS_SCHED_ERR_SESSION;
        overlay[ids[c]] = 1;
        break;
      case TS_EV_DEPART:
        if (st == 0) return TS_SCHED_ERR_SESSION;
        overlay[ids[c]] = 0;
        break;
      case TS_EV_ACTIVATE:
        if (st != 2) return TS_SCHED_ERR_SESSION;
        overlay[ids[c]] = 1;
        break;
      case TS_EV_IDLE:
        if (st != 1) return TS_SCHED_ERR_SESSION;
        overlay[ids[c]] = 2;
        break;
      default:
        return TS_SCHED_ERR_ARG;
    }
  }
  return TS_SCHED_OK;
}

// Applies checked changes and initialises the placement from phi(t-); returns a_t.
int32_t apply_changes(ts_sched& s, int32_t n, const int32_t* kinds, const int64_t* ids,
                      const int64_t* state_bytes) {
  int32_t a_t = 0;
  std::set<int64_t> touched;
  for (int32_t c = 0; c < n; ++c) {
    const int64_t id = ids[c];
    touched.insert(id);
    switch (kinds[c]) {
      case TS_EV_ARRIVE:
        s.sessions[id] = Session{true, -1, state_bytes ? state_bytes[c] : 0};
        ++s.n_active;
        ++a_t;
        break;
      case TS_EV_DEPART:
        take(s, id);
        if (s.sessions[id].active) --s.n_active;
        s.sessions.erase(id);
        break;
      case TS_EV_ACTIVATE:
        s.sessions[id].active = true;
        ++s.n_active;
        ++a_t;
        break;
      case TS_EV_IDLE:  // the slot is released below, if the session ends the epoch idle
        s.sessions[id].active = false;
        --s.n_active;
        break;
    }
  }
  for (int64_t id : touched) {
    auto it = s.sessions.find(id);
    if (it == s.sessions.end()) {
      s.waiting.erase(id);
      continue;
    }
    if (!it->second.active) take(s, id);
    if (it->second.active && it->second.gpu < 0)
      s.waiting.insert(id);
    else
      s.waiting.erase(id);
  }
  return a_t;
}

}  // namespace

extern "C" {

int ts_sched_abi_version(void) { return TS_SCHED_ABI_VERSION; }

int ts_sched_create(const ts_sched_params* params, ts_sched** out) {
  if (!params || !out || !params_ok(params)) return TS_SCHED_ERR_ARG;
  ts_sched* s = new (std::nothrow) ts_sched;
  if (!s) return TS_SCHED_ERR_NOMEM;
  try {
    s->p = *params;
    s->by_load.resize(params->K + 1);
    s->window.assign(params->window, 0);
    for (int32_t i = 0; i < params->m_init; ++i) add_gpu(*s);
  } catch (const std::bad_alloc&) {
    delete s;
    return TS_SCHED_ERR_NOMEM;
  }
  s->rho_hat = params->level_rho[0];
  s->lambda = params->level_lambda[0];
  *out = s;
  return TS_SCHED_OK;
}

void ts_sched_destroy(ts_sched* s) { delete s; }

int ts_sched_step(ts_sched* s, int32_t n, const int32_t* kinds, const int64_t* ids,
                  const int64_t* state_bytes, ts_sched_decision* out) {
  if (!s || n < 0 || n > TS_SCHED_MAX_CHANGES || (n > 0 && (!kinds || !ids)))
    return TS_SCHED_ERR_ARG;
  try {
    const int bad = check_changes(*s, n, kinds, ids, state_bytes);
    if (bad != TS_SCHED_OK) return bad;
    const int32_t a_t = apply_changes(*s, n, kinds, ids, state_bytes);

    Stats st;
    place(*s, st);
    const int32_t m_prev = (int32_t)s->gpus.size();
    const int32_t n_req = s->n_active;
    const double rho = rho_max_now(*s);
    int32_t m_tar = m_prev;
    if (rho > s->rho_hat + s->p.delta)
      m_tar = std::max(target_budget(*s, n_req), m_prev);
    else if (rho < s->rho_hat - s->p.delta)
      m_tar = std::min(target_budget(*s, n_req), m_prev);

    if (m_tar < m_prev) {
      // scale-in: pick the GPUs to free, move their sessions onto the rest, then remove them
      std::vector<int32_t> removed;
      for (int32_t ld = 0; ld <= s->p.K && (int32_t)removed.size() < m_prev - m_tar; ++ld)
        for (auto r = s->by_load[ld].rbegin();
             r != s->by_load[ld].rend() && (int32_t)removed.size() < m_prev - m_tar; ++r)
          removed.push_back(*r);
      int32_t displaced = 0;
      for (int32_t g : removed) {
        const std::vector<int64_t> on(s->gpus[g].begin(), s->gpus[g].end());
        for (int64_t i : on) {
          take(*s, i);
          s->waiting.insert(i);
          ++displaced;
        }
        s->by_load[0].erase(g);
        s->gpus.erase(g);
      }
      Stats sub;
      place(*s, sub);
      st.placed += sub.placed - displaced;
      st.migrations += sub.migrations + displaced;
    } else if (m_tar > m_prev) {
      // scale-out: add the GPUs, then place and rebalance onto them
      for (int32_t r = 0; r < m_tar - m_prev; ++r) add_gpu(*s);
      place(*s, st);
    }
    update_parameters(*s, a_t);

    if (out) {
      ts_sched_decision d = {};
      d.m = (int32_t)s->gpus.size();
      d.m_target = m_tar;
      d.placed = st.placed;
      d.migrations = st.migrations;
      d.pending = (int32_t)s->waiting.size();
      d.n_req = n_req;
      d.level = s->level;
      d.bottleneck_ms = bottleneck(*s);
      d.rho_max = rho_max_now(*s);
      d.rho_hat = s->rho_hat;
      d.lambda = s->lambda;
      d.volatility = s->sigma;
      *out = d;
    }
  } catch (const std::bad_alloc&) {
    return TS_SCHED_ERR_NOMEM;
  }
  return TS_SCHED_OK;
}

int ts_sched_placement(const ts_sched* s, int64_t* ids, int32_t* gpus, int32_t cap,
                       int32_t* count) {
  if (!s || !count || cap < 0 || (cap > 0 && (!ids || !gpus))) return TS_SCHED_ERR_ARG;
  int32_t n = 0;
  for (auto& kv : s->sessions) {
    if (n < cap) {
      ids[n] = kv.first;
      gpus[n] = kv.second.gpu;
    }
    ++n;
  }
  *count = n;
  return TS_SCHED_OK;
}

int ts_sched_gpus(const ts_sched* s, int32_t* gpu_ids, int32_t* loads, int32_t cap,
                  int32_t* count) {
  if (!s || !count || cap < 0 || (cap > 0 && (!gpu_ids || !loads))) return TS_SCHED_ERR_ARG;
  int32_t n = 0;
  for (auto& g : s->gpus) {
    if (n < cap) {
      gpu_ids[n] = g.first;
      loads[n] = (int32_t)g.second.size();
    }
    ++n;
  }
  *count = n;
  return TS_SCHED_OK;
}

}  // extern "C"
