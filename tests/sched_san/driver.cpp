// driver.cpp -- drives libts_sched's C ABI (include/ts_sched.h) with random valid and invalid
// epoch batches; built together with csrc/sched.cpp under AddressSanitizer and UBSan by
// tests/test_sched_sanitized.py (host code only).  Checks after every epoch:
//  * the decision against the scheduler's own placement and GPU list: n_req = active sessions,
//    m = GPUs within [m_min, m_max], loads <= K and equal to the placed sessions per GPU, idle
//    sessions unplaced, pending = active sessions without a GPU, pending > 0 only with every
//    GPU full at m = m_max, the bottleneck = max l(load), rho_max = max load / K (+inf while
//    pending), level within 1..L;
//  * a rejected batch (unknown session, duplicate arrival, wrong state, bad kind, negative size,
//    or a bad argument) changes nothing: a twin scheduler that never saw it makes bit-identical
//    decisions afterwards;
//  * invalid parameter sets are refused by ts_sched_create.
// usage: driver [configs] [epochs] [seed]; exit status 0 when every check holds.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <vector>

#include "ts_sched.h"

namespace {

struct Rng {  // xorshift64*
  uint64_t s;
  explicit Rng(uint64_t seed) : s(seed * 0x9E3779B97F4A7C15ull + 1) {}
  uint64_t next() {
    s ^= s >> 12; s ^= s << 25; s ^= s >> 27;
    return s * 0x2545F4914F6CDD1Dull;
  }
  int32_t range(int32_t lo, int32_t hi) { return lo + (int32_t)(next() % (uint64_t)(hi - lo + 1)); }
  double unit() { return (double)(next() >> 11) * (1.0 / 9007199254740992.0); }
};

int g_fail = 0;
#define CHECK(cond, ...)                                  \
  do {                                                    \
    if (!(cond)) {                                        \
      std::fprintf(stderr, "check failed: %s: ", #cond);  \
      std::fprintf(stderr, __VA_ARGS__);                  \
      std::fprintf(stderr, "\n");                         \
      ++g_fail;                                           \
      return false;                                       \
    }                                                     \
  } while (0)

ts_sched_params random_params(Rng& r) {
  ts_sched_params p;
  std::memset(&p, 0, sizeof p);
  p.K = r.range(1, 8);
  p.m_min = r.range(0, 3);
  p.m_max = p.m_min + r.range(0, 40);
  p.m_init = r.range(p.m_min, p.m_max);
  double l = r.unit() < 0.5 ? 0.0 : 5.0 * r.unit();
  for (int n = 0; n <= p.K; ++n) {
    p.chunk_latency[n] = l;
    l += r.unit() < 0.2 ? 0.0 : 10.0 + 90.0 * r.unit();
  }
  p.eta = 0.1 + 2.0 * r.unit();
  p.mig_alpha_ms = r.unit() < 0.3 ? 0.0 : 50.0 * r.unit();
  p.mig_beta_ms_per_byte = r.unit() < 0.3 ? 0.0 : 1e-8 * r.unit();
  p.delta = 0.2 * r.unit();
  p.window = r.range(1, 20);
  p.levels = r.range(1, 4);
  double b = 0.5 * r.unit();
  for (int i = 0; i < p.levels; ++i) {
    p.level_bound[i] = b;
    b += 0.1 + r.unit();
    p.level_lambda[i] = 0.5 + r.unit();
    p.level_rho[i] = 0.3 + 0.7 * r.unit();
  }
  return p;
}

struct Shadow {
  std::map<int64_t, bool> active;  // live sessions: id -> active
  int64_t next_id = 1;
};

// a valid batch of changes for the shadow state (applied to the shadow)
void valid_batch(Rng& r, Shadow& sh, std::vector<int32_t>& kinds, std::vector<int64_t>& ids,
                 std::vector<int64_t>& bytes) {
  kinds.clear(); ids.clear(); bytes.clear();
  const int n = r.range(0, 12);
  for (int c = 0; c < n; ++c) {
    const int what = r.range(0, 9);
    if (what < 4 || sh.active.empty()) {  // arrival
      const int64_t id = sh.next_id++;
      kinds.push_back(TS_EV_ARRIVE); ids.push_back(id); bytes.push_back((int64_t)(r.next() % (1ull << 33)));
      sh.active[id] = true;
      continue;
    }
    auto it = sh.active.begin();
    std::advance(it, r.range(0, (int32_t)sh.active.size() - 1));
    const int64_t id = it->first;
    if (what < 6) {
      kinds.push_back(TS_EV_DEPART);
      sh.active.erase(it);
    } else if (it->second) {
      kinds.push_back(TS_EV_IDLE);
      it->second = false;
    } else {
      kinds.push_back(TS_EV_ACTIVATE);
      it->second = true;
    }
    ids.push_back(id);
    bytes.push_back(0);
  }
}

// one invalid change appended to a (valid) batch; the shadow is left unchanged
void make_invalid(Rng& r, const Shadow& sh, std::vector<int32_t>& kinds, std::vector<int64_t>& ids,
                  std::vector<int64_t>& bytes) {
  const int what = r.range(0, 5);
  int64_t live = sh.active.empty() ? 0 : sh.active.begin()->first;
  bool live_active = sh.active.empty() ? false : sh.active.begin()->second;
  // the batch may already have changed that session; pick a case that is invalid regardless
  switch (what) {
    case 0: kinds.push_back(TS_EV_DEPART); ids.push_back(sh.next_id + 1000); bytes.push_back(0); break;
    case 1: kinds.push_back(TS_EV_ACTIVATE); ids.push_back(sh.next_id + 1001); bytes.push_back(0); break;
    case 2: kinds.push_back(TS_EV_ARRIVE); ids.push_back(sh.next_id + 1002); bytes.push_back(-5); break;
    case 3: kinds.push_back(7); ids.push_back(live); bytes.push_back(0); break;
    case 4:  // the same new session arriving twice in one batch
      kinds.push_back(TS_EV_ARRIVE); ids.push_back(sh.next_id + 1003); bytes.push_back(1);
      kinds.push_back(TS_EV_ARRIVE); ids.push_back(sh.next_id + 1003); bytes.push_back(1);
      break;
    default:  // idle twice in a row
      kinds.push_back(TS_EV_ARRIVE); ids.push_back(sh.next_id + 1004); bytes.push_back(1);
      kinds.push_back(TS_EV_IDLE); ids.push_back(sh.next_id + 1004); bytes.push_back(0);
      kinds.push_back(TS_EV_IDLE); ids.push_back(sh.next_id + 1004); bytes.push_back(0);
      break;
  }
  (void)live_active;
}

bool same_decision(const ts_sched_decision& a, const ts_sched_decision& b) {
  return std::memcmp(&a, &b, sizeof a) == 0;
}

bool check_epoch(const ts_sched* s, const ts_sched_params& p, const Shadow& sh,
                 const ts_sched_decision& d) {
  const int32_t cap = 1 << 16;
  std::vector<int64_t> pid(cap);
  std::vector<int32_t> pg(cap), gid(cap), gl(cap);
  int32_t ns = 0, ng = 0;
  CHECK(ts_sched_placement(s, pid.data(), pg.data(), cap, &ns) == TS_SCHED_OK, "placement");
  CHECK(ts_sched_gpus(s, gid.data(), gl.data(), cap, &ng) == TS_SCHED_OK, "gpus");
  CHECK(ns == (int32_t)sh.active.size(), "%d sessions vs %zu", ns, sh.active.size());
  CHECK(ng == d.m, "gpus %d vs m %d", ng, d.m);
  CHECK(d.m >= p.m_min && d.m <= p.m_max, "m %d outside [%d, %d]", d.m, p.m_min, p.m_max);
  std::map<int32_t, int32_t> load;
  for (int32_t g = 0; g < ng; ++g) {
    CHECK(gl[g] >= 0 && gl[g] <= p.K, "load %d", gl[g]);
    CHECK(g == 0 || gid[g] > gid[g - 1], "gpu order");
    load[gid[g]] = 0;
  }
  int32_t n_active = 0, unplaced_active = 0;
  for (int32_t i = 0; i < ns; ++i) {
    auto it = sh.active.find(pid[i]);
    CHECK(it != sh.active.end(), "unknown session %lld", (long long)pid[i]);
    CHECK(i == 0 || pid[i] > pid[i - 1], "session order");
    if (!it->second) {
      CHECK(pg[i] == -1, "idle session %lld placed", (long long)pid[i]);
      continue;
    }
    ++n_active;
    if (pg[i] < 0) { ++unplaced_active; continue; }
    CHECK(load.count(pg[i]) == 1, "session on unknown GPU %d", pg[i]);
    ++load[pg[i]];
  }
  CHECK(d.n_req == n_active, "n_req %d vs %d", d.n_req, n_active);
  CHECK(d.pending == unplaced_active, "pending %d vs %d", d.pending, unplaced_active);
  double L = 0.0, rmax = 0.0;
  bool any = false;
  for (int32_t g = 0; g < ng; ++g) {
    CHECK(load[gid[g]] == gl[g], "gpu %d load %d vs placed %d", gid[g], gl[g], load[gid[g]]);
    if (!any || p.chunk_latency[gl[g]] > L) L = p.chunk_latency[gl[g]];
    any = true;
    rmax = std::fmax(rmax, (double)gl[g] / p.K);
    if (d.pending > 0) CHECK(gl[g] == p.K, "pending with a free slot");
  }
  if (d.pending > 0) CHECK(d.m == p.m_max, "pending below m_max");
  CHECK(d.bottleneck_ms == L, "bottleneck %g vs %g", d.bottleneck_ms, L);
  if (d.pending > 0) CHECK(std::isinf(d.rho_max) && d.rho_max > 0, "rho_max while pending");
  else CHECK(d.rho_max == rmax, "rho_max %g vs %g", d.rho_max, rmax);
  CHECK(d.level >= 1 && d.level <= p.levels, "level %d", d.level);
  CHECK(d.placed >= 0 && d.migrations >= 0, "counts");
  CHECK(std::isfinite(d.volatility) && d.volatility >= 0.0, "volatility");
  return true;
}

}  // namespace

int main(int argc, char** argv) {
  const int configs = argc > 1 ? std::atoi(argv[1]) : 40;
  const int epochs = argc > 2 ? std::atoi(argv[2]) : 120;
  const uint64_t seed = argc > 3 ? std::strtoull(argv[3], nullptr, 10) : 1;
  Rng r(seed);
  if (ts_sched_abi_version() != TS_SCHED_ABI_VERSION) return 1;
  int rejected = 0, steps = 0;
  for (int cfg = 0; cfg < configs && g_fail == 0; ++cfg) {
    // invalid parameter sets are refused
    ts_sched_params bad = random_params(r);
    ts_sched* none = nullptr;
    switch (cfg % 6) {
      case 0: bad.K = 0; break;
      case 1: bad.m_init = bad.m_max + 1; break;
      case 2: bad.chunk_latency[1] = bad.chunk_latency[0] - 1.0; break;
      case 3: bad.eta = NAN; break;
      case 4: bad.window = 0; break;
      default: bad.level_rho[0] = 1.5; break;
    }
    if (ts_sched_create(&bad, &none) != TS_SCHED_ERR_ARG || none != nullptr) {
      std::fprintf(stderr, "bad params accepted (case %d)\n", cfg % 6);
      return 1;
    }
    if (ts_sched_create(nullptr, &none) != TS_SCHED_ERR_ARG) return 1;

    const ts_sched_params p = random_params(r);
    ts_sched *a = nullptr, *b = nullptr;
    if (ts_sched_create(&p, &a) != TS_SCHED_OK || ts_sched_create(&p, &b) != TS_SCHED_OK) return 1;
    Shadow sh;
    std::vector<int32_t> kinds;
    std::vector<int64_t> ids, bytes;
    for (int e = 0; e < epochs && g_fail == 0; ++e) {
      if (r.unit() < 0.15) {  // a rejected batch first, on scheduler a only
        Shadow tmp = sh;
        valid_batch(r, tmp, kinds, ids, bytes);
        make_invalid(r, sh, kinds, ids, bytes);
        ts_sched_decision junk;
        const int rc = ts_sched_step(a, (int32_t)kinds.size(), kinds.data(), ids.data(), bytes.data(), &junk);
        if (rc == TS_SCHED_OK) {
          std::fprintf(stderr, "invalid batch accepted (config %d epoch %d)\n", cfg, e);
          return 1;
        }
        if (ts_sched_step(a, -1, kinds.data(), ids.data(), nullptr, &junk) != TS_SCHED_ERR_ARG ||
            ts_sched_step(a, 1, nullptr, ids.data(), nullptr, &junk) != TS_SCHED_ERR_ARG)
          return 1;
        ++rejected;
      }
      valid_batch(r, sh, kinds, ids, bytes);
      ts_sched_decision da, db;
      const int32_t n = (int32_t)kinds.size();
      const int64_t* by = r.unit() < 0.1 ? nullptr : bytes.data();
      if (ts_sched_step(a, n, kinds.data(), ids.data(), by, &da) != TS_SCHED_OK ||
          ts_sched_step(b, n, kinds.data(), ids.data(), by, &db) != TS_SCHED_OK) {
        std::fprintf(stderr, "valid batch refused (config %d epoch %d)\n", cfg, e);
        return 1;
      }
      ++steps;
      if (!same_decision(da, db)) {
        std::fprintf(stderr, "twin schedulers diverged (config %d epoch %d)\n", cfg, e);
        return 1;
      }
      if (!check_epoch(a, p, sh, da)) std::fprintf(stderr, "  at config %d epoch %d\n", cfg, e);
    }
    ts_sched_destroy(a);
    ts_sched_destroy(b);
  }
  std::printf("configs %d, epochs %d, rejected batches %d, failures %d\n", configs, steps, rejected, g_fail);
  return g_fail == 0 ? 0 : 1;
}
