/*
 * ts_sched.h -- C ABI of libts_sched.so: the paper's closed-loop session scheduler (CPU).
 *
 * The paper's scheduler (Sec. 5) runs at every event -- a session arriving, departing, or
 * switching between active and idle -- and jointly decides where each session runs and how
 * many GPUs are provisioned:
 *  - placement controller (Sec. 5.2.1): sessions that are active but unplaced are assigned one
 *    by one to the feasible GPU (fewer than K sessions) that minimises the resulting bottleneck
 *    per-chunk latency, ties to the less-loaded GPU; then migration-aware min-max rebalancing
 *    moves one session at a time off the bottleneck GPU g_max while the best gain
 *    Gamma = L - L' - eta * kappa_i is positive, kappa_i = alpha + beta * state bytes being the
 *    session's migration cost in the alpha-beta model.  L = l(n_gmax) is the bottleneck and L'
 *    the larger latency of the two GPUs the move changes, l(n_gmax - 1) and l(n_j' + 1): the
 *    maximum over all GPUs whenever g_max is the only bottleneck GPU, and still positive when
 *    several GPUs share the bottleneck, where the all-GPU maximum could never drop by one move;
 *    equal gains go to the less-loaded target, as in assignment;
 *  - autoscaling controller (Sec. 5.2.2): with rho_max = max_j n_j / K from placement, scale out
 *    when rho_max > rho_hat + delta and in when rho_max < rho_hat - delta (hysteresis), to
 *    M_tar = ceil(N_req / (K * rho_hat)) (proportional target tracking);
 *  - the closed loop of Alg. 1: place, compute M_tar, then for scale-in rebalance onto the
 *    reduced set before removing GPUs and for scale-out add GPUs before rebalancing (one call of
 *    ts_sched_step is one decision epoch);
 *  - adaptive parameters (App. A): the volatility sigma(t) = std of the newly activated session
 *    counts over the last W events is quantised to a level whose profiled (lambda, rho*) pair
 *    becomes the active (lambda, rho_hat) for the following events.
 * Everything is deterministic: sessions are handled in increasing id order and every tie is
 * broken by a fixed rule (documented at each step in csrc/sched.cpp).
 *
 * Ownership: ts_sched_create allocates the handle, ts_sched_destroy frees it; every array argument
 * is a host pointer owned by the caller and only read (or written, for the query calls) during
 * the call.
 * Threading: a ts_sched handle is not thread-safe; distinct handles are independent.
 * Errors: functions return a ts_sched_status; a call that returns an error changes nothing.
 */
#ifndef TS_SCHED_H
#define TS_SCHED_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TS_SCHED_ABI_VERSION 1
#define TS_SCHED_MAX_LEVELS 16
#define TS_SCHED_MAX_K 64
#define TS_SCHED_MAX_GPUS (1 << 20)     /* bound of m_max */
#define TS_SCHED_MAX_WINDOW 4096        /* bound of the volatility window W */
#define TS_SCHED_MAX_CHANGES (1 << 20)  /* session changes in one epoch */

typedef enum ts_sched_status {
  TS_SCHED_OK = 0,
  TS_SCHED_ERR_ARG = 1,      /* NULL pointer or parameter out of range */
  TS_SCHED_ERR_SESSION = 2,  /* unknown session, duplicate arrival, or event invalid in its state */
  TS_SCHED_ERR_NOMEM = 3
} ts_sched_status;

typedef enum ts_sched_event_kind {
  TS_EV_ARRIVE = 0,    /* a new session, active (needs a GPU) */
  TS_EV_DEPART = 1,    /* the session terminates; its slot and state are released */
  TS_EV_ACTIVATE = 2,  /* an idle (suspended) session becomes active again */
  TS_EV_IDLE = 3       /* an active session goes idle: it is suspended and its slot released */
} ts_sched_event_kind;

/* Scheduler parameters.  Latencies in milliseconds. */
typedef struct ts_sched_params {
  int32_t K;                 /* max concurrent sessions per GPU, 1..TS_SCHED_MAX_K */
  int32_t m_min, m_max;      /* bounds of the GPU budget, 0 <= m_min <= m_max <= TS_SCHED_MAX_GPUS */
  int32_t m_init;            /* initial budget, m_min <= m_init <= m_max */
  double chunk_latency[TS_SCHED_MAX_K + 1]; /* per-chunk latency l(n) of a GPU hosting n
                                               sessions, n = 0..K: finite and non-decreasing in
                                               n (co-location slows every session, Sec. 5.1);
                                               l(0), an empty GPU, is usually 0 */
  double eta;                /* weight of the migration cost in the gain, > 0 */
  double mig_alpha_ms;       /* alpha-beta migration cost: kappa = alpha + beta * state bytes */
  double mig_beta_ms_per_byte;
  double delta;              /* hysteresis half-width around rho_hat, >= 0 */
  int32_t window;            /* volatility window W in epochs, 1..TS_SCHED_MAX_WINDOW */
  int32_t levels;            /* L, 1..TS_SCHED_MAX_LEVELS; levels = 1 disables adaptation */
  double level_bound[TS_SCHED_MAX_LEVELS]; /* upper volatility bound of levels 1..L-1 (increasing);
                                              level L is unbounded */
  double level_lambda[TS_SCHED_MAX_LEVELS];
  double level_rho[TS_SCHED_MAX_LEVELS];   /* target utilisation rho* of each level, (0, 1] */
} ts_sched_params;

/* What one event decided. */
typedef struct ts_sched_decision {
  int32_t m;                 /* GPU budget M(t) after the event */
  int32_t m_target;          /* M_tar(t) computed by the autoscaler (== m unless scaled) */
  int32_t placed;            /* sessions given a GPU from the unplaced-active set U(t) (not
                                counting sessions of GPUs removed by scale-in) */
  int32_t migrations;        /* moves of a placed session to another GPU: rebalancing moves plus
                                sessions displaced from GPUs removed by scale-in */
  int32_t pending;           /* active sessions left without a GPU (all GPUs full at m_max) */
  int32_t n_req;             /* N_req(t): active sessions (placed or pending) */
  int32_t level;             /* volatility level in force after the event, 1..L */
  double bottleneck_ms;      /* L(t): max per-chunk latency over the GPUs */
  double rho_max;            /* max_j n_j / K after the event; +infinity while pending > 0 */
  double rho_hat;            /* target utilisation in force after the event */
  double lambda;             /* latency weight in force after the event */
  double volatility;         /* sigma(t) */
} ts_sched_decision;

typedef struct ts_sched ts_sched;

/* Creates a scheduler; *out receives the handle (free with ts_sched_destroy). */
int ts_sched_create(const ts_sched_params* params, ts_sched** out);
void ts_sched_destroy(ts_sched* s);

/* One decision epoch t of Alg. 1.  The epoch first applies `n` session changes in order (a time
 * bin of the trace may hold several arrivals and activations, and `n` may be 0 for a bin with
 * none): kinds[c] in ts_sched_event_kind, ids[c] the session, state_bytes[c] its state size in
 * bytes (used by ARRIVE for the migration cost; state_bytes may be NULL for all zeros).  Then it
 * runs place -> scale -> place/resize and finally records a_t = the number of ARRIVE and ACTIVATE
 * changes in the epoch for the volatility window.  If any change is invalid (unknown session,
 * duplicate arrival, ACTIVATE of an active or IDLE of an idle session, negative size, unknown
 * kind) the call returns the error and the scheduler is left exactly as before.  `out` may be
 * NULL. */
int ts_sched_step(ts_sched* s, int32_t n, const int32_t* kinds, const int64_t* ids,
                  const int64_t* state_bytes, ts_sched_decision* out);

/* Current placement: writes up to `cap` (session id, GPU id or -1 if unplaced) pairs in
 * increasing session id order; *count receives the number of sessions. */
int ts_sched_placement(const ts_sched* s, int64_t* ids, int32_t* gpus, int32_t cap,
                       int32_t* count);

/* Current GPUs: writes up to `cap` (GPU id, sessions on it) pairs in increasing GPU id order;
 * *count receives the number of GPUs (= M). */
int ts_sched_gpus(const ts_sched* s, int32_t* gpu_ids, int32_t* loads, int32_t cap,
                  int32_t* count);

int ts_sched_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* TS_SCHED_H */
