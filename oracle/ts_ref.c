/*
 * ts_ref.c -- fp64 CPU oracle for segment-local, non-causal multi-head softmax attention.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may link, load or call this file;
 * only the tests, the smoke check and the benchmark's CPU-baseline leg use it.  It shares no
 * code, header, table or helper with the HIP library.
 *
 * What it computes (the plain definition, not a tiled algorithm):
 *   The paper's runtime serves several sessions on one GPU by packing the ready sessions into
 *   one coalesced chunk batch and running the model once for the batch (Sec. 3.1, "Concurrent
 *   chunk execution"), while each session keeps its state in an isolated per-session region
 *   (Sec. 6.1, "Session memory layout").  Inside the model's attention this makes every token
 *   attend only to the tokens of its own session: segment s of the packed batch is the token
 *   range [cu[s], cu[s+1]).  For token t of segment s, head h and channel c:
 *       z_j      = scale * sum_{c'} Q[t,h,c'] * K[j,h,c']      for every j in segment s
 *       m        = max_j z_j
 *       w_j      = exp(z_j - m)
 *       O[t,h,c] = (sum_j w_j * V[j,h,c]) / (sum_j w_j)
 *   Attention is non-causal: j ranges over the whole segment, before and after t.  Subtracting
 *   m changes nothing in exact arithmetic; it only keeps exp() finite.
 *
 * Arithmetic: everything in double, libm exp(), plain left-to-right summation.
 * Inputs: either doubles, or bfloat16 bit patterns (uint16) widened exactly (bf16 -> fp32 is a
 * 16-bit left shift, fp32 -> double is exact).  Layout: token-major [T][H][d], contiguous.
 * Rows are independent, so callers may ask for any subset of (token, head) rows; the row loop
 * is an OpenMP parallel for.
 *
 * A second entry point computes chunk queries against per-session key/value ranges with
 * the log-sum-exp of every row (defined above ts_ref_attn_kv_rows_bf16).
 *
 * Parity pins (tests/test_oracle.py, tests/test_oracle_kv.py): mpmath brute force at 50
 * digits, torch's CPU float64 scaled_dot_product_attention per segment, scipy's logsumexp,
 * closed forms (one key, two keys, identical keys, constant V, dominant key), invariants (shift,
 * permutation, segment independence, convex hull, merging two key ranges by their lse).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { REF_OK = 0, REF_ERR_ARG = 1, REF_ERR_SEGMENTS = 2, REF_ERR_ROW = 3, REF_ERR_NOMEM = 4 };

/* bfloat16 bit pattern -> double, exact. */
static double widen_bf16(uint16_t bits) {
  uint32_t u = ((uint32_t)bits) << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/* Index of the segment holding token t: the s with cu[s] <= t < cu[s+1].  Empty segments
 * (cu[s] == cu[s+1]) hold no token and are never returned. */
static int32_t find_segment(const int32_t* cu, int32_t nseq, int64_t t) {
  int32_t lo = 0, hi = nseq; /* invariant: cu[lo] <= t < cu[hi] */
  while (hi - lo > 1) {
    int32_t mid = lo + (hi - lo) / 2;
    if ((int64_t)cu[mid] <= t) lo = mid; else hi = mid;
  }
  return lo;
}

static int check_segments(const int32_t* cu, int32_t nseq) {
  if (cu[0] != 0) return REF_ERR_SEGMENTS;
  for (int32_t s = 0; s < nseq; s++)
    if (cu[s + 1] < cu[s]) return REF_ERR_SEGMENTS;
  return REF_OK;
}

/* One input element, either from a double array or a bf16 array. */
typedef struct {
  const double* f64;
  const uint16_t* b16;
} tensor_t;

static inline double elem(tensor_t x, int64_t i) { return x.f64 ? x.f64[i] : widen_bf16(x.b16[i]); }

/* Computes one output row O[t,h,:] into out[0..d); z is scratch of length >= segment length. */
static void attend_row(tensor_t q, tensor_t k, tensor_t v, const int32_t* cu, int32_t nseq,
                       int32_t H, int32_t d, double scale, int64_t t, int32_t h, double* z,
                       double* out, double* weights_out) {
  int32_t s = find_segment(cu, nseq, t);
  int64_t j0 = cu[s], j1 = cu[s + 1];
  int64_t row_stride = (int64_t)H * d;
  int64_t qoff = t * row_stride + (int64_t)h * d;

  /* scores z_j = scale * <Q[t,h,:], K[j,h,:]> */
  double m = -INFINITY;
  for (int64_t j = j0; j < j1; j++) {
    int64_t koff = j * row_stride + (int64_t)h * d;
    double dot = 0.0;
    for (int32_t c = 0; c < d; c++) dot += elem(q, qoff + c) * elem(k, koff + c);
    double zj = scale * dot;
    z[j - j0] = zj;
    if (zj > m) m = zj;
  }
  /* weights w_j = exp(z_j - m) and their sum */
  double den = 0.0;
  for (int64_t j = j0; j < j1; j++) {
    double w = exp(z[j - j0] - m);
    z[j - j0] = w;
    den += w;
  }
  /* O = sum_j w_j V[j] / sum_j w_j */
  for (int32_t c = 0; c < d; c++) out[c] = 0.0;
  for (int64_t j = j0; j < j1; j++) {
    int64_t voff = j * row_stride + (int64_t)h * d;
    double w = z[j - j0];
    for (int32_t c = 0; c < d; c++) out[c] += w * elem(v, voff + c);
  }
  for (int32_t c = 0; c < d; c++) out[c] /= den;
  if (weights_out)
    for (int64_t j = j0; j < j1; j++) weights_out[j - j0] = z[j - j0] / den;
}

static int attn_rows(tensor_t q, tensor_t k, tensor_t v, const int32_t* cu, int32_t nseq,
                     int32_t H, int32_t d, double scale, const int64_t* row_t,
                     const int32_t* row_h, int64_t nrows, double* out) {
  if (!cu || !out || nseq < 1 || H < 1 || d < 1 || nrows < 0) return REF_ERR_ARG;
  if ((nrows > 0) && (!row_t || !row_h)) return REF_ERR_ARG;
  int rc = check_segments(cu, nseq);
  if (rc) return rc;
  int64_t T = cu[nseq];
  int32_t maxlen = 0;
  for (int32_t s = 0; s < nseq; s++)
    if (cu[s + 1] - cu[s] > maxlen) maxlen = cu[s + 1] - cu[s];
  for (int64_t r = 0; r < nrows; r++)
    if (row_t[r] < 0 || row_t[r] >= T || row_h[r] < 0 || row_h[r] >= H) return REF_ERR_ROW;

  int failed = 0;
#pragma omp parallel
  {
    double* z = (double*)malloc(sizeof(double) * (size_t)(maxlen > 0 ? maxlen : 1));
    if (!z) {
#pragma omp atomic write
      failed = 1;
    }
#pragma omp for schedule(dynamic, 4)
    for (int64_t r = 0; r < nrows; r++) {
      if (z) attend_row(q, k, v, cu, nseq, H, d, scale, row_t[r], row_h[r], z, out + r * d, NULL);
    }
    free(z);
  }
  return failed ? REF_ERR_NOMEM : REF_OK;
}

/* Rows of O for (token row_t[r], head row_h[r]), r < nrows, from bf16 inputs; out is [nrows][d]. */
int ts_ref_attn_rows_bf16(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                          const int32_t* cu_seqlens, int32_t nseq, int32_t H, int32_t d,
                          double scale, const int64_t* row_t, const int32_t* row_h, int64_t nrows,
                          double* out) {
  if (!q || !k || !v) return REF_ERR_ARG;
  tensor_t tq = {NULL, q}, tk = {NULL, k}, tv = {NULL, v};
  return attn_rows(tq, tk, tv, cu_seqlens, nseq, H, d, scale, row_t, row_h, nrows, out);
}

/* Same, from double inputs. */
int ts_ref_attn_rows_f64(const double* q, const double* k, const double* v,
                         const int32_t* cu_seqlens, int32_t nseq, int32_t H, int32_t d,
                         double scale, const int64_t* row_t, const int32_t* row_h, int64_t nrows,
                         double* out) {
  if (!q || !k || !v) return REF_ERR_ARG;
  tensor_t tq = {q, NULL}, tk = {k, NULL}, tv = {v, NULL};
  return attn_rows(tq, tk, tv, cu_seqlens, nseq, H, d, scale, row_t, row_h, nrows, out);
}

/* Softmax weights w_j / sum w of one row (token t, head h) over its segment, from double
 * inputs; weights has room for the segment length.  Also writes the row's output to out[d]. */
int ts_ref_attn_weights_f64(const double* q, const double* k, const double* v,
                            const int32_t* cu_seqlens, int32_t nseq, int32_t H, int32_t d,
                            double scale, int64_t t, int32_t h, double* weights, double* out) {
  if (!q || !k || !v || !cu_seqlens || !weights || !out || nseq < 1 || H < 1 || d < 1)
    return REF_ERR_ARG;
  int rc = check_segments(cu_seqlens, nseq);
  if (rc) return rc;
  if (t < 0 || t >= cu_seqlens[nseq] || h < 0 || h >= H) return REF_ERR_ROW;
  int32_t s = find_segment(cu_seqlens, nseq, t);
  int32_t len = cu_seqlens[s + 1] - cu_seqlens[s];
  double* z = (double*)malloc(sizeof(double) * (size_t)len);
  if (!z) return REF_ERR_NOMEM;
  tensor_t tq = {q, NULL}, tk = {k, NULL}, tv = {v, NULL};
  attend_row(tq, tk, tv, cu_seqlens, nseq, H, d, scale, t, h, z, out, weights);
  free(z);
  return REF_OK;
}

/*
 * Chunk queries against per-session key/value ranges, with the log-sum-exp of every row.
 *
 * A chunk-autoregressive streaming model generates each new chunk conditioned on the cached
 * state of the session's earlier chunks (Sec. 2, "Streaming video generation workflow"); that
 * cache is part of the session's isolated state region (Sec. 6.1, "Session memory layout"), and
 * one model call serves the coalesced batch of ready sessions (Sec. 3.1).  Segment s of such a
 * batch has its queries at rows [cu_q[s], cu_q[s+1]) of Q and its keys and values at rows
 * [cu_k[s], cu_k[s+1]) of K and V -- typically the session's cached tokens followed by the
 * chunk's own -- and every query attends to every key of its segment.  For query row t of
 * segment s, head h and channel c:
 *     z_j      = scale * sum_{c'} Q[t,h,c'] * K[j,h,c']     for j in [cu_k[s], cu_k[s+1])
 *     m        = max_j z_j
 *     lse      = m + log(sum_j exp(z_j - m))                (= log sum_j exp z_j)
 *     O[t,h,c] = sum_j exp(z_j - m) V[j,h,c] / sum_j exp(z_j - m)
 * A segment without keys has the empty sum: O = 0 and lse = -inf.  With cu_q == cu_k this is
 * the self-attention above.  Same arithmetic rules: double, libm exp/log, left-to-right sums.
 */
static void attend_kv_row(tensor_t q, tensor_t k, tensor_t v, const int32_t* cu_q,
                          const int32_t* cu_k, int32_t nseq, int32_t H, int32_t d, double scale,
                          int64_t t, int32_t h, double* z, double* out, double* lse) {
  int32_t s = find_segment(cu_q, nseq, t);
  int64_t kb = cu_k[s], ke = cu_k[s + 1];
  int64_t row_stride = (int64_t)H * d;
  int64_t qrow = t * row_stride + (int64_t)h * d;
  for (int32_t c = 0; c < d; c++) out[c] = 0.0;
  if (ke == kb) {
    *lse = -INFINITY;
    return;
  }
  /* scores and their maximum */
  double m = -INFINITY;
  for (int64_t j = kb; j < ke; j++) {
    int64_t krow = j * row_stride + (int64_t)h * d;
    double dot = 0.0;
    for (int32_t c = 0; c < d; c++) dot += elem(q, qrow + c) * elem(k, krow + c);
    z[j - kb] = scale * dot;
    if (z[j - kb] > m) m = z[j - kb];
  }
  /* unnormalised weights, their sum, the weighted sum of V rows */
  double den = 0.0;
  for (int64_t j = kb; j < ke; j++) {
    double w = exp(z[j - kb] - m);
    den += w;
    int64_t vrow = j * row_stride + (int64_t)h * d;
    for (int32_t c = 0; c < d; c++) out[c] += w * elem(v, vrow + c);
  }
  for (int32_t c = 0; c < d; c++) out[c] = out[c] / den;
  *lse = m + log(den);
}

static int attn_kv_rows(tensor_t q, tensor_t k, tensor_t v, const int32_t* cu_q,
                        const int32_t* cu_k, int32_t nseq, int32_t H, int32_t d, double scale,
                        const int64_t* row_t, const int32_t* row_h, int64_t nrows, double* out,
                        double* lse) {
  if (!cu_q || !cu_k || !out || !lse || nseq < 1 || H < 1 || d < 1 || nrows < 0)
    return REF_ERR_ARG;
  if ((nrows > 0) && (!row_t || !row_h)) return REF_ERR_ARG;
  int rc = check_segments(cu_q, nseq);
  if (rc) return rc;
  rc = check_segments(cu_k, nseq);
  if (rc) return rc;
  int64_t Tq = cu_q[nseq];
  int32_t maxlen = 0;
  for (int32_t s = 0; s < nseq; s++)
    if (cu_k[s + 1] - cu_k[s] > maxlen) maxlen = cu_k[s + 1] - cu_k[s];
  for (int64_t r = 0; r < nrows; r++)
    if (row_t[r] < 0 || row_t[r] >= Tq || row_h[r] < 0 || row_h[r] >= H) return REF_ERR_ROW;

  int failed = 0;
#pragma omp parallel
  {
    double* z = (double*)malloc(sizeof(double) * (size_t)(maxlen > 0 ? maxlen : 1));
    if (!z) {
#pragma omp atomic write
      failed = 1;
    }
#pragma omp for schedule(dynamic, 4)
    for (int64_t r = 0; r < nrows; r++) {
      if (z)
        attend_kv_row(q, k, v, cu_q, cu_k, nseq, H, d, scale, row_t[r], row_h[r], z, out + r * d,
                      lse + r);
    }
    free(z);
  }
  return failed ? REF_ERR_NOMEM : REF_OK;
}

/* Rows (token row_t[r] of q, head row_h[r]) of chunk-vs-cache attention from bf16 inputs:
 * q is [Tq][H][d] with Tq = cu_q[nseq], k and v are [Tk][H][d] with Tk = cu_k[nseq].
 * out is [nrows][d], lse is [nrows]. */
int ts_ref_attn_kv_rows_bf16(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                             const int32_t* cu_q, const int32_t* cu_k, int32_t nseq, int32_t H,
                             int32_t d, double scale, const int64_t* row_t, const int32_t* row_h,
                             int64_t nrows, double* out, double* lse) {
  if (!q || !k || !v) return REF_ERR_ARG;
  tensor_t tq = {NULL, q}, tk = {NULL, k}, tv = {NULL, v};
  return attn_kv_rows(tq, tk, tv, cu_q, cu_k, nseq, H, d, scale, row_t, row_h, nrows, out, lse);
}

/* Same, from double inputs. */
int ts_ref_attn_kv_rows_f64(const double* q, const double* k, const double* v,
                            const int32_t* cu_q, const int32_t* cu_k, int32_t nseq, int32_t H,
                            int32_t d, double scale, const int64_t* row_t, const int32_t* row_h,
                            int64_t nrows, double* out, double* lse) {
  if (!q || !k || !v) return REF_ERR_ARG;
  tensor_t tq = {q, NULL}, tk = {k, NULL}, tv = {v, NULL};
  return attn_kv_rows(tq, tk, tv, cu_q, cu_k, nseq, H, d, scale, row_t, row_h, nrows, out, lse);
}

/* Number of OpenMP threads a parallel region of the oracle uses. */
int ts_ref_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}
