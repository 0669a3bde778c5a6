// driver.cpp -- the host-side argument checks of libts_attn's C ABI (csrc/ts_attn.cpp and
// csrc/attn_plan.cpp) under AddressSanitizer and UBSan, built with g++ by
// tests/test_abi_sanitized.py together with launch_stubs.cpp (no device code).  Every entry
// point is called over a grid of extreme sizes, head counts, head dims, scales, pointer
// alignments and overlaps; pointers are fake and never dereferenced by the checks.  A call that
// passes the checks goes on to device set-up, which fails here (no GPU, or the stubbed kernel
// configuration), so nothing is launched.  Checks: every call returns a defined status, and
// the cases with a known answer (oversized heads, oversized segments, empty problems, bad
// pointers) return it.  Exit status 0 when all hold; UBSan aborts on any undefined behaviour.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <limits>
#include <vector>

#include "ts_attn.h"

namespace {

int g_fail = 0;
int64_t g_calls = 0;

bool known_status(int s) { return s >= TS_OK && s <= TS_ERR_SCRATCH; }

void expect(bool cond, const char* what, long long a, long long b, long long c) {
  if (!cond) {
    if (g_fail < 20) std::fprintf(stderr, "FAIL %s (%lld, %lld, %lld)\n", what, a, b, c);
    ++g_fail;
  }
}

void* fake(uintptr_t a) { return reinterpret_cast<void*>(a); }

}  // namespace

int main() {
  const int32_t I32MIN = std::numeric_limits<int32_t>::min(), I32MAX = std::numeric_limits<int32_t>::max();
  const std::vector<int32_t> sizes = {I32MIN, -1, 0, 1, 63, 64, 255, 256, 257, 65279, 65280,
                                      1 << 24, 1 << 27, 1 << 30, I32MAX};
  const std::vector<int32_t> heads = {I32MIN, -1, 0, 1, 40, 1 << 16, 1 << 23, I32MAX};
  const std::vector<int32_t> dims = {-1, 0, 64, 100, 128};
  const float nan = std::numeric_limits<float>::quiet_NaN(), inf = std::numeric_limits<float>::infinity();
  const std::vector<float> scales = {0.0f, 0.088f, -1.0f, nan, inf, -inf};
  // q, k, v, o far apart (no overlap for any size below 2^44), 16-byte aligned
  void *q = fake(1ull << 44), *k = fake(2ull << 44), *v = fake(3ull << 44), *o = fake(4ull << 44);
  int32_t* cu = static_cast<int32_t*>(fake(5ull << 44));
  float* lse = static_cast<float*>(fake(6ull << 44));

  // dense: ts_attn_fwd(B, L, H, d, scale)
  for (int32_t B : sizes)
    for (int32_t L : sizes)
      for (int32_t H : heads)
        for (int32_t d : dims)
          for (float sc : scales) {
            const int s = ts_attn_fwd(q, k, v, o, B, L, H, d, sc, nullptr);
            ++g_calls;
            expect(known_status(s), "dense status", B, L, H);
            const bool shape_ok = B >= 0 && L >= 0 && H >= 1;
            if (shape_ok && (d == 64 || d == 128) && std::isfinite(sc)) {
              const int64_t row = (int64_t)H * d * 2;
              if (row * 256 >= ((int64_t)1 << 31)) expect(s == TS_ERR_SHAPE, "dense oversized head", B, L, H);
              else if (((int64_t)L + 256) * row >= ((int64_t)1 << 31)) expect(s == TS_ERR_SHAPE, "dense oversized L", B, L, H);
            }
            if (!shape_ok) expect(s != TS_OK, "dense negative accepted", B, L, H);
          }
  // null / misaligned / aliased pointers on a valid shape
  expect(ts_attn_fwd(nullptr, k, v, o, 1, 64, 2, 64, 1.0f, nullptr) == TS_ERR_NULL, "null q", 0, 0, 0);
  expect(ts_attn_fwd(fake((1ull << 44) + 8), k, v, o, 1, 64, 2, 64, 1.0f, nullptr) == TS_ERR_ALIGN, "misaligned", 0, 0, 0);
  expect(ts_attn_fwd(q, k, v, fake((1ull << 44) + 4096), 1, 64, 2, 64, 1.0f, nullptr) == TS_ERR_ALIAS, "alias", 0, 0, 0);
  expect(ts_attn_fwd(q, k, v, o, 0, 64, 2, 64, 1.0f, nullptr) == TS_OK, "empty batch", 0, 0, 0);
  expect(ts_attn_fwd(q, k, v, o, 3, 0, 2, 64, 1.0f, nullptr) == TS_OK, "empty sequence", 0, 0, 0);

  // packed: ts_attn_fwd_varlen(nseq, max_seqlen, total, H, d)
  for (int32_t nseq : sizes)
    for (int32_t maxl : sizes)
      for (int32_t total : sizes)
        for (int32_t H : heads)
          for (int32_t d : dims) {
            const int s = ts_attn_fwd_varlen(q, k, v, o, cu, nseq, maxl, total, H, d, 0.1f, nullptr);
            ++g_calls;
            expect(known_status(s), "varlen status", nseq, maxl, total);
            if (H == I32MAX && (d == 64 || d == 128) && nseq >= 0 && maxl >= 0 && total >= 0)
              expect(s == TS_ERR_SHAPE, "varlen huge H", nseq, maxl, total);
          }
  expect(ts_attn_fwd_varlen(q, k, v, o, nullptr, 1, 64, 64, 2, 64, 1.0f, nullptr) == TS_ERR_NULL, "null cu", 0, 0, 0);
  // tensors of zero rows may be NULL (an empty torch tensor has a NULL data pointer)
  expect(ts_attn_fwd(nullptr, nullptr, nullptr, nullptr, 0, 64, 2, 64, 1.0f, nullptr) == TS_OK, "empty dense, NULL tensors", 0, 0, 0);
  expect(ts_attn_fwd_varlen(nullptr, nullptr, nullptr, nullptr, cu, 2, 0, 0, 2, 64, 1.0f, nullptr) == TS_OK, "empty packed, NULL tensors", 0, 0, 0);
  expect(ts_attn_fwd_varlen(nullptr, k, v, o, cu, 1, 64, 64, 2, 64, 1.0f, nullptr) == TS_ERR_NULL, "NULL q with rows", 0, 0, 0);
  expect(ts_attn_fwd_kvcache(nullptr, nullptr, nullptr, nullptr, nullptr, cu, cu, 1, 0, 0, 0, 0, 2, 64, 1.0f, 0, nullptr) == TS_OK, "empty chunk, NULL tensors", 0, 0, 0);
  expect(ts_attn_fwd_kvcache(q, nullptr, nullptr, o, nullptr, cu, cu, 1, 64, 0, 64, 0, 2, 80, 1.0f, 0, nullptr) == TS_ERR_HEAD_DIM, "NULL k/v of zero rows", 0, 0, 0);
  expect(ts_attn_fwd_kvcache(q, nullptr, v, o, nullptr, cu, cu, 1, 64, 64, 64, 64, 2, 64, 1.0f, 0, nullptr) == TS_ERR_NULL, "NULL k with rows", 0, 0, 0);

  // chunk vs cache: ts_attn_fwd_kvcache(nseq, max_q, max_k, total_q, total_k, H, d, splits)
  const std::vector<int32_t> few = {I32MIN, -1, 0, 1, 257, 65279, 1 << 27, I32MAX};
  const std::vector<int32_t> splits = {-1, 0, 1, 16, 17, I32MAX};
  for (int32_t nseq : few)
    for (int32_t mq : few)
      for (int32_t mk : few)
        for (int32_t tq : few)
          for (int32_t tk : few)
            for (int32_t H : heads)
              for (int32_t ns : splits) {
                const int s = ts_attn_fwd_kvcache(q, k, v, o, (ns & 1) ? lse : nullptr, cu, cu, nseq, mq,
                                                  mk, tq, tk, H, 128, 0.1f, ns, nullptr);
                ++g_calls;
                expect(known_status(s), "kv status", nseq, mq, H);
                if (ns < 0 || ns > 16) expect(s != TS_OK, "bad splits accepted", nseq, ns, H);
                const int s2 = ts_attn_fwd_kvcache_noalloc(q, k, v, o, (ns & 1) ? lse : nullptr, cu, cu,
                                                           nseq, mq, mk, tq, tk, H, 128, 0.1f, ns,
                                                           nullptr);
                ++g_calls;
                expect(known_status(s2), "kv noalloc status", nseq, mq, H);
                // the same checks, plus the scratch bound of a forced split count
                expect(s2 == s || s2 == TS_ERR_SCRATCH, "kv noalloc differs", nseq, tq, ns);
              }
  expect(ts_attn_fwd_kvcache(q, k, v, o, static_cast<float*>(fake((6ull << 44) + 2)), cu, cu, 1, 64, 64, 64, 64, 2, 64, 1.0f, 0, nullptr) ==
             TS_ERR_ALIGN, "misaligned lse", 0, 0, 0);
  // allocation-free chunk call: 2 splits of 32768 query rows at H = 2, d = 128 need 64 MiB of
  // partials, more than its 32 MiB scratch; 4096 rows (8 MiB) fit
  expect(ts_attn_fwd_kvcache_noalloc(q, k, v, o, nullptr, cu, cu, 1, 32768, 64, 32768, 64, 2, 128, 1.0f, 2, nullptr) ==
             TS_ERR_SCRATCH, "noalloc scratch bound", 0, 0, 0);
  expect(ts_attn_fwd_kvcache_noalloc(nullptr, nullptr, nullptr, nullptr, nullptr, cu, cu, 1, 0, 0, 0, 0, 2, 64, 1.0f, 0, nullptr) == TS_OK,
         "noalloc empty chunk", 0, 0, 0);

  // state copy: ranges with extreme offsets and sizes, extreme buffer sizes
  const int64_t I64MAX = std::numeric_limits<int64_t>::max();
  const std::vector<int64_t> off = {-16, -1, 0, 16, 1 << 20, (int64_t)1 << 40, I64MAX - 15, I64MAX};
  const std::vector<int64_t> bufs = {-1, 0, 16, (int64_t)1 << 40, I64MAX};
  for (int64_t sb : bufs)
    for (int64_t db : bufs)
      for (int64_t so : off)
        for (int64_t d_o : off)
          for (int64_t n : off) {
            const int64_t r[3] = {so, d_o, n};
            const int s = ts_state_copy(q, sb, o, db, r, 1, nullptr);
            ++g_calls;
            expect(known_status(s), "copy status", so, d_o, n);
            if (sb >= 0 && db >= 0 && (so < 0 || d_o < 0 || n < 0)) expect(s != TS_OK, "copy negative", so, d_o, n);
          }
  expect(ts_state_copy(q, 64, o, 64, nullptr, 1, nullptr) == TS_ERR_NULL, "null ranges", 0, 0, 0);
  expect(ts_state_copy(q, 64, o, 64, nullptr, 0, nullptr) == TS_OK, "no ranges", 0, 0, 0);

  for (int s = -2; s <= TS_ERR_CAPTURE + 2; ++s) expect(ts_attn_status_str(s) != nullptr, "status string", s, 0, 0);
  std::printf("calls %lld, failures %d\n", (long long)g_calls, g_fail);
  return g_fail == 0 ? 0 : 1;
}
