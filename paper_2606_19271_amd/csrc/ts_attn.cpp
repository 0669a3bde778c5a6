// ts_attn.cpp -- the C ABI of libts_attn.so (declared in include/ts_attn.h): argument checks,
// per-device set-up, the workspace of packed batches, and the launches.
#include "ts_attn.h"

#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <mutex>

#include "attn_launch.h"

namespace {

constexpr int kMaxDevices = 64;
constexpr int64_t kByteLimit = (int64_t)1 << 31;
constexpr int64_t kGridLimit = (int64_t)1 << 23;  // workgroups per launch (x 512 threads < 2^32)
constexpr int32_t kMaxSplits = 16;                 // key ranges per query tile of a split call

struct DeviceState {
  std::once_flag once;
  std::atomic<bool> set_up{false};  // init_device has run (whatever its outcome)
  int status = TS_ERR_UNSUPPORTED;  // TS_OK once the device is known to be usable
  int dev = -1;
  int xcd_chunk = 32;
  int cus = 256;
  void* scratch = nullptr;          // this device's copy of the static scratch array
  std::once_flag pool_once;         // the pool is made by the first call that needs it
  hipMemPool_t pool = nullptr;      // null if its creation failed
  // The workspace of the packed and chunk calls (see run_packed): grown when a call needs more,
  // held until the process ends; `done` is recorded after each call that used it.
  std::mutex ws_mu;
  void* ws = nullptr;
  size_t ws_size = 0;
  hipEvent_t ws_done = nullptr;
  bool ws_used = false;
};

DeviceState g_dev[kMaxDevices];

// One-time set-up of a device, with that device current: architecture, kernel attributes and the
// device address of the static scratch array (each device holds its own copy of the array).
void init_device(int dev, DeviceState* st) {
  hipDeviceProp_t p;
  st->dev = dev;
  if (hipGetDeviceProperties(&p, dev) != hipSuccess) { st->status = TS_ERR_HIP; return; }
  if (strncmp(p.gcnArchName, "gfx950", 6) != 0) { st->status = TS_ERR_UNSUPPORTED; return; }
  // gfx950: 8 XCDs; one 512-thread workgroup resides per CU.
  st->xcd_chunk = p.multiProcessorCount / 8 > 0 ? p.multiProcessorCount / 8 : 1;
  st->cus = p.multiProcessorCount;
  if (tsattn::configure_kernels() != hipSuccess) { st->status = TS_ERR_HIP; return; }
  void* ptr = nullptr;
  if (tsattn::scratch_address(&ptr) != hipSuccess || ptr == nullptr) {
    (void)hipGetLastError();
    st->status = TS_ERR_HIP;
    return;
  }
  st->scratch = ptr;
  st->status = TS_OK;
}

// The device's stream-ordered memory pool for the workspaces of packed calls too large for the
// cached workspace (see run_packed), created on first use (never under capture: those calls refuse
// a capturing stream before this).
hipMemPool_t device_pool(DeviceState* st) {
  std::call_once(st->pool_once, [st] {
    hipMemPoolProps props;
    memset(&props, 0, sizeof props);
    props.allocType = hipMemAllocationTypePinned;
    props.location.type = hipMemLocationTypeDevice;
    props.location.id = st->dev;
    hipMemPool_t pool = nullptr;
    if (hipMemPoolCreate(&pool, &props) != hipSuccess) { (void)hipGetLastError(); return; }
    uint64_t keep = UINT64_MAX;  // keep freed workspaces in the pool between calls
    if (hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &keep) != hipSuccess) {
      (void)hipGetLastError();
      (void)hipMemPoolDestroy(pool);
      return;
    }
    st->pool = pool;
  });
  return st->pool;
}

// Whether stream s is recording a HIP graph.  A failed query (which leaves an error behind that
// a later launch check would report) is cleared and read as "not capturing".
bool capturing(hipStream_t s) {
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(s, &cs) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  return cs != hipStreamCaptureStatusNone;
}

// The calling thread's current device, initialised once -- never under stream capture, where
// the set-up's pool creation and kernel attributes have no place (TS_ERR_CAPTURE).
DeviceState* current_device(int* status, hipStream_t s) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    *status = TS_ERR_UNSUPPORTED;
    return nullptr;
  }
  DeviceState* st = &g_dev[dev];
  if (!st->set_up.load(std::memory_order_acquire) && capturing(s)) {
    *status = TS_ERR_CAPTURE;
    return nullptr;
  }
  std::call_once(st->once, [dev, st] {
    init_device(dev, st);
    st->set_up.store(true, std::memory_order_release);
  });
  *status = st->status;
  return st->status == TS_OK ? st : nullptr;
}

bool misaligned(const void* p) { return ((uintptr_t)p & 15u) != 0; }

bool overlaps(const void* a, const void* b, int64_t bytes) {
  uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
  return x < y + (uintptr_t)bytes && y < x + (uintptr_t)bytes;
}

// [a, a + na) and [b, b + nb) share a byte (empty ranges share none).
bool ranges_overlap(const void* a, int64_t na, const void* b, int64_t nb) {
  uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
  return na > 0 && nb > 0 && x < y + (uintptr_t)nb && y < x + (uintptr_t)na;
}

// Shared checks of both entry points; tokens = rows of q/k/v/o, longest = longest segment.
// Tensors of zero rows are never dereferenced, so their pointers may be NULL (torch gives an
// empty tensor a NULL data pointer).
int check_common(const void* q, const void* k, const void* v, const void* o, int64_t tokens,
                 int64_t longest, int32_t H, int32_t d, float scale) {
  if (tokens > 0 && (!q || !k || !v || !o)) return TS_ERR_NULL;
  if (H < 1 || tokens < 0 || longest < 0) return TS_ERR_SHAPE;
  if (d != 64 && d != 128) return TS_ERR_HEAD_DIM;
  if (!isfinite(scale)) return TS_ERR_SCALE;
  if (misaligned(q) || misaligned(k) || misaligned(v) || misaligned(o)) return TS_ERR_ALIGN;
  const int64_t row_bytes = (int64_t)H * d * 2;
  // (longest + 256) * row_bytes < kByteLimit, written so that nothing overflows for any H; it
  // also bounds row_bytes below 2^23, so tokens * row_bytes fits easily
  if (longest + 256 > (kByteLimit - 1) / row_bytes) return TS_ERR_SHAPE;
  if (tokens > (int64_t)1 << 31) return TS_ERR_SHAPE;
  const int64_t bytes = tokens * row_bytes;
  if (overlaps(o, q, bytes) || overlaps(o, k, bytes) || overlaps(o, v, bytes)) return TS_ERR_ALIAS;
  return TS_OK;
}

bool validate_mode() {
  const char* e = getenv("TS_ATTN_VALIDATE");
  return e && e[0] == '1';
}

// Checks of the chunk-vs-cache call: q/o hold tq rows, k/v tk rows; segments are at most
// max_q queries and max_k keys long.  As in check_common, q/o may be NULL when tq = 0 and k/v
// when tk = 0 (queries without keys read no key: O = 0, lse = -inf).
int check_kv(const void* q, const void* k, const void* v, const void* o, const float* lse,
             int64_t tq, int64_t tk, int64_t max_q, int64_t max_k, int32_t H, int32_t d,
             float scale) {
  if ((tq > 0 && (!q || !o)) || (tk > 0 && (!k || !v))) return TS_ERR_NULL;
  if (H < 1 || tq < 0 || tk < 0 || max_q < 0 || max_k < 0) return TS_ERR_SHAPE;
  if (d != 64 && d != 128) return TS_ERR_HEAD_DIM;
  if (!isfinite(scale)) return TS_ERR_SCALE;
  if (misaligned(q) || misaligned(k) || misaligned(v) || misaligned(o)) return TS_ERR_ALIGN;
  if (((uintptr_t)lse & 3u) != 0) return TS_ERR_ALIGN;
  const int64_t row_bytes = (int64_t)H * d * 2;
  if (max_q + 256 > (kByteLimit - 1) / row_bytes || max_k + 256 > (kByteLimit - 1) / row_bytes)
    return TS_ERR_SHAPE;  // as in check_common, without overflow for any H
  if (tq > (int64_t)1 << 31 || tk > (int64_t)1 << 31) return TS_ERR_SHAPE;
  const int64_t qb = tq * row_bytes, kb = tk * row_bytes;
  if (ranges_overlap(o, qb, q, qb) || ranges_overlap(o, qb, k, kb) || ranges_overlap(o, qb, v, kb))
    return TS_ERR_ALIAS;
  if (lse) {
    const int64_t lb = tq * H * 4;
    if (ranges_overlap(lse, lb, q, qb) || ranges_overlap(lse, lb, k, kb) ||
        ranges_overlap(lse, lb, v, kb) || ranges_overlap(lse, lb, o, qb))
      return TS_ERR_ALIAS;
  }
  return TS_OK;
}

// Key ranges per query tile when the caller leaves the choice to the library.  One 512-thread
// workgroup runs per CU, so `items` work items take ceil(items / cus) rounds, each as long as
// one item's key tiles.  Query tiles that already fill the GPU are not split (the partials would
// only add traffic); otherwise n minimises rounds(items * n) * ceil(tiles / n), the smallest n
// winning ties, with at least 4 key tiles per range.
int32_t auto_splits(int cus, int32_t total_q, int32_t max_k, int32_t H, int32_t d) {
  const int64_t items = (int64_t)H * ((total_q + tsattn::kQueryTile - 1) / tsattn::kQueryTile);
  const int64_t kt = tsattn::key_tile(d);
  const int64_t tiles = ((int64_t)max_k + kt - 1) / kt;
  if (items <= 0 || items >= cus || tiles < 8) return 1;
  int32_t best = 1;
  int64_t best_cost = INT64_MAX;
  for (int32_t n = 1; n <= kMaxSplits && tiles / n >= 4; ++n) {
    const int64_t rounds = (items * n + cus - 1) / cus;
    const int64_t cost = rounds * ((tiles + n - 1) / n);
    if (cost < best_cost) { best_cost = cost; best = n; }
  }
  return best;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Bytes of device scratch a packed call needs: the plan and, with n > 1 key ranges, the float32
// partial lse [n][tq][H] and O [n][tq][H][d], each part 256-byte aligned.
int64_t scratch_bytes(int32_t nseq, int32_t n, int32_t tq, int32_t H, int32_t d) {
  int64_t b = (int64_t)align256((size_t)tsattn::plan_ints(nseq) * sizeof(int32_t));
  if (n > 1) {
    b += (int64_t)align256((size_t)n * tq * H * sizeof(float));
    b += (int64_t)n * tq * H * d * (int64_t)sizeof(float);
  }
  return b;
}

// Points a.plan (and, for a split call, a.part_lse / a.part_o) into buf, laid out as in
// scratch_bytes.
void carve(tsattn::PackedArgs& a, char* buf) {
  const size_t plan_bytes = align256((size_t)tsattn::plan_ints(a.nseq) * sizeof(int32_t));
  a.plan = (int32_t*)buf;
  if (a.n_split > 1) {
    const size_t lse_bytes = align256((size_t)a.n_split * a.total_q * a.H * sizeof(float));
    a.part_lse = (float*)(buf + plan_bytes);
    a.part_o = (float*)(buf + plan_bytes + lse_bytes);
  }
}

// A batch of one segment runs without the planning kernel: its only valid offsets are {0, total_q}
// and {0, total_k}, which the attention and merge kernels check themselves (a mismatch makes the
// call a device-side no-op, as a rejected plan does).  Totals beyond the stated maximum lengths
// admit no valid offsets at all, so such a call is a no-op without any device work.
bool one_segment_possible(const tsattn::PackedArgs& a) {
  return a.total_q <= a.max_q && a.total_k <= a.max_k;
}

// Launch of a packed call whose plan (and partials) sit in buf, and the validation-mode read-back
// of the plan's error flag (a host synchronization, in validation mode only).
int launch_with(tsattn::PackedArgs a, char* buf, bool single, bool validate, hipStream_t s) {
  carve(a, buf);
  if (single) a.plan = nullptr;  // a split call of one segment: partials only
  int rc = tsattn::launch_packed(a, s) == hipSuccess ? TS_OK : TS_ERR_HIP;
  if (rc == TS_OK && validate) {
    int32_t head[2] = {0, 0};
    if (hipMemcpyAsync(head, a.plan, sizeof head, hipMemcpyDeviceToHost, s) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess)
      rc = TS_ERR_HIP;
    else if (head[1] != 0)
      rc = TS_ERR_SEGMENTS;
  }
  return rc;
}

// Workspaces up to this size come from the device's cached workspace; larger ones (long split
// calls) from a stream-ordered pool allocation of their own.
constexpr size_t kWorkspaceCache = (size_t)256 << 20;

int run_packed(DeviceState* st, tsattn::PackedArgs a, hipStream_t s) {
  const bool validate = validate_mode();
  // validation mode keeps the plan, whose error flag it reads back
  const bool single = a.nseq == 1 && !validate;
  if (single) {
    if (!one_segment_possible(a)) return TS_OK;
    if (a.n_split == 1) {  // no device memory at all
      a.plan = nullptr;
      return tsattn::launch_packed(a, s) == hipSuccess ? TS_OK : TS_ERR_HIP;
    }
  }
  const size_t bytes = (size_t)scratch_bytes(a.nseq, a.n_split, a.total_q, a.H, a.d);
  if (bytes <= kWorkspaceCache) {
    // The device's cached workspace.  A stream-ordered allocation per call would be simpler, but
    // HIP's hipMallocFromPoolAsync / hipFreeAsync pair makes the host wait for the stream (every
    // call would block its thread until the GPU caught up).  Instead each call makes its stream
    // wait, on the GPU, for the previous user's event, and records its own: calls on one stream
    // stay in order and calls on different streams take the workspace one after the other.
    std::lock_guard<std::mutex> lock(st->ws_mu);
    if (!st->ws_done && hipEventCreateWithFlags(&st->ws_done, hipEventDisableTiming) != hipSuccess) {
      st->ws_done = nullptr;
      return TS_ERR_HIP;
    }
    if (st->ws_used && hipStreamWaitEvent(s, st->ws_done, 0) != hipSuccess) return TS_ERR_HIP;
    if (st->ws_size < bytes) {  // grow: the old workspace is released once its last user is done
      const size_t want = std::max(bytes, std::min(kWorkspaceCache, 2 * st->ws_size));
      if (st->ws) {
        if (hipEventSynchronize(st->ws_done) != hipSuccess || hipFree(st->ws) != hipSuccess)
          return TS_ERR_HIP;
        st->ws = nullptr;
        st->ws_size = 0;
      }
      if (hipMalloc(&st->ws, want) != hipSuccess) {
        (void)hipGetLastError();
        st->ws = nullptr;
        return TS_ERR_NOMEM;
      }
      st->ws_size = want;
    }
    int rc = launch_with(a, (char*)st->ws, single, validate, s);
    if (hipEventRecord(st->ws_done, s) != hipSuccess && rc == TS_OK) rc = TS_ERR_HIP;
    st->ws_used = true;
    return rc;
  }
  hipMemPool_t pool = device_pool(st);
  if (!pool) return TS_ERR_NOMEM;
  char* buf = nullptr;
  if (hipMallocFromPoolAsync((void**)&buf, bytes, pool, s) != hipSuccess) return TS_ERR_NOMEM;
  int rc = launch_with(a, buf, single, validate, s);
  if (hipFreeAsync(buf, s) != hipSuccess && rc == TS_OK) rc = TS_ERR_HIP;
  return rc;
}

// Checks shared by both chunk-vs-cache entry points (everything but the stream and the memory).
int check_kvcache_call(const void* q, const void* k, const void* v, const void* o,
                       const float* lse, const int32_t* cu_seqlens_q, const int32_t* cu_seqlens_k,
                       int32_t nseq, int32_t max_seqlen_q, int32_t max_seqlen_k, int32_t total_q,
                       int32_t total_k, int32_t H, int32_t d, float scale, int32_t num_splits) {
  if (!cu_seqlens_q || !cu_seqlens_k) return TS_ERR_NULL;
  if (nseq < 0 || num_splits < 0 || num_splits > kMaxSplits) return TS_ERR_SHAPE;
  int rc = check_kv(q, k, v, o, lse, total_q, total_k, max_seqlen_q, max_seqlen_k, H, d, scale);
  if (rc != TS_OK) return rc;
  if (tsattn::packed_grid_bound(total_q, nseq, H, kMaxSplits) >= kGridLimit) return TS_ERR_SHAPE;
  if (tsattn::merge_blocks(total_q, H, d) >= ((int64_t)1 << 31)) return TS_ERR_SHAPE;
  return TS_OK;
}

// Device-visible address of a copy operand: device memory of the current device, or pinned
// (page-locked, mapped) host memory.  Anything else -- pageable host memory, managed memory,
// another device's memory -- is refused, since the copy kernel would fault on it.
int copy_operand(const void* p, int dev, const void** devp, bool* host) {
  hipPointerAttribute_t a;
  if (hipPointerGetAttributes(&a, p) != hipSuccess) {
    (void)hipGetLastError();  // clear the error this lookup leaves behind
    return TS_ERR_MEMORY;
  }
  if (a.type == hipMemoryTypeDevice && a.device == dev) {
    *devp = p;
    *host = false;
    return TS_OK;
  }
  if (a.type == hipMemoryTypeHost && a.devicePointer != nullptr) {
    const char* base_h = (const char*)a.hostPointer;
    const char* base_d = (const char*)a.devicePointer;
    *devp = base_h ? base_d + ((const char*)p - base_h) : base_d;
    *host = true;
    return TS_OK;
  }
  return TS_ERR_MEMORY;
}

// A packed or chunk call on the device's static scratch array: the allocation-free entry point,
// and the allocating ones on a capturing stream (where the workspace's event waits and growth, or
// a pool allocation, have no place).  n = 0 takes the library's choice, lowered until its partial
// results fit the scratch; a forced n that does not fit returns TS_ERR_SCRATCH.  Validation mode
// does not apply: invalid offsets make the call a device-side no-op.
int run_static(DeviceState* st, tsattn::PackedArgs a, int32_t n, hipStream_t s) {
  if (n == 0) {
    n = auto_splits(st->cus, a.total_q, a.max_k, a.H, a.d);
    while (n > 1 && scratch_bytes(a.nseq, n, a.total_q, a.H, a.d) > tsattn::kScratchBytes) --n;
  } else if (scratch_bytes(a.nseq, n, a.total_q, a.H, a.d) > tsattn::kScratchBytes) {
    return TS_ERR_SCRATCH;
  }
  a.n_split = n;
  carve(a, (char*)st->scratch);
  if (a.nseq == 1) {
    if (!one_segment_possible(a)) return TS_OK;
    a.plan = nullptr;
  }
  return tsattn::launch_packed(a, s) == hipSuccess ? TS_OK : TS_ERR_HIP;
}

}  // namespace

extern "C" {

int ts_attn_abi_version(void) { return TS_ATTN_ABI_VERSION; }

const char* ts_attn_status_str(int status) {
  switch (status) {
    case TS_OK: return "TS_OK";
    case TS_ERR_NULL: return "TS_ERR_NULL: a required pointer is NULL";
    case TS_ERR_SHAPE: return "TS_ERR_SHAPE: invalid or oversized shape";
    case TS_ERR_HEAD_DIM: return "TS_ERR_HEAD_DIM: head dim must be 64 or 128";
    case TS_ERR_SCALE: return "TS_ERR_SCALE: scale must be finite";
    case TS_ERR_ALIGN: return "TS_ERR_ALIGN: tensor pointers must be 16-byte aligned";
    case TS_ERR_ALIAS: return "TS_ERR_ALIAS: o overlaps q, k or v";
    case TS_ERR_UNSUPPORTED: return "TS_ERR_UNSUPPORTED: no usable gfx950 device";
    case TS_ERR_HIP: return "TS_ERR_HIP: HIP runtime or launch failure";
    case TS_ERR_NOMEM: return "TS_ERR_NOMEM: device scratch allocation failed";
    case TS_ERR_SEGMENTS: return "TS_ERR_SEGMENTS: invalid cu_seqlens contents";
    case TS_ERR_MEMORY: return "TS_ERR_MEMORY: pointer is neither device memory of the current device nor pinned host memory";
    case TS_ERR_CAPTURE: return "TS_ERR_CAPTURE: this call cannot be recorded into a HIP graph (packed and copy calls, or a device's first call)";
    case TS_ERR_SCRATCH: return "TS_ERR_SCRATCH: the call needs more device scratch than the allocation-free entry point holds";
    default: return "unknown ts_status";
  }
}

int ts_attn_fwd(const void* q, const void* k, const void* v, void* o, int32_t B, int32_t L,
                int32_t H, int32_t d, float scale, void* stream) {
  if (B < 0 || L < 0) return TS_ERR_SHAPE;
  int rc = check_common(q, k, v, o, (int64_t)B * L, L, H, d, scale);
  if (rc != TS_OK) return rc;
  if ((int64_t)B * H * ((L + 255) / 256) >= kGridLimit) return TS_ERR_SHAPE;
  if (B == 0 || L == 0) return TS_OK;
  DeviceState* st = current_device(&rc, (hipStream_t)stream);
  if (!st) return rc;
  tsattn::DenseArgs a{q, k, v, o, B, L, H, d, scale, st->xcd_chunk};
  return tsattn::launch_dense(a, (hipStream_t)stream) == hipSuccess ? TS_OK : TS_ERR_HIP;
}

int ts_attn_fwd_varlen(const void* q, const void* k, const void* v, void* o,
                       const int32_t* cu_seqlens, int32_t nseq, int32_t max_seqlen,
                       int32_t total_tokens, int32_t H, int32_t d, float scale, void* stream) {
  if (!cu_seqlens) return TS_ERR_NULL;
  if (nseq < 0 || max_seqlen < 0 || total_tokens < 0) return TS_ERR_SHAPE;
  int rc = check_common(q, k, v, o, total_tokens, max_seqlen, H, d, scale);
  if (rc != TS_OK) return rc;
  if (tsattn::packed_grid_bound(total_tokens, nseq, H, 1) >= kGridLimit) return TS_ERR_SHAPE;
  if (nseq == 0 || total_tokens == 0) return TS_OK;
  DeviceState* st = current_device(&rc, (hipStream_t)stream);  // TS_ERR_CAPTURE for a first call
  if (!st) return rc;
  tsattn::PackedArgs a{q, k, v, o, nullptr, cu_seqlens, cu_seqlens, nseq, max_seqlen, max_seqlen,
                       total_tokens, total_tokens, H, d, 1, scale, st->xcd_chunk,
                       nullptr, nullptr, nullptr};
  if (capturing((hipStream_t)stream)) return run_static(st, a, 1, (hipStream_t)stream);
  return run_packed(st, a, (hipStream_t)stream);
}

int ts_attn_fwd_kvcache(const void* q, const void* k, const void* v, void* o, float* lse,
                        const int32_t* cu_seqlens_q, const int32_t* cu_seqlens_k, int32_t nseq,
                        int32_t max_seqlen_q, int32_t max_seqlen_k, int32_t total_q,
                        int32_t total_k, int32_t H, int32_t d, float scale, int32_t num_splits,
                        void* stream) {
  int rc = check_kvcache_call(q, k, v, o, lse, cu_seqlens_q, cu_seqlens_k, nseq, max_seqlen_q,
                              max_seqlen_k, total_q, total_k, H, d, scale, num_splits);
  if (rc != TS_OK) return rc;
  if (nseq == 0 || total_q == 0) return TS_OK;
  DeviceState* st = current_device(&rc, (hipStream_t)stream);  // TS_ERR_CAPTURE for a first call
  if (!st) return rc;
  tsattn::PackedArgs a{q, k, v, o, lse, cu_seqlens_q, cu_seqlens_k, nseq, max_seqlen_q,
                       max_seqlen_k, total_q, total_k, H, d, 1, scale, st->xcd_chunk,
                       nullptr, nullptr, nullptr};
  if (capturing((hipStream_t)stream)) return run_static(st, a, num_splits, (hipStream_t)stream);
  a.n_split = num_splits > 0 ? num_splits : auto_splits(st->cus, total_q, max_seqlen_k, H, d);
  return run_packed(st, a, (hipStream_t)stream);
}

int ts_attn_fwd_kvcache_noalloc(const void* q, const void* k, const void* v, void* o, float* lse,
                                const int32_t* cu_seqlens_q, const int32_t* cu_seqlens_k,
                                int32_t nseq, int32_t max_seqlen_q, int32_t max_seqlen_k,
                                int32_t total_q, int32_t total_k, int32_t H, int32_t d,
                                float scale, int32_t num_splits, void* stream) {
  int rc = check_kvcache_call(q, k, v, o, lse, cu_seqlens_q, cu_seqlens_k, nseq, max_seqlen_q,
                              max_seqlen_k, total_q, total_k, H, d, scale, num_splits);
  if (rc != TS_OK) return rc;
  if (nseq == 0 || total_q == 0) return TS_OK;
  // a forced split count is checked against the scratch before the device is touched
  if (scratch_bytes(nseq, num_splits > 0 ? num_splits : 1, total_q, H, d) > tsattn::kScratchBytes)
    return TS_ERR_SCRATCH;
  DeviceState* st = current_device(&rc, (hipStream_t)stream);
  if (!st) return rc;
  tsattn::PackedArgs a{q, k, v, o, lse, cu_seqlens_q, cu_seqlens_k, nseq, max_seqlen_q,
                       max_seqlen_k, total_q, total_k, H, d, 1, scale, st->xcd_chunk,
                       nullptr, nullptr, nullptr};
  return run_static(st, a, num_splits, (hipStream_t)stream);
}

int ts_state_copy(const void* src, int64_t src_bytes, void* dst, int64_t dst_bytes,
                  const int64_t* ranges, int32_t nranges, void* stream) {
  if (nranges < 0 || src_bytes < 0 || dst_bytes < 0) return TS_ERR_SHAPE;
  if (nranges == 0) return TS_OK;
  if (!src || !dst || !ranges) return TS_ERR_NULL;
  if (misaligned(src) || misaligned(dst)) return TS_ERR_ALIGN;
  if (ranges_overlap(src, src_bytes, dst, dst_bytes)) return TS_ERR_ALIAS;
  for (int32_t r = 0; r < nranges; ++r) {
    const int64_t so = ranges[3 * r], d_o = ranges[3 * r + 1], n = ranges[3 * r + 2];
    if (so < 0 || d_o < 0 || n < 0) return TS_ERR_SHAPE;
    if (((so | d_o | n) & 15) != 0) return TS_ERR_ALIGN;
    if (so > src_bytes || n > src_bytes - so || d_o > dst_bytes || n > dst_bytes - d_o)
      return TS_ERR_SHAPE;
  }
  if (capturing((hipStream_t)stream)) return TS_ERR_CAPTURE;  // operand lookups are not stream work
  int rc = TS_OK;
  DeviceState* st = current_device(&rc, (hipStream_t)stream);
  if (!st) return rc;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return TS_ERR_HIP;
  const void* s_dev = nullptr;
  const void* d_dev = nullptr;
  bool s_host = false, d_host = false;
  if ((rc = copy_operand(src, dev, &s_dev, &s_host)) != TS_OK) return rc;
  if ((rc = copy_operand(dst, dev, &d_dev, &d_host)) != TS_OK) return rc;
  const int64_t chunk = tsattn::copy_chunk_bytes();
  tsattn::CopyList list;
  for (int32_t r0 = 0; r0 < nranges; r0 += tsattn::kMaxCopyRanges) {
    list.n = nranges - r0 < tsattn::kMaxCopyRanges ? nranges - r0 : tsattn::kMaxCopyRanges;
    list.first_chunk[0] = 0;
    for (int32_t i = 0; i < list.n; ++i) {
      const int64_t* e = ranges + 3 * (int64_t)(r0 + i);
      list.src[i] = e[0];
      list.dst[i] = e[1];
      list.bytes[i] = e[2];
      // ceil(bytes / chunk) without forming bytes + chunk - 1 (bytes may be near INT64_MAX)
      list.first_chunk[i + 1] = list.first_chunk[i] + e[2] / chunk + (e[2] % chunk != 0);
    }
    if (list.first_chunk[list.n] >= ((int64_t)1 << 31)) return TS_ERR_SHAPE;
    if (tsattn::launch_state_copy(s_dev, (void*)d_dev, list, s_host, d_host, (hipStream_t)stream) !=
        hipSuccess)
      return TS_ERR_HIP;
  }
  return TS_OK;
}

}  // extern "C"
