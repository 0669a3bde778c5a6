// ts_attn.cpp -- the C ABI of libts_attn.so (declared in include/ts_attn.h): argument checks,
// per-device set-up, the plan buffer of packed batches, and the launches.
#include "ts_attn.h"

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <mutex>

#include "attn_launch.h"

namespace {

constexpr int kMaxDevices = 64;
constexpr int64_t kByteLimit = (int64_t)1 << 31;
constexpr int64_t kGridLimit = (int64_t)1 << 23;  // workgroups per launch (x 512 threads < 2^32)

struct DeviceState {
  std::once_flag once;
  int status = TS_ERR_UNSUPPORTED;  // TS_OK once the device is known to be usable
  int xcd_chunk = 32;
  hipMemPool_t pool = nullptr;
};

DeviceState g_dev[kMaxDevices];

void init_device(int dev, DeviceState* st) {
  hipDeviceProp_t p;
  if (hipGetDeviceProperties(&p, dev) != hipSuccess) { st->status = TS_ERR_HIP; return; }
  if (strncmp(p.gcnArchName, "gfx950", 6) != 0) { st->status = TS_ERR_UNSUPPORTED; return; }
  // gfx950: 8 XCDs; one 512-thread workgroup resides per CU.
  st->xcd_chunk = p.multiProcessorCount / 8 > 0 ? p.multiProcessorCount / 8 : 1;
  if (tsattn::configure_kernels() != hipSuccess) { st->status = TS_ERR_HIP; return; }
  hipMemPoolProps props;
  memset(&props, 0, sizeof props);
  props.allocType = hipMemAllocationTypePinned;
  props.location.type = hipMemLocationTypeDevice;
  props.location.id = dev;
  if (hipMemPoolCreate(&st->pool, &props) != hipSuccess) { st->status = TS_ERR_HIP; return; }
  uint64_t keep = UINT64_MAX;  // keep freed plan buffers in the pool between calls
  if (hipMemPoolSetAttribute(st->pool, hipMemPoolAttrReleaseThreshold, &keep) != hipSuccess) {
    st->status = TS_ERR_HIP;
    return;
  }
  st->status = TS_OK;
}

// The calling thread's current device, initialised once.
DeviceState* current_device(int* status) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    *status = TS_ERR_UNSUPPORTED;
    return nullptr;
  }
  DeviceState* st = &g_dev[dev];
  std::call_once(st->once, init_device, dev, st);
  *status = st->status;
  return st->status == TS_OK ? st : nullptr;
}

bool misaligned(const void* p) { return ((uintptr_t)p & 15u) != 0; }

bool overlaps(const void* a, const void* b, int64_t bytes) {
  uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
  return x < y + (uintptr_t)bytes && y < x + (uintptr_t)bytes;
}

// Shared checks of both entry points; tokens = rows of q/k/v/o, longest = longest segment.
int check_common(const void* q, const void* k, const void* v, const void* o, int64_t tokens,
                 int64_t longest, int32_t H, int32_t d, float scale) {
  if (!q || !k || !v || !o) return TS_ERR_NULL;
  if (H < 1 || tokens < 0 || longest < 0) return TS_ERR_SHAPE;
  if (d != 64 && d != 128) return TS_ERR_HEAD_DIM;
  if (!isfinite(scale)) return TS_ERR_SCALE;
  if (misaligned(q) || misaligned(k) || misaligned(v) || misaligned(o)) return TS_ERR_ALIGN;
  const int64_t row_bytes = (int64_t)H * d * 2;
  if ((longest + 256) * row_bytes >= kByteLimit) return TS_ERR_SHAPE;
  if (tokens > (int64_t)1 << 31 || tokens * row_bytes / row_bytes != tokens) return TS_ERR_SHAPE;
  const int64_t bytes = tokens * row_bytes;
  if (overlaps(o, q, bytes) || overlaps(o, k, bytes) || overlaps(o, v, bytes)) return TS_ERR_ALIAS;
  return TS_OK;
}

bool validate_mode() {
  const char* e = getenv("TS_ATTN_VALIDATE");
  return e && e[0] == '1';
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
  DeviceState* st = current_device(&rc);
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
  if (tsattn::varlen_grid_bound(total_tokens, nseq, H) >= kGridLimit) return TS_ERR_SHAPE;
  if (nseq == 0 || total_tokens == 0) return TS_OK;
  DeviceState* st = current_device(&rc);
  if (!st) return rc;
  hipStream_t s = (hipStream_t)stream;
  int32_t* plan = nullptr;
  const size_t plan_bytes = (size_t)tsattn::plan_ints(nseq) * sizeof(int32_t);
  if (hipMallocFromPoolAsync((void**)&plan, plan_bytes, st->pool, s) != hipSuccess)
    return TS_ERR_NOMEM;
  tsattn::VarlenArgs a{q, k, v, o, cu_seqlens, nseq, max_seqlen, total_tokens, H, d, scale,
                       st->xcd_chunk, plan};
  rc = tsattn::launch_varlen(a, s) == hipSuccess ? TS_OK : TS_ERR_HIP;
  if (rc == TS_OK && validate_mode()) {
    int32_t head[2] = {0, 0};
    if (hipMemcpyAsync(head, plan, sizeof head, hipMemcpyDeviceToHost, s) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess)
      rc = TS_ERR_HIP;
    else if (head[1] != 0)
      rc = TS_ERR_SEGMENTS;
  }
  if (hipFreeAsync(plan, s) != hipSuccess && rc == TS_OK) rc = TS_ERR_HIP;
  return rc;
}

}  // extern "C"
