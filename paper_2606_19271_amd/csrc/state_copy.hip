// state_copy.hip -- batched byte-range copies between device memory and pinned host memory.
//
// The paper's runtime suspends an idle session by copying its persistent state from GPU memory
// to host memory, and resumes it by restoring the state to the GPU chosen for it (Sec. 3.1,
// "GPU-CPU state offloading"); only the session's isolated state region moves (Sec. 6.1,
// "Session memory layout").  In a packed token-major batch a session's cached keys or values are
// one contiguous byte range, so suspend, resume and the compaction of a packed batch after
// sessions leave are all lists of range copies: dst[d, d + n) = src[s, s + n).
//
// Design: one launch copies up to kMaxRanges ranges, passed by value in the kernel arguments
// (no device allocation, no host-to-device upload).  Every range is cut into 32 KiB chunks; one
// 256-thread workgroup copies one chunk with 16-byte accesses, eight loads in flight per thread
// before the stores, so a host-memory side keeps many PCIe requests outstanding.  The chunk
// index space is dense: a prefix over the ranges' chunk counts maps a workgroup to its range.
// Pinned host memory is reached directly at its (unified) virtual address; the side that lives
// in host memory uses non-temporal accesses, which bypass the GPU caches.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "attn_launch.h"

namespace tsstate {

constexpr int kThreads = 256;
constexpr int kPerThread = 8;                      // 16-byte vectors per thread per chunk
constexpr int64_t kChunk = kThreads * kPerThread * 16;  // 32 KiB
static_assert(kChunk == tsattn::kCopyChunkBytes, "chunk size shared with the host planning");

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

template <bool kNtLoad, bool kNtStore>
__global__ void __launch_bounds__(kThreads)
state_copy_kernel(const char* __restrict__ src, char* __restrict__ dst, tsattn::CopyList list) {
  const int64_t c = blockIdx.x;
  // the range holding chunk c: last r with first_chunk[r] <= c (empty ranges own no chunk)
  int lo = 0, hi = list.n;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (list.first_chunk[mid] <= c) lo = mid; else hi = mid;
  }
  const int64_t off = (c - list.first_chunk[lo]) * kChunk;
  const int64_t left = list.bytes[lo] - off;
  const int nvec = (int)((left < kChunk ? left : kChunk) >> 4);
  const u32x4* s = (const u32x4*)(src + list.src[lo] + off);
  u32x4* d = (u32x4*)(dst + list.dst[lo] + off);
  u32x4 r[kPerThread];
#pragma unroll
  for (int u = 0; u < kPerThread; ++u) {
    const int i = threadIdx.x + u * kThreads;
    if (i < nvec) r[u] = kNtLoad ? __builtin_nontemporal_load(&s[i]) : s[i];
  }
#pragma unroll
  for (int u = 0; u < kPerThread; ++u) {
    const int i = threadIdx.x + u * kThreads;
    if (i < nvec) {
      if (kNtStore) __builtin_nontemporal_store(r[u], &d[i]);
      else d[i] = r[u];
    }
  }
}

}  // namespace tsstate

namespace tsattn {

hipError_t launch_state_copy(const void* src, void* dst, const CopyList& list, bool src_host,
                             bool dst_host, hipStream_t st) {
  const int64_t chunks = list.first_chunk[list.n];
  if (chunks <= 0) return hipSuccess;
  const dim3 grid((unsigned)chunks), block(tsstate::kThreads);
  const char* s = (const char*)src;
  char* d = (char*)dst;
  if (src_host && dst_host)
    hipLaunchKernelGGL((tsstate::state_copy_kernel<true, true>), grid, block, 0, st, s, d, list);
  else if (src_host)
    hipLaunchKernelGGL((tsstate::state_copy_kernel<true, false>), grid, block, 0, st, s, d, list);
  else if (dst_host)
    hipLaunchKernelGGL((tsstate::state_copy_kernel<false, true>), grid, block, 0, st, s, d, list);
  else
    hipLaunchKernelGGL((tsstate::state_copy_kernel<false, false>), grid, block, 0, st, s, d, list);
  return hipGetLastError();
}

}  // namespace tsattn
