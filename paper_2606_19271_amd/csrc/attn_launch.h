// attn_launch.h -- internal interface between the C ABI layer (ts_attn.cpp) and the kernels
// (attn_kernels.hip).  Not installed; the public interface is include/ts_attn.h.
#pragma once
#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace tsattn {

struct DenseArgs {
  const void* q;
  const void* k;
  const void* v;
  void* o;
  int32_t B, L, H, d;
  float scale;
  int xcd_chunk;  // consecutive items per XCD (CUs per XCD x workgroups per CU)
};

// A packed batch: segment s has queries [cu_q[s], cu_q[s+1]) of q/o and keys/values
// [cu_k[s], cu_k[s+1]) of k/v (cu_k == cu_q for self-attention).  With n_split > 1 every
// (segment, head, query tile) is split over n_split key ranges whose partial results go to
// part_o / part_lse and are merged into o (and lse) by a second kernel.
struct PackedArgs {
  const void* q;
  const void* k;
  const void* v;
  void* o;
  float* lse;            // device [total_q][H] or null
  const int32_t* cu_q;   // device
  const int32_t* cu_k;   // device
  int32_t nseq, max_q, max_k, total_q, total_k, H, d, n_split;
  float scale;
  int xcd_chunk;
  int32_t* plan;         // device, plan_ints(nseq) entries; null for a batch of one segment
                         // run without the planning kernel
  float* part_o;         // device [n_split][total_q][H][d] (n_split > 1)
  float* part_lse;       // device [n_split][total_q][H] (n_split > 1)
};

// Sizes shared by the kernels and the host-side planning (attn_plan.cpp).
constexpr int kQueryTile = 256;             // queries per work item of the attention kernels
constexpr int kMergeThreads = 256;          // threads per workgroup of the merge kernel
// Keys per K/V tile of the attention kernels at head width d (64 or 128).
constexpr int key_tile(int d) { return d == 64 ? 128 : 64; }
constexpr int64_t kCopyChunkBytes = 32768;  // bytes copied by one state-copy workgroup
// Bytes of the static device scratch array of the allocation-free chunk call (plan and split
// partials), one per device, held from the library's load until the process ends.
constexpr int64_t kScratchBytes = (int64_t)32 << 20;

// Upper bound of the number of work items of a packed batch (its launch grid).
int64_t packed_grid_bound(int32_t total_q, int32_t nseq, int32_t H, int32_t n_split);
// Workgroups of the merge kernel of a split call.
int64_t merge_blocks(int32_t total_q, int32_t H, int32_t d);
// int32 entries of the plan buffer for nseq segments.
int64_t plan_ints(int32_t nseq);

// Up to kMaxCopyRanges byte-range copies of one state-copy launch (passed by value as a kernel
// argument): range r copies bytes[r] bytes from src + src[r] to dst + dst[r]; first_chunk is the
// prefix over the ranges of ceil(bytes / copy_chunk_bytes()), first_chunk[n] = chunks in all.
constexpr int kMaxCopyRanges = 64;
struct CopyList {
  int64_t src[kMaxCopyRanges];
  int64_t dst[kMaxCopyRanges];
  int64_t bytes[kMaxCopyRanges];
  int64_t first_chunk[kMaxCopyRanges + 1];
  int32_t n;
};
int64_t copy_chunk_bytes();
// src_host / dst_host: that side is pinned host memory (accessed non-temporally).
hipError_t launch_state_copy(const void* src, void* dst, const CopyList& list, bool src_host,
                             bool dst_host, hipStream_t st);

hipError_t configure_kernels();
// Device address of the current device's copy of the static scratch array (kScratchBytes).
hipError_t scratch_address(void** ptr);
hipError_t launch_dense(const DenseArgs& a, hipStream_t st);
hipError_t launch_packed(const PackedArgs& a, hipStream_t st);

}  // namespace tsattn
