// attn_launch.h -- internal interface between the C ABI layer (ts_attn.cpp) and the kernels
// (attn_kernels.hip).  Not installed; the public interface is include/ts_attn.h.
#pragma once
#include <hip/hip_runtime.h>
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

struct VarlenArgs {
  const void* q;
  const void* k;
  const void* v;
  void* o;
  const int32_t* cu_seqlens;  // device
  int32_t nseq, max_seqlen, total_tokens, H, d;
  float scale;
  int xcd_chunk;
  int32_t* plan;  // device, plan_ints(nseq) entries
};

// Upper bound of the number of work items of a packed batch (its launch grid).
int64_t varlen_grid_bound(int32_t total_tokens, int32_t nseq, int32_t H);
// int32 entries of the plan buffer for nseq segments.
int64_t plan_ints(int32_t nseq);
// Queries per work item.
int query_tile();

hipError_t configure_kernels();
hipError_t launch_dense(const DenseArgs& a, hipStream_t st);
hipError_t launch_varlen(const VarlenArgs& a, hipStream_t st);

}  // namespace tsattn
