// attn_plan.cpp -- host-side sizes of the launches (grids, plan buffer, copy chunks), shared by
// the argument checks of ts_attn.cpp and the launch code; no device code.
#include <stdint.h>

#include "attn_launch.h"

namespace tsattn {

int64_t packed_grid_bound(int32_t total_q, int32_t nseq, int32_t H, int32_t n_split) {
  // sum_s ceil(Lq_s / tile) <= ceil(Tq / tile) + nseq
  return (int64_t)H * n_split * (((int64_t)total_q + kQueryTile - 1) / kQueryTile + nseq);
}

int64_t merge_blocks(int32_t total_q, int32_t H, int32_t d) {
  return ((int64_t)total_q * H * (d / 8) + kMergeThreads - 1) / kMergeThreads;
}

int64_t plan_ints(int32_t nseq) { return 2 + 2 * (int64_t)nseq; }

int64_t copy_chunk_bytes() { return kCopyChunkBytes; }

}  // namespace tsattn
