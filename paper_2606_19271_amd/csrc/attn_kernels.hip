// attn_kernels.hip -- gfx950 (CDNA4) kernels of the fused segment-local attention.
//
// Computes, for every segment s of a packed batch, token t of s and head h,
//   O[t,h,:] = softmax_j(scale * <Q[t,h,:], K[j,h,:]>) V[j,h,:],  j over segment s (non-causal),
// the attention of the model call that serves one coalesced chunk batch (paper Sec. 3.1), with
// sessions kept apart as their isolated state regions require (Sec. 6.1).
//
// Design (one work item = one (segment, head, 256-query tile); one 512-thread workgroup each):
//  * 8 waves, each owning 32 queries.  The wave computes S^T = K Q^T on 32x32x16 bf16 MFMAs,
//    so that a lane holds all scores of ONE query (its column): the row max is in-lane, plus
//    one cross-half exchange (v_permlane32_swap).  The row sums of the weights are formed on
//    the matrix core, by a 16x16x32 MFMA per 16 keys with a 0/1 operand that adds the two lanes
//    of each query.
//  * The exponentiated scores P^T, packed to bf16, are already the B operand of the next
//    product O^T += V^T P^T once the keys inside each 16-key step are taken in the order the
//    accumulator holds them (a sum over keys does not care about their order); V^T's fragments
//    come from row-major V in LDS through the gfx950 transpose read ds_read_b64_tr_b16.
//  * The two waves that share a SIMD run a ping-pong: one issues the MFMAs of a tile (S = K Q^T
//    of the next tile and O += V P of the previous one) at raised priority while the other
//    issues the softmax VALU work, and they swap roles at each workgroup barrier.  On gfx950
//    v_exp_f32 shares the VALU pipe with the other vector ops, while MFMAs run in the matrix
//    core, so the softmax can hide under the other wave's matrix work.
//  * K and V tiles of 64 keys (128 at d = 64) are staged in LDS in rings of four (K) and three (V), laid out
//    (K padded, V XOR-swizzled) so that the MFMA operand reads are free of bank conflicts.  They
//    arrive by LDS DMA (buffer_load ... lds), which needs no registers and no LDS write
//    instructions, issued only in the vector steps; the raw buffer descriptor's range check
//    returns zeros past the segment's last row.  The first K operands of each matrix step are
//    read at the end of the preceding vector step, so their latency overlaps the barrier.
//  * Online softmax in the log2 domain (exp2 with scale*log2(e) folded into one FMA).  A tile
//    is first exponentiated against the running maximum as it stands; only if some weight
//    would exceed 2^40 times the largest so far (or on the first and the last tile) is the
//    tile's maximum taken and the O accumulator rescaled.  Keeping a stale maximum is exact in
//    real arithmetic (the final division by the running sum cancels the common factor), so for
//    ordinary inputs the per-tile max reduction and the O rescale disappear.
//  * Scheduling: the launch has one workgroup per item; blockIdx is remapped so that the 32
//    workgroups resident at once on one XCD (the hardware deals workgroups to the 8 XCDs
//    round robin) take 32 consecutive query tiles of the same head and share its K/V in that
//    XCD's L2.  For packed batches a planning kernel first orders segments longest first.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "attn_launch.h"

namespace tsattn {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8;
typedef __attribute__((address_space(3))) u32x4 lds_u32x4;
typedef __attribute__((address_space(3))) char lds_char;
typedef __attribute__((address_space(3))) void lds_void;


constexpr int kBM = kQueryTile;  // queries per work item
constexpr int kWaves = 8;      // waves per workgroup, 32 queries each
constexpr int kThreads = kWaves * 64;
constexpr float kLog2e = 1.4426950408889634f;
constexpr unsigned kRsrcWord3 = 0x00020000u;  // raw buffer, 32-bit data format (gfx9 family)

// LDS layout: a ring of three V tiles (first, so every V address fits the 16-bit immediate of a
// DS instruction), then a ring of four K tiles; V_j sits in stage j % 3 and K_j in j % 4.  Tiles arrive by
// LDS DMA (buffer_load ... lds: lane i of an instruction lands at base + 16 i), 1 KiB per
// instruction.
//  * K rows are padded by one 16-byte chunk (stride 2d + 16 bytes), so the 16 rows one b128 K
//    read touches per 16 lanes fall on distinct banks.  DMA lanes that land in a pad chunk fetch
//    a harmless duplicate.
//  * V rows are unpadded; the 16-byte chunk c of row r is stored at chunk position c ^ vswz(r),
//    which keeps the transposed V reads free of bank conflicts.
template <int D>
struct Geo {
  // Keys per K/V tile.  A matrix step costs the same number of MFMA clocks at both head widths
  // (32 32x32x16 MFMAs per wave): 64 keys at d = 128, 128 keys at d = 64, so the fixed costs of
  // a step (two barriers, the DMA issue, the waits) weigh the same against its matrix work.
  static constexpr int kBN = key_tile(D);
  static constexpr int kChunks = D / 8;                  // 16-byte chunks per row of d bf16
  static constexpr int kKRow = D * 2 + 16;               // padded K row stride (bytes)
  static constexpr int kVRow = D * 2;                    // V row stride (bytes)
  static constexpr int kKTile = kBN * kKRow;
  static constexpr int kVTile = kBN * kVRow;
  static constexpr int kKStages = 4;                     // K_j in stage j % 4
  static constexpr int kVStages = 3;                     // V_j in stage j % 3
  static constexpr int kVRing = 0;                       // byte offset of the V ring
  static constexpr int kKRing = kVStages * kVTile;       // byte offset of the K ring
  static constexpr int kLds = kKStages * kKTile + kVStages * kVTile;
  static constexpr int kGroupWaves = kWaves / 2;
  static constexpr int kKDma = kKTile / 1024;            // DMA instructions per K tile (17 / 18)
  static constexpr int kVDma = kVTile / 1024;            // per V tile (16 / 16)
  static constexpr int kKDmaMax = (kKDma + kGroupWaves - 1) / kGroupWaves;  // per wave, at most
  static constexpr int kKDmaMin = kKDma / kGroupWaves;                      // per wave, at least
  static constexpr int kVDmaPerWave = kVDma / kGroupWaves;
  // Pair steps of the softmax's exp work (16 per tile at d = 128, 32 at d = 64) between two of
  // the vector step's DMA instructions.  Issued back to back, the four vector-step waves of a CU
  // queue 16 KiB at once on its 64 B/clk address path, and each wave's exp work waits behind
  // its own share of that queue.
  static constexpr int kDmaEvery = 4;
  static_assert(kKTile % 1024 == 0 && kVTile % 1024 == 0 && kVDma % kGroupWaves == 0, "DMA split");
  static_assert(kVStages * kVTile <= 65536, "V addresses must fit the DS immediate");
  __host__ __device__ static constexpr int vswz(int r) {
    return D == 128 ? (((r & 3) << 2) | ((r >> 2) & 3)) : ((((r >> 1) & 1) << 2) | ((r >> 2) & 3));
  }
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           (int)kRsrcWord3);
}

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// max over the two 32-lane halves of the wave (lane l and lane l^32).
__device__ __forceinline__ float half_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// One work item: queries [q_begin, q_begin + kBM) of a segment, head h, against the 64-key
// tiles [tile_begin, tile_begin + ntiles) of the segment's keys.  For self-attention the query
// and key rows of a segment coincide; for chunk queries against a session's cache they are
// separate ranges of q/o and of k/v.
struct Item {
  int64_t q_start;  // first query token of the segment (row of q and o)
  int64_t k_start;  // first key token of the segment (row of k and v)
  int q_len;        // queries of the segment
  int k_len;        // keys of the segment
  int h;            // head
  int q_begin;      // first query of the tile, relative to the segment
  int tile_begin;   // first key tile of the item
  int ntiles;       // key tiles of the item
};

// Query tiles per (sequence, head) kept in the main item order of a dense call: all nq, unless the
// last tile is ragged enough to leave a wave without queries.  Such a tile's workgroup runs its
// phases faster than its neighbours (its idle waves skip their compute), so the items after it
// on its CU would drift out of step with the items that stream the same keys and values on the
// same XCD, and lose their shared L2 hits; these tiles are run after all full ones instead.
// (Packed and chunk calls keep their per-segment order: there the ragged tiles share their key
// ranges with the segment's other tiles, and moving them away from those costs more L2 hits.)
__host__ __device__ inline int main_query_tiles(int len) {
  const int nq = (len + kBM - 1) / kBM, tail = len % kBM;
  return tail != 0 && (tail + 31) / 32 < kWaves ? nq - 1 : nq;
}

// Where the results of an item go.  kFinal: O as bf16 [Tq][H][D] and, when lse is not null,
// the natural log-sum-exp of every row as float [Tq][H].  kPartial (one key range of a split
// call): the normalised O of that range as float [splits][Tq][H][D] and its log-sum-exp as
// float [splits][Tq][H], combined afterwards by attn_merge_kernel.
enum OutMode { kFinal = 0, kPartial = 1 };
struct Out {
  __bf16* o;
  float* lse;
  float* part_o;
  float* part_lse;
  int64_t tq;  // query rows of the whole call (one split's slab is tq x H rows)
  int split;   // key range of this item (kPartial)
};

constexpr float kLn2 = 0.6931471805599453f;

// XCD-aware order: workgroup b runs on XCD b % 8; consecutive workgroups of one XCD take
// `chunk` consecutive items, and every 8*chunk workgroups cover 8*chunk consecutive items,
// so the global order is kept at that granularity.  The r items after the last whole span are
// dealt the same way: XCD x takes a contiguous block of its ceil((r - x) / 8) of them.
// Bijective on [0, total).
__device__ __forceinline__ int remap_block(int b, int total, int chunk) {
  const int span = 8 * chunk;
  const int full = (total / span) * span;
  const int x = b & 7;
  if (b < full) {
    const int j = b >> 3;
    return (j / chunk) * span + x * chunk + (j % chunk);
  }
  const int r = total - full, j = (b - full) >> 3;  // j-th tail workgroup of XCD x
  const int q = r >> 3, rem = r & 7;                // XCD x has q + (x < rem) of them
  return full + x * q + min(x, rem) + j;
}

// S^T = K Q^T for one key tile: 32-key blocks (two at d = 128, four at d = 64), each an
// accumulation over d in steps of 16.  Accumulator register r of block kb holds key
// 32*kb + 8*(r/4) + 4*hb + r%4 of the tile for the lane's query (lane & 31).  The blocks' MFMAs
// alternate, so that each Q fragment is the B operand of consecutive MFMAs: under the power cap
// an operand held over consecutive MFMAs costs less switching energy, and the clock rises
// accordingly (measured +0.6 % for two).  MFMA i uses the K fragment (kk, kb) = (i / nkb, i % nkb)
// with nkb blocks per tile; the first kPreReads of them were read ahead into kp.
constexpr int kPreReads = 8;

template <int D>
__device__ __forceinline__ const lds_char* k_frag(const lds_char* kt, int kk, int kb, int lane) {
  using G = Geo<D>;
  return kt + (32 * kb + (lane & 31)) * G::kKRow + (lane >> 5) * 16 + kk * 32;
}

// The K fragments of a tile's first kPreReads S MFMAs.
template <int D>
__device__ __forceinline__ void k_preread(const lds_char* __restrict__ kt, bf16x8 (&kp)[kPreReads],
                                          int lane) {
  constexpr int kKB = Geo<D>::kBN / 32;  // 32-key blocks per tile
#pragma unroll
  for (int i = 0; i < kPreReads; ++i)
    kp[i] = *(const lds_bf16x8*)k_frag<D>(kt, i / kKB, i % kKB, lane);
}

template <int D>
__device__ __forceinline__ void qk_tile(const lds_char* __restrict__ kt, const bf16x8 (&qf)[D / 16],
                                        const bf16x8 (&kp)[kPreReads],
                                        f32x16 (&s)[Geo<D>::kBN / 32], int lane) {
  constexpr int kKB = Geo<D>::kBN / 32;
#pragma unroll
  for (int kb = 0; kb < kKB; ++kb) s[kb] = f32x16{};
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk)
#pragma unroll
    for (int kb = 0; kb < kKB; ++kb) {
      const int i = kKB * kk + kb;
      bf16x8 a = i < kPreReads ? kp[i] : *(const lds_bf16x8*)k_frag<D>(kt, kk, kb, lane);
      s[kb] = mfma32(a, qf[kk], s[kb]);
    }
}

// Lane offsets of the transposed V reads inside a V tile: for 8-row group r2 and 32-channel
// block db, the 8 bytes of row 8 r2 + vr (+16 t) that this lane addresses.  Within each
// 16-lane group, lane 4R + c addresses 4 channels of key row R, and after the transpose lane j
// holds channel j of those 4 rows.
template <int D>
struct VOffsets {
  int off[2][D / 32];
  __device__ __forceinline__ explicit VOffsets(int lane) {
    using G = Geo<D>;
    const int g = lane >> 4, i16 = lane & 15;
    const int vr = 4 * (g >> 1) + (i16 >> 2);        // key row inside an 8-key group
    const int vch = 2 * (g & 1) + ((i16 & 3) >> 1);  // 16-byte chunk inside a 64-byte block
    const int vhalf = 8 * (i16 & 1);                 // 8-byte half of that chunk
#pragma unroll
    for (int r2 = 0; r2 < 2; ++r2)
#pragma unroll
      for (int db = 0; db < D / 32; ++db) {
        const int row = 8 * r2 + vr;  // the swizzle depends on the row mod 16 only
        off[r2][db] = row * G::kVRow + (((4 * db + vch) ^ G::vswz(row)) << 4) + vhalf;
      }
  }
};

// Row sums of the weights on the matrix core: one 16x16x32 MFMA per 16-key step.  The B operand
// is the step's weight fragment p[t] as it is (lane l: 8 keys of query l & 31), which this MFMA
// reads as column l & 15, k = 8 (l >> 4) + 0..7; the A operand is 1 on the k-groups {G, G ^ 2}
// of the rows 4G..4G+3 and 0 elsewhere.  Result row 4G + r, column n is then the sum of lanes
// 16G + n and 16(G ^ 2) + n -- the two lanes of one query, l and l ^ 32 -- and it lands in
// exactly those lanes, in all four accumulator registers.  The sum is formed from exactly the
// bf16 weights the PV product uses, so a row dominated by one key returns that key's value
// exactly.  Summing in the vector step instead costs two VALU instructions per weight (a pair of
// bf16 is widened by a shift and a mask and added; v_dot2_f32_bf16 issues to the matrix core and
// stalls behind the other wave's MFMAs), and that step is the longer of the two.

// A operand of the row-sum MFMA for this lane: bf16 1.0 where the lane's k-group is one of the
// two groups its row block sums, else 0.
__device__ __forceinline__ bf16x8 row_sum_selector(int lane) {
  const int g = lane >> 4, mg = (lane & 15) >> 2;
  const unsigned one = (g == mg || g == (mg ^ 2)) ? 0x3f803f80u : 0u;
  return __builtin_bit_cast(bf16x8, u32x4{one, one, one, one});
}

// The row sums of one tile's weights, on two accumulators in turn: switching the matrix core
// between the 32x32x16 and the 16x16x32 shape costs about 6 clocks each way (measured), so the
// four row-sum MFMAs are issued together, and two chains keep them from waiting on each other.
template <int NT>
__device__ __forceinline__ void row_sums(bf16x8 sel, const bf16x8 (&p)[NT], f32x4 (&l)[2]) {
#pragma unroll
  for (int t = 0; t < NT; ++t)
    l[t & 1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(sel, p[t], l[t & 1], 0, 0, 0);
}

// O^T += V^T P^T for one 64-key tile.  p[t] holds the bf16 weights
// of keys 16t + 8*(m/4) + 4*hb + m%4 (m = 0..7) -- the accumulator order of qk_tile -- and the
// V^T fragments are read in that same key order with the transpose read: elements 0-3 from rows
// 16t + 4hb + 0..3, elements 4-7 from rows 16t + 8 + 4hb + 0..3.
template <int D>
__device__ __forceinline__ void pv_tile(const lds_char* __restrict__ vt, const VOffsets<D>& vo,
                                        const bf16x8 (&p)[Geo<D>::kBN / 16], f32x16 (&o)[D / 32]) {
  using G = Geo<D>;
#pragma unroll
  for (int t = 0; t < G::kBN / 16; ++t)
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
      const lds_char* base = vt + 16 * t * G::kVRow;
      bf16x4 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(base + vo.off[0][db]));
      bf16x4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(base + vo.off[1][db]));
      bf16x8 a = {v0[0], v0[1], v0[2], v0[3], v1[0], v1[1], v1[2], v1[3]};
      o[db] = mfma32(a, p[t], o[db]);
    }
}

// Nothing to issue (see exp_pack).
struct NoIssue {
  __device__ void operator()(int) const {}
};

// exp2(S*c - m_c) for the 32 scores of the lane, packed to the bf16 B operands of the PV
// product.  Returns the bitwise OR of the packed words: bit 14 of a bf16 is the top bit of its
// exponent, set exactly when the (non-negative) value is at least 2 or not finite, so
// (OR & 0x40004000) != 0 flags a tile whose weights are not all below 2.
// issue(0 .. kIssue - 1) is called in order, instruction i at the start of pair step
// i * kEvery (kEvery = 0: all at the start): the vector step's K/V DMA instructions go there.
template <int NT, bool kMasked, int kIssue = 0, int kEvery = 0, typename Issue = NoIssue>
__device__ __forceinline__ unsigned exp_pack(const f32x16 (&s)[NT / 2], bf16x8 (&p)[NT],
                                             float m_c, float c, int keys_valid, int hb,
                                             Issue&& issue = Issue{}) {
  static_assert(kEvery * (kIssue - 1) < NT * 4, "issue points");
  unsigned any = 0;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
#pragma unroll
    for (int m = 0; m < 8; m += 2) {
      const int step = 4 * t + m / 2;
      if (kIssue > 0 && (kEvery == 0 ? step == 0 : step % kEvery == 0 && step / kEvery < kIssue)) {
        // the scheduling barriers keep the scheduler from gathering the memory instructions at
        // the top again
        __builtin_amdgcn_sched_barrier(0);
        if (kEvery == 0) {
#pragma unroll
          for (int i = 0; i < kIssue; ++i) issue(i);
        } else {
          issue(step / (kEvery > 0 ? kEvery : 1));
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      float x0 = s[t >> 1][8 * (t & 1) + m], x1 = s[t >> 1][8 * (t & 1) + m + 1];
      float e0 = __builtin_amdgcn_exp2f(__builtin_fmaf(x0, c, -m_c));
      float e1 = __builtin_amdgcn_exp2f(__builtin_fmaf(x1, c, -m_c));
      if (kMasked) {
        int key0 = 16 * t + 8 * (m >> 2) + 4 * hb + (m & 3);
        if (key0 >= keys_valid) e0 = 0.0f;
        if (key0 + 1 >= keys_valid) e1 = 0.0f;
      }
      f32x2 e = {e0, e1};
      bf16x2 pb = __builtin_convertvector(e, bf16x2);
      p[t][m] = pb[0];
      p[t][m + 1] = pb[1];
      any |= __builtin_bit_cast(unsigned, pb);
    }
  }
  return any;
}

// Online softmax of one tile of scores (the lane's query): turns S into bf16 weights
// P = exp2(S*c - m_c).  Their sum is accumulated by the matrix step (row_sums).
//
// m_c is the running maximum (log2 units of the scaled scores) raised by kBias, so the largest
// weight seen so far is 2^-kBias; the bias cancels in O / l and is part of the log-sum-exp.
// m_c is not recomputed per tile.  A full tile first tries the current m_c: if every weight of
// every lane is below 2 -- at most 2^(kBias + 1) times the largest weight so far -- the fp32
// accumulators stay far from overflow and the tile is done; exact in real arithmetic, since the
// final division by l cancels the common factor.  Otherwise (the first tile, where m_c = -inf, a
// score far above the running maximum, or the masked last tile) the tile's true maximum is
// taken, m_c moves up to it (plus the bias), and the accumulators of O and l -- which hold the
// products of the earlier tiles, relative to the old m_c -- are multiplied by
// alpha = 2^(m_c,old - m_c,new) before the next matrix step adds these weights to them.  Doing
// that here, in the rare slow path of the vector step, keeps the matrix step free of branches.
constexpr float kBias = 39.0f;

// issue(0 .. kIssue - 1): instructions to spread over the tile's exp work (see exp_pack); all
// of them are issued once, on every path.
template <int D, bool kMasked, int kIssue, typename Issue>
__device__ __forceinline__ void softmax_tile(f32x16 (&s)[Geo<D>::kBN / 32],
                                             bf16x8 (&p)[Geo<D>::kBN / 16], float& m_c,
                                             f32x16 (&o)[D / 32], f32x4 (&l)[2], float c,
                                             int keys_valid, int lane, Issue&& issue) {
  constexpr int kBN = Geo<D>::kBN;
  const int hb = lane >> 5;
  if (!kMasked) {
    const unsigned any =
        exp_pack<kBN / 16, false, kIssue, Geo<D>::kDmaEvery>(s, p, m_c, c, kBN, hb, issue);
    if (__builtin_amdgcn_ballot_w64((any & 0x40004000u) != 0) == 0) return;
  }
  if (kMasked) {
#pragma unroll
    for (int i = 0; i < kIssue; ++i) issue(i);
  }
  if (kMasked) {
#pragma unroll
    for (int kb = 0; kb < kBN / 32; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        int key = 32 * kb + 8 * (r >> 2) + 4 * hb + (r & 3);
        if (key >= keys_valid) s[kb][r] = -INFINITY;
      }
  }
  float mt = s[0][0];
#pragma unroll
  for (int kb = 0; kb < kBN / 32; ++kb)
#pragma unroll
    for (int r = 0; r < 16; ++r) mt = fmaxf(mt, s[kb][r]);
  mt = half_max(mt);
  // c >= 0, so the max commutes with the scaling
  const float m_new = fmaxf(m_c, __builtin_fmaf(mt, c, kBias));
  const float alpha = __builtin_amdgcn_exp2f(m_c - m_new);  // 0 on the first tile (m_c = -inf)
  m_c = m_new;
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
  l[0] *= alpha;
  l[1] *= alpha;
  exp_pack<kBN / 16, kMasked>(s, p, m_c, c, keys_valid, hb);
}

// Lane offsets (bytes, relative to the tile's first row in global memory) of one wave's share
// of the LDS DMA of a K or a V tile.  The four waves of a group split a tile: DMA instruction
// n = gw + 4u of the tile fills LDS bytes [1024 n, 1024 n + 1024) of it, lane i bytes
// 1024 n + 16 i.
template <int D>
__device__ __forceinline__ void dma_offsets_k(int gw, int lane, int row_bytes,
                                              int* koff) {
  using G = Geo<D>;
#pragma unroll
  for (int u = 0; u < G::kKDmaMax; ++u) {
    const int b = 1024 * (gw + G::kGroupWaves * u) + 16 * lane;
    const int row = b / G::kKRow, colb = b % G::kKRow;
    const int chunk = colb < D * 2 ? colb / 16 : 0;  // pad lanes fetch chunk 0 again
    koff[u] = row * row_bytes + chunk * 16;
  }
}
template <int D>
__device__ __forceinline__ void dma_offsets_v(int gw, int lane, int row_bytes,
                                              int* voff) {
  using G = Geo<D>;
#pragma unroll
  for (int u = 0; u < G::kVDmaPerWave; ++u) {
    const int b = 1024 * (gw + G::kGroupWaves * u) + 16 * lane;
    const int row = b / G::kVRow;
    const int chunk = ((b % G::kVRow) / 16) ^ G::vswz(row);
    voff[u] = row * row_bytes + chunk * 16;
  }
}

// This wave's share of the DMA of the K tile whose first key is key0 (rows past the segment
// end read as zeros through the descriptor's range check).  kFrom skips the first kFrom
// instructions (issued one by one with dma_k_one).
template <int D, int kFrom = 0>
__device__ __forceinline__ void dma_k(__amdgpu_buffer_rsrc_t rk, int key0, int row_bytes,
                                      lds_char* tile, const int* koff, int gw) {
  using G = Geo<D>;
  const int skip = key0 * row_bytes;
#pragma unroll
  for (int u = kFrom; u < G::kKDmaMax; ++u) {
    const int n = gw + G::kGroupWaves * u;
    if (u < G::kKDmaMin || n < G::kKDma)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (lds_void*)(tile + 1024 * n), 16, koff[u] + skip,
                                               0, 0, 0);
  }
}
// Instruction u < kKDmaMin of that share (every wave issues these, without a branch).
template <int D>
__device__ __forceinline__ void dma_k_one(__amdgpu_buffer_rsrc_t rk, int key0, int row_bytes,
                                          lds_char* tile, const int* koff, int gw, int u) {
  using G = Geo<D>;
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (lds_void*)(tile + 1024 * (gw + G::kGroupWaves * u)),
                                           16, koff[u] + key0 * row_bytes, 0, 0, 0);
}
template <int D>
__device__ __forceinline__ void dma_v(__amdgpu_buffer_rsrc_t rv, int key0, int row_bytes,
                                      lds_char* tile, const int* voff, int gw) {
  using G = Geo<D>;
  const int skip = key0 * row_bytes;
#pragma unroll
  for (int u = 0; u < G::kVDmaPerWave; ++u)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (lds_void*)(tile + 1024 * (gw + G::kGroupWaves * u)),
                                             16, voff[u] + skip, 0, 0, 0);
}
template <int D>
__device__ __forceinline__ void dma_v_one(__amdgpu_buffer_rsrc_t rv, int key0, int row_bytes,
                                          lds_char* tile, const int* voff, int gw, int u) {
  using G = Geo<D>;
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (lds_void*)(tile + 1024 * (gw + G::kGroupWaves * u)),
                                           16, voff[u] + key0 * row_bytes, 0, 0, 0);
}

// Waits until at most N of this wave's vector-memory operations are outstanding.
template <int N>
__device__ __forceinline__ void wait_vmem() {
  static_assert(N >= 0 && N < 16, "vmcnt field");
  __builtin_amdgcn_s_waitcnt(0x0F70 | N);  // gfx9 encoding: expcnt and lgkmcnt left open
}

// Workgroup barrier without a memory fence (the waits before it are explicit); the empty asm
// statements keep the compiler from moving memory accesses across it.
__device__ __forceinline__ void block_sync() {
  __asm__ volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  __asm__ volatile("" ::: "memory");
}

// The matrix step of tile j: the row sums of P_{j-1}, S_j = K_j Q^T, then O += V_{j-1} P_{j-1},
// in one basic block.  None of the first MFMAs waits for the LDS: the row sums read registers
// only, and the K fragments of the first kPreReads S MFMAs were read in the vector step before
// the barrier.  After that the issue order is pinned so that each MFMA's LDS operand is
// requested kPreReads MFMAs earlier (one b128 read per S MFMA, two transpose reads per PV MFMA).
template <int D, bool kPV>
__device__ __forceinline__ constexpr int m_step_reads(int i) {
  constexpr int kBN = Geo<D>::kBN;
  constexpr int kRS = kPV ? kBN / 16 : 0;  // row-sum MFMAs
  constexpr int kQK = (kBN / 32) * (D / 16);
  if (i < kRS) return 0;
  i -= kRS;
  return i < kQK ? (i < kPreReads ? 0 : 1) : 2;
}

template <int D, bool kPV>
__device__ __forceinline__ void m_step(const lds_char* __restrict__ kt, const lds_char* __restrict__ vt,
                                       const VOffsets<D>& vo, const bf16x8 (&qf)[D / 16],
                                       const bf16x8 (&kp)[kPreReads],
                                       f32x16 (&s)[Geo<D>::kBN / 32],
                                       const bf16x8 (&p)[Geo<D>::kBN / 16], f32x16 (&o)[D / 32],
                                       bf16x8 sel, f32x4 (&l)[2], int lane) {
  constexpr int kBN = Geo<D>::kBN;
  if (kPV) row_sums(sel, p, l);
  qk_tile<D>(kt, qf, kp, s, lane);
  if (kPV) pv_tile<D>(vt, vo, p, o);
  // MFMAs: row sums (4), S (16 at d = 128), PV (16 at d = 128)
  constexpr int kN = (kPV ? kBN / 16 : 0) + (kBN / 32) * (D / 16) + (kPV ? (kBN / 16) * (D / 32) : 0);
#pragma unroll
  for (int i = 0; i < kN; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    const int next = i + kPreReads;  // MFMA whose operands are requested now
    const int reads = next < kN ? m_step_reads<D, kPV>(next) : 0;
    if (reads == 1) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    else if (reads == 2) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
  }
}

// One work item, software-pipelined across the two waves that share each SIMD.
//
// Per 64-key tile j a wave runs two steps: M(j) -- the matrix step: S_j = K_j Q^T and
// O += V_{j-1} P_{j-1} on MFMA -- and V(j) -- the vector step: the online softmax S_j -> P_j.
// Waves 0-3 (group A) and waves 4-7 (group B) sit on the four SIMDs in pairs (wave w and w+4
// share SIMD w % 4), and group B runs one step behind group A, with a workgroup barrier between
// steps: while one wave of a SIMD keeps the matrix core busy, the other issues its softmax VALU
// work.  The matrix step raises its wave priority so its MFMAs issue first, and it does no
// global-memory work at all.
//
// K/V staging is by LDS DMA, issued in the vector steps only: group A fetches K_{j+3} in V(j)
// into a ring of four stages, group B fetches V_{j+2} into a ring of three, and each wave waits
// for the fetch of its previous vector step right before the barrier that closes V(j).  Phases
// (A's M(j) = 2j, A's V(j) = B's M(j) = 2j + 1, B's V(j) = 2j + 2): K_m is complete before
// phase 2m - 2 and V_{m-1} before phase 2m; a stage is refilled only after the barrier that
// follows its last reader (B's M(m) at 2m + 1 for K_m, refilled at 2m + 3; B's M(m + 1) at
// 2m + 3 for V_m, refilled at 2m + 5).  K_{j+1} is therefore complete and visible during
// phases 2j .. 2j + 2, so both groups read the K fragments of their next matrix step's first
// MFMAs at the end of V(j), before its barrier; the LDS latency then overlaps the barrier wait
// instead of delaying the first MFMA.  Fetches past the segment end read zeros and land in
// stages nobody reads any more, so the schedule has no branches.  The two groups are separate
// instantiations, so each has a straight-line schedule.
template <int D, int kMode>
__device__ __forceinline__ void write_result(const Item& it, const Out& out,
                                             const f32x16 (&oacc)[D / 32], float l_tot, float m_c,
                                             int H, int qrow, int hb);

//
// kActive = false is the same schedule for a wave whose 32 queries all lie past the segment's end
// (in a ragged last query tile): it issues its share of the K/V DMA, waits for it and takes every
// barrier, so the workgroup's schedule is unchanged, but it skips the MFMA, softmax and LDS-read
// work and writes nothing.  Under the power cap the idle matrix and vector work is worth clock
// to the rest of the chip.
template <int D, bool kGroupB, int kMode, bool kActive>
__device__ __forceinline__ void run_item_group(const Item& it, const __bf16* __restrict__ q,
                                               const __bf16* __restrict__ k,
                                               const __bf16* __restrict__ v, const Out& out,
                                               int H, float c, bool negate_q, char* smem) {
  using G = Geo<D>;
  constexpr int kBN = G::kBN;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int gw = wave & (G::kGroupWaves - 1);  // wave inside its group
  const int hb = lane >> 5, col = lane & 31;
  const int row_bytes = H * D * 2;
  // element offsets of (first query, h) and (first key, h); byte ranges of the segment's rows
  const int64_t qbase = (it.q_start * H + it.h) * D;
  const int64_t kbase = (it.k_start * H + it.h) * D;
  const uint32_t q_bytes = (uint32_t)(it.q_len - 1) * (uint32_t)row_bytes + D * 2;
  const uint32_t k_bytes = (uint32_t)(it.k_len - 1) * (uint32_t)row_bytes + D * 2;
  __amdgpu_buffer_rsrc_t rq = make_rsrc(q + qbase, q_bytes);
  __amdgpu_buffer_rsrc_t rk = make_rsrc(k + kbase, k_bytes);
  __amdgpu_buffer_rsrc_t rv = make_rsrc(v + kbase, k_bytes);
  lds_char* const lds = (lds_char*)smem;
  auto ktile = [&](int stage) { return lds + G::kKRing + stage * G::kKTile; };
  auto vtile = [&](int stage) { return lds + G::kVRing + stage * G::kVTile; };
  const VOffsets<D> vo(lane);
  int koff[G::kKDmaMax], voff[G::kVDmaPerWave];
  if (!kGroupB) dma_offsets_k<D>(gw, lane, row_bytes, koff);
  else dma_offsets_v<D>(gw, lane, row_bytes, voff);
  // this group's fetch of the item's tile j: K_j (group A) into stage j % 4, V_j (group B) into
  // stage vstage, which the caller keeps equal to j % 3
  // Fetches run up to kFetchAhead tiles past the item's last one (into stages nobody reads).
  // Their tile index stops at the segment's end, where every row reads as zero: then no byte
  // offset exceeds (k_len + 2 kBN - 1) rows, which the host's size limit, (len + 256) rows of
  // H * D * 2 bytes below 2^31, keeps within int range at both tile sizes.
  const int seg_tiles = (it.k_len + kBN - 1) / kBN;
  auto fetch = [&](int j, int vstage) {
    const int key0 = min(it.tile_begin + j, seg_tiles) * kBN;
    if (!kGroupB) dma_k<D>(rk, key0, row_bytes, ktile(j & 3), koff, gw);
    else dma_v<D>(rv, key0, row_bytes, vtile(vstage), voff, gw);
  };
  // The same fetch in two parts, for the vector steps: each of the kSpread instructions that
  // every wave issues (without a branch) on its own, to be spread over the softmax, and then
  // the one more K instruction of some waves of group A.
  static_assert(G::kKDmaMin == G::kVDmaPerWave, "one spread for both fetching groups");
  constexpr int kSpread = G::kVDmaPerWave;
  auto fetch_one = [&](int j, int vstage, int u) {
    const int key0 = min(it.tile_begin + j, seg_tiles) * kBN;
    if (!kGroupB) dma_k_one<D>(rk, key0, row_bytes, ktile(j & 3), koff, gw, u);
    else dma_v_one<D>(rv, key0, row_bytes, vtile(vstage), voff, gw, u);
  };
  auto fetch_rest = [&](int j) {
    const int key0 = min(it.tile_begin + j, seg_tiles) * kBN;
    if (!kGroupB) dma_k<D, kSpread>(rk, key0, row_bytes, ktile(j & 3), koff, gw);
  };
  constexpr int kFetchAhead = kGroupB ? 2 : 3;  // tiles between a fetch and its first reader
  constexpr int kFetchWait = kGroupB ? G::kVDmaPerWave : G::kKDmaMin;  // fewest per wave

  // Q fragments (B operand of S^T = K Q^T): query col of this wave, channels 16kk + 8hb + 0..7
  const int qrow = it.q_begin + 32 * wave + col;
  bf16x8 qf[D / 16];
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) {
    u32x4 raw = {};
    if constexpr (kActive)
      raw = __builtin_amdgcn_raw_buffer_load_b128(rq, qrow * row_bytes + (2 * kk + hb) * 16, 0, 0);
    if (negate_q) raw ^= u32x4{0x80008000u, 0x80008000u, 0x80008000u, 0x80008000u};
    qf[kk] = __builtin_bit_cast(bf16x8, raw);
  }

  f32x16 oacc[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db) oacc[db] = f32x16{};
  f32x16 s[kBN / 32];
  bf16x8 p[kBN / 16];
  bf16x8 kp[kPreReads];  // K fragments of the next matrix step's first MFMAs
  f32x4 lacc[2] = {};  // row sums of the weights, two chains (every element: the query's sum)
  const bf16x8 sel = row_sum_selector(lane);
  float m_c = -INFINITY;

  const int ntiles = it.ntiles;
  // valid keys of the item's last tile: fewer than kBN only on the segment's ragged last tile
  const int last_keys = min(kBN, it.k_len - (it.tile_begin + ntiles - 1) * kBN);
  // vector step j: fetch tile j + kFetchAhead (a V tile into stage vst2 = (j + 2) % 3), its
  // instructions spread over the softmax S_j -> P_j, wait for the fetch of the previous vector
  // step, read the first K fragments of
  // M(j + 1); kMasked on the last tile only, which has no M(j + 1) S product.  The barrier that
  // closes the step opens the next iteration, so the loop's branch is taken before it and the
  // matrix step that follows the barrier starts with its first MFMA.
  auto vstep = [&](int j, int vst2, auto masked) {
    constexpr bool kMasked = decltype(masked)::value;
    auto issue = [&](int u) { fetch_one(j + kFetchAhead, vst2, u); };
    if constexpr (kActive) {
      softmax_tile<D, kMasked, kSpread>(s, p, m_c, oacc, lacc, c, kMasked ? last_keys : kBN, lane,
                                        issue);
    } else {
#pragma unroll
      for (int u = 0; u < kSpread; ++u) issue(u);
    }
    fetch_rest(j + kFetchAhead);
    wait_vmem<kFetchWait>();
    if (kActive && !kMasked) k_preread<D>(ktile((j + 1) & 3), kp, lane);
  };
  using Full = std::false_type;
  using Last = std::true_type;

  // prologue: tiles 0 .. kFetchAhead - 1 of this group's operand, complete before anyone reads
  // them
  fetch(0, 0);
  fetch(1, 1);
  if (!kGroupB) fetch(2, 2);
  wait_vmem<0>();
  block_sync();
  if constexpr (kActive) k_preread<D>(ktile(0), kp, lane);
  if (kGroupB) block_sync();  // group B starts one step behind

  // ---- M(0) and V(0)
  if constexpr (kActive) {
    __builtin_amdgcn_s_setprio(1);
    m_step<D, false>(ktile(0), vtile(0), vo, qf, kp, s, p, oacc, sel, lacc, lane);
    __builtin_amdgcn_s_setprio(0);
  }
  block_sync();
  if (ntiles == 1)
    vstep(0, 2, Last{});
  else
    vstep(0, 2, Full{});
  // ---- tiles 1..: K_j sits in stage j % 4; V_{j-1} in vs = (j + 2) % 3, where V_{j+2} goes next
  int vs = 0;
  auto tile = [&](int j, auto masked) {
    block_sync();  // closes V(j - 1)
    if constexpr (kActive) {
      __builtin_amdgcn_s_setprio(1);
      m_step<D, true>(ktile(j & 3), vtile(vs), vo, qf, kp, s, p, oacc, sel, lacc, lane);
      __builtin_amdgcn_s_setprio(0);
    }
    block_sync();
    vstep(j, vs, masked);
    vs = vs == 2 ? 0 : vs + 1;
  };
  int j = 1;
  for (; j < ntiles - 1; ++j) tile(j, Full{});
  if (j == ntiles - 1) tile(j, Last{});
  // ---- M(ntiles): the last product, V_{ntiles-1} in stage (ntiles - 1) % 3 = vs now
  block_sync();  // closes V(ntiles - 1)
  if constexpr (kActive) {
    row_sums(sel, p, lacc);
    pv_tile<D>(vtile(vs), vo, p, oacc);
  }
  if (!kGroupB) block_sync();  // matches group B's extra barrier at the start
  wait_vmem<0>();  // the fetches past the end must land before the workgroup leaves

  if constexpr (kActive)
    write_result<D, kMode>(it, out, oacc, lacc[0][0] + lacc[1][0], m_c, H, qrow, hb);
}

// The epilogue of one wave: O = O / l for its 32 query rows, and the row's natural log-sum-exp
// lse = (m_c + log2 l) ln 2 (m_c is in log2 units of the scaled scores).  l_tot = 0 marks an
// item without keys: O = 0 and lse = -inf.  Rows past the segment end are dropped by the
// descriptors' range checks.
template <int D, int kMode>
__device__ __forceinline__ void write_result(const Item& it, const Out& out,
                                             const f32x16 (&oacc)[D / 32], float l_tot, float m_c,
                                             int H, int qrow, int hb) {
  const float inv = l_tot > 0.0f ? 1.0f / l_tot : 0.0f;
  const float lse = l_tot > 0.0f ? (m_c + log2f(l_tot)) * kLn2 : -INFINITY;
  const uint32_t lse_bytes = ((uint32_t)(it.q_len - 1) * (uint32_t)H + 1) * 4;
  if (kMode == kFinal) {
    const int row_bytes = H * D * 2;
    const uint32_t q_bytes = (uint32_t)(it.q_len - 1) * (uint32_t)row_bytes + D * 2;
    __amdgpu_buffer_rsrc_t ro = make_rsrc(out.o + (it.q_start * H + it.h) * D, q_bytes);
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        f32x4 x = {oacc[db][4 * g4] * inv, oacc[db][4 * g4 + 1] * inv, oacc[db][4 * g4 + 2] * inv,
                   oacc[db][4 * g4 + 3] * inv};
        bf16x4 b = __builtin_convertvector(x, bf16x4);
        u32x2 w = __builtin_bit_cast(u32x2, b);
        const int ch = 32 * db + 8 * g4 + 4 * hb;  // first of 4 channels
        __builtin_amdgcn_raw_buffer_store_b64(w, ro, qrow * row_bytes + ch * 2, 0, 0);
      }
    if (out.lse != nullptr && hb == 0) {
      __amdgpu_buffer_rsrc_t rl = make_rsrc(out.lse + it.q_start * H + it.h, lse_bytes);
      __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(lse), rl, qrow * H * 4, 0, 0);
    }
  } else {
    const int64_t slab = (int64_t)out.split * out.tq;  // first row of this split's slab
    const uint32_t o_bytes = ((uint32_t)(it.q_len - 1) * (uint32_t)H + 1) * D * 4;
    __amdgpu_buffer_rsrc_t rpo = make_rsrc(out.part_o + ((slab + it.q_start) * H + it.h) * D, o_bytes);
    // Byte offsets of fp32 rows reach twice the bf16 ones: with (q_len + 256) * H * D * 2 < 2^31
    // (the host's size limit) and qrow < q_len + 256 they stay below 2^32, so they are formed in
    // unsigned 32-bit arithmetic (the buffer offset register is unsigned) without wrapping.
    const uint32_t row_off = (uint32_t)qrow * (uint32_t)(H * D) * 4u;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        f32x4 x = {oacc[db][4 * g4] * inv, oacc[db][4 * g4 + 1] * inv, oacc[db][4 * g4 + 2] * inv,
                   oacc[db][4 * g4 + 3] * inv};
        const uint32_t ch = 32 * db + 8 * g4 + 4 * hb;
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, x), rpo,
                                               __builtin_bit_cast(int, row_off + ch * 4u), 0, 0);
      }
    if (hb == 0) {
      __amdgpu_buffer_rsrc_t rl = make_rsrc(out.part_lse + (slab + it.q_start) * H + it.h, lse_bytes);
      __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(lse), rl, qrow * H * 4, 0, 0);
    }
  }
}

// ---- Thin items: a query tile of at most 32 queries (the ragged last tile of a segment).
//
// In the main schedule such a tile keeps one wave busy and seven idle for the item's whole key
// range.  Here all eight waves share it: wave w takes the 16 queries 16 (w & 1) + 0..15 of the
// tile and, of every K/V tile, the kBN / 64 blocks of 16 keys 16 (4 t + (w >> 1)) + 0..15, so
// that each K/V tile is consumed by the eight waves together.  Per 16-key block a wave computes
// S^T = K Q^T on 16x16x32 MFMAs (lane l: query l & 15, keys 4 (l >> 4) + 0..3), exponentiates
// it with its own online maximum, and accumulates O^T += V^T P^T on 16x16x16 MFMAs, whose B
// operand is exactly the lane's four weights and whose A operand (V^T for 16 channels, keys
// 4 (l >> 4) + 0..3) is one transpose read.  At the end the four waves that hold the same
// queries combine their partial (max, sum, O) through LDS, as partial results over disjoint
// key sets: O = sum_k 2^(m_k - M) O_k / sum_k 2^(m_k - M) l_k with M = max_k m_k.
//
// Schedule: one barrier per K/V tile.  Waves 0-3 fetch K tiles, waves 4-7 V tiles, both two tiles
// ahead into rings of three stages (the first three stages of the main schedule's rings); tile j
// sits in stage j % 3.  The fetch into stage (j + 2) % 3 is issued after the barrier that closed
// tile j - 1, the stage's last reader, and each wave waits for its fetch of tile j + 1 before the
// barrier that closes tile j.
constexpr int kThinQueries = 32;  // query tiles with at most this many queries take this path

__device__ __forceinline__ f32x4 mfma16k32(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma16k16(bf16x4 a, bf16x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4, a),
                                                   __builtin_bit_cast(s16x4, b), c, 0, 0, 0);
}

template <int D, int kMode>
__device__ __forceinline__ void run_thin_item(const Item& it, const __bf16* __restrict__ q,
                                              const __bf16* __restrict__ k,
                                              const __bf16* __restrict__ v, const Out& out, int H,
                                              float c, bool negate_q, char* smem) {
  using G = Geo<D>;
  constexpr int kBN = G::kBN;
  constexpr int kSub = kBN / 64;  // 16-key blocks of a wave per K/V tile
  constexpr int kCB = D / 16;     // 16-channel blocks of O
  constexpr int kWait = G::kKDmaMin;
  static_assert(G::kKDmaMin == G::kVDmaPerWave, "one wait count for both fetching groups");
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool fetch_v = wave >= kWaves / 2;
  const int gw = wave & (G::kGroupWaves - 1);
  const int qb = wave & 1, kq = wave >> 1;
  const int g = lane >> 4, i16 = lane & 15;
  const int row_bytes = H * D * 2;
  const int64_t qbase = (it.q_start * H + it.h) * D;
  const int64_t kbase = (it.k_start * H + it.h) * D;
  const uint32_t q_bytes = (uint32_t)(it.q_len - 1) * (uint32_t)row_bytes + D * 2;
  const uint32_t k_bytes = (uint32_t)(it.k_len - 1) * (uint32_t)row_bytes + D * 2;
  __amdgpu_buffer_rsrc_t rq = make_rsrc(q + qbase, q_bytes);
  __amdgpu_buffer_rsrc_t rk = make_rsrc(k + kbase, k_bytes);
  __amdgpu_buffer_rsrc_t rv = make_rsrc(v + kbase, k_bytes);
  lds_char* const lds = (lds_char*)smem;
  auto ktile = [&](int stage) { return lds + G::kKRing + stage * G::kKTile; };
  auto vtile = [&](int stage) { return lds + G::kVRing + stage * G::kVTile; };
  int koff[G::kKDmaMax], voff[G::kVDmaPerWave];
  if (!fetch_v) dma_offsets_k<D>(gw, lane, row_bytes, koff);
  else dma_offsets_v<D>(gw, lane, row_bytes, voff);
  // as in the main schedule, fetches past the segment's end clamp their tile index there
  const int seg_tiles = (it.k_len + kBN - 1) / kBN;
  auto fetch = [&](int j, int stage) {
    const int key0 = min(it.tile_begin + j, seg_tiles) * kBN;
    if (!fetch_v) dma_k<D>(rk, key0, row_bytes, ktile(stage), koff, gw);
    else dma_v<D>(rv, key0, row_bytes, vtile(stage), voff, gw);
  };

  // Q fragments (B operand of the 16x16x32 S MFMAs): query i16 of block qb, channels
  // 32 kk + 8 g + 0..7
  const int qrow = it.q_begin + 16 * qb + i16;
  bf16x8 qf[D / 32];
#pragma unroll
  for (int kk = 0; kk < D / 32; ++kk) {
    u32x4 raw = __builtin_amdgcn_raw_buffer_load_b128(rq, qrow * row_bytes + (32 * kk + 8 * g) * 2,
                                                      0, 0);
    if (negate_q) raw ^= u32x4{0x80008000u, 0x80008000u, 0x80008000u, 0x80008000u};
    qf[kk] = __builtin_bit_cast(bf16x8, raw);
  }
  // LDS offsets inside a tile: the K row of this lane in 16-key block t is 16 (4 t + kq) + i16;
  // the V rows of its transpose reads are 16 (4 t + kq) + 4 g + 0..3, and the swizzle depends on
  // the row mod 16 only, so the offset of channel block cb is the same for every block t.
  const int krow0 = (16 * kq + i16) * G::kKRow + 16 * g;
  const int vr16 = 4 * g + (i16 >> 2);
  int voffs[kCB];
#pragma unroll
  for (int cb = 0; cb < kCB; ++cb)
    voffs[cb] = (16 * kq + vr16) * G::kVRow +
                (((2 * cb + ((i16 & 3) >> 1)) ^ G::vswz(vr16)) << 4) + 8 * (i16 & 1);

  f32x4 o[kCB];
#pragma unroll
  for (int cb = 0; cb < kCB; ++cb) o[cb] = f32x4{};
  float m_c = -INFINITY, l_part = 0.0f;
  const int ntiles = it.ntiles;
  const int last_keys = min(kBN, it.k_len - (it.tile_begin + ntiles - 1) * kBN);

  fetch(0, 0);
  fetch(1, 1);
  wait_vmem<kWait>();
  block_sync();
  int st = 0;  // stage of tile j
  for (int j = 0; j < ntiles; ++j) {
    const int st2 = st == 0 ? 2 : st - 1;  // (j + 2) % 3
    fetch(j + 2, st2);
    const lds_char* kt = ktile(st);
    const lds_char* vt = vtile(st);
    f32x4 s[kSub];
#pragma unroll
    for (int t = 0; t < kSub; ++t) {
      s[t] = f32x4{};
#pragma unroll
      for (int kk = 0; kk < D / 32; ++kk) {
        const bf16x8 a = *(const lds_bf16x8*)(kt + krow0 + 64 * t * G::kKRow + 64 * kk);
        s[t] = mfma16k32(a, qf[kk], s[t]);
      }
    }
    // keys past the segment's end exist only in its last tile
    const bool masked = j == ntiles - 1 && last_keys < kBN;
    auto exps = [&](bf16x4 (&p)[kSub]) {
      unsigned any = 0;
#pragma unroll
      for (int t = 0; t < kSub; ++t)
#pragma unroll
        for (int r = 0; r < 4; r += 2) {
          float e0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[t][r], c, -m_c));
          float e1 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[t][r + 1], c, -m_c));
          const int key0 = 16 * (4 * t + kq) + 4 * g + r;
          if (masked && key0 >= last_keys) e0 = 0.0f;
          if (masked && key0 + 1 >= last_keys) e1 = 0.0f;
          f32x2 e = {e0, e1};
          bf16x2 pb = __builtin_convertvector(e, bf16x2);
          p[t][r] = pb[0];
          p[t][r + 1] = pb[1];
          any |= __builtin_bit_cast(unsigned, pb);
        }
      return any;
    };
    bf16x4 p[kSub];
    const unsigned any = exps(p);
    // as in the main schedule: the tile keeps the wave's maximum unless a weight reaches 2
    // (first tile, a score far above the maximum so far) or keys are masked
    if (masked || __builtin_amdgcn_ballot_w64((any & 0x40004000u) != 0) != 0) {
      float mt = -INFINITY;
#pragma unroll
      for (int t = 0; t < kSub; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int key = 16 * (4 * t + kq) + 4 * g + r;
          if (!masked || key < last_keys) mt = fmaxf(mt, s[t][r]);
        }
      mt = fmaxf(mt, __shfl_xor(mt, 16));
      mt = fmaxf(mt, __shfl_xor(mt, 32));
      // a wave can see no valid key at all in a masked tile (its blocks lie past the end);
      // then its maximum, and everything it has accumulated, stay as they are
      if (mt != -INFINITY) {
        const float m_new = fmaxf(m_c, __builtin_fmaf(mt, c, kBias));
        const float alpha = __builtin_amdgcn_exp2f(m_c - m_new);  // 0 while m_c = -inf
        m_c = m_new;
#pragma unroll
        for (int cb = 0; cb < kCB; ++cb) o[cb] *= alpha;
        l_part *= alpha;
      }
      exps(p);
    }
#pragma unroll
    for (int t = 0; t < kSub; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) l_part += (float)p[t][r];
#pragma unroll
    for (int t = 0; t < kSub; ++t)
#pragma unroll
      for (int cb = 0; cb < kCB; ++cb) {
        const bf16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
            (lds_bf16x4*)(vt + 64 * t * G::kVRow + voffs[cb]));
        o[cb] = mfma16k16(a, p[t], o[cb]);
      }
    wait_vmem<kWait>();
    block_sync();
    st = st == 2 ? 0 : st + 1;
  }
  wait_vmem<0>();  // the fetches past the end land before the rings are reused
  block_sync();

  // Combine the four key subsets of each query block through LDS: O_k as float
  // [wave][16 queries][D], (m_k, l_k) as float2 [wave][16 queries] after it.
  float l = l_part + __shfl_xor(l_part, 16);
  l += __shfl_xor(l, 32);
  typedef __attribute__((address_space(3))) f32x4 lds_f32x4;
  typedef __attribute__((address_space(3))) f32x2 lds_f32x2;
  typedef __attribute__((address_space(3))) float lds_float;
  lds_float* const obuf = (lds_float*)lds;
  lds_f32x2* const mlbuf = (lds_f32x2*)(lds + kWaves * 16 * D * 4);
  static_assert(kWaves * 16 * D * 4 + kWaves * 16 * 8 <= G::kLds, "combine buffer fits the rings");
#pragma unroll
  for (int cb = 0; cb < kCB; ++cb)
    *(lds_f32x4*)(obuf + (wave * 16 + i16) * D + 16 * cb + 4 * g) = o[cb];
  if (g == 0) mlbuf[wave * 16 + i16] = f32x2{m_c, l};
  __syncthreads();
  // wave w now finishes queries of block qb = w & 1, channels (D / 4) (w >> 1) + (D / 16) g + ..:
  // the waves holding block qb are qb + 2 kq2, kq2 = 0..3
  constexpr int kCh = D / 16;  // channels per lane
  const int ch0 = (D / 4) * kq + kCh * g;
  float mk[4], lk[4], big = -INFINITY;
#pragma unroll
  for (int k2 = 0; k2 < 4; ++k2) {
    const f32x2 ml = mlbuf[(qb + 2 * k2) * 16 + i16];
    mk[k2] = ml[0];
    lk[k2] = ml[1];
    big = fmaxf(big, mk[k2]);
  }
  float acc[kCh] = {}, lsum = 0.0f;
#pragma unroll
  for (int k2 = 0; k2 < 4; ++k2) {
    const float w = big == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(mk[k2] - big);
    lsum += w * lk[k2];
    const lds_float* src = obuf + ((qb + 2 * k2) * 16 + i16) * D + ch0;
#pragma unroll
    for (int x = 0; x < kCh; x += 4) {
      const f32x4 ov = *(const lds_f32x4*)(src + x);
#pragma unroll
      for (int y = 0; y < 4; ++y) acc[x + y] += w * ov[y];
    }
  }
  const float inv = lsum > 0.0f ? 1.0f / lsum : 0.0f;
  const float lse = lsum > 0.0f ? (big + log2f(lsum)) * kLn2 : -INFINITY;
  const uint32_t lse_bytes = ((uint32_t)(it.q_len - 1) * (uint32_t)H + 1) * 4;
  if (kMode == kFinal) {
    __amdgpu_buffer_rsrc_t ro = make_rsrc(out.o + qbase, q_bytes);
#pragma unroll
    for (int x = 0; x < kCh; x += 4) {
      f32x4 y = {acc[x] * inv, acc[x + 1] * inv, acc[x + 2] * inv, acc[x + 3] * inv};
      bf16x4 b = __builtin_convertvector(y, bf16x4);
      __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, b), ro,
                                            qrow * row_bytes + (ch0 + x) * 2, 0, 0);
    }
    if (out.lse != nullptr && kq == 0 && g == 0) {
      __amdgpu_buffer_rsrc_t rl = make_rsrc(out.lse + it.q_start * H + it.h, lse_bytes);
      __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(lse), rl, qrow * H * 4, 0, 0);
    }
  } else {
    const int64_t slab = (int64_t)out.split * out.tq;
    const uint32_t o_bytes = ((uint32_t)(it.q_len - 1) * (uint32_t)H + 1) * D * 4;
    __amdgpu_buffer_rsrc_t rpo = make_rsrc(out.part_o + ((slab + it.q_start) * H + it.h) * D, o_bytes);
    // unsigned offsets, as in write_result
    const uint32_t row_off = (uint32_t)qrow * (uint32_t)(H * D) * 4u;
#pragma unroll
    for (int x = 0; x < kCh; x += 4) {
      f32x4 y = {acc[x] * inv, acc[x + 1] * inv, acc[x + 2] * inv, acc[x + 3] * inv};
      __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, y), rpo,
                                             __builtin_bit_cast(int, row_off + (uint32_t)(ch0 + x) * 4u),
                                             0, 0);
    }
    if (kq == 0 && g == 0) {
      __amdgpu_buffer_rsrc_t rl = make_rsrc(out.part_lse + (slab + it.q_start) * H + it.h, lse_bytes);
      __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(lse), rl, qrow * H * 4, 0, 0);
    }
  }
}

// kThin = false compiles the thin path out, for launches that have no query tile of at most
// kThinQueries queries (the full tiles' code is then exactly that of a build without it).
template <int D, int kMode, bool kThin = true>
__device__ __forceinline__ void run_item(const Item& it, const __bf16* __restrict__ q,
                                         const __bf16* __restrict__ k, const __bf16* __restrict__ v,
                                         const Out& out, int H, float c, bool negate_q, char* smem) {
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (it.ntiles <= 0) {  // no keys in this item (the whole workgroup leaves together)
    const int lane = threadIdx.x & 63;
    f32x16 zero[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db) zero[db] = f32x16{};
    write_result<D, kMode>(it, out, zero, 0.0f, -INFINITY, H, it.q_begin + 32 * wave + (lane & 31),
                           lane >> 5);
    return;
  }
  if (kThin && it.q_len - it.q_begin <= kThinQueries) {
    run_thin_item<D, kMode>(it, q, k, v, out, H, c, negate_q, smem);
    return;
  }
  const bool active = it.q_begin + 32 * wave < it.q_len;  // some query of this wave is in range
  if (wave >= kWaves / 2) {
    if (active) run_item_group<D, true, kMode, true>(it, q, k, v, out, H, c, negate_q, smem);
    else run_item_group<D, true, kMode, false>(it, q, k, v, out, H, c, negate_q, smem);
  } else {
    if (active) run_item_group<D, false, kMode, true>(it, q, k, v, out, H, c, negate_q, smem);
    else run_item_group<D, false, kMode, false>(it, q, k, v, out, H, c, negate_q, smem);
  }
}

// kThin: L mod kBM is in 1..kThinQueries, so the last query tile of every sequence is thin.
template <int D, bool kThin>
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
attn_dense_kernel(const __bf16* __restrict__ q, const __bf16* __restrict__ k,
                  const __bf16* __restrict__ v, __bf16* __restrict__ o, int L, int H, int nq,
                  int nfull, int total, int chunk, float c, int negate_q) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int item = remap_block(blockIdx.x, total, chunk);
  // items [0, n_main): query tiles 0 .. nfull - 1 of every (sequence, head), head-major; then, when
  // nfull < nq, the last query tile of every (sequence, head)
  const int n_main = total - (nq - nfull) * (total / nq);
  int bh, qt;
  if (item < n_main) {
    bh = item / nfull;
    qt = item % nfull;
  } else {
    bh = item - n_main;
    qt = nq - 1;
  }
  Item it;
  it.q_start = it.k_start = (int64_t)(bh / H) * L;
  it.q_len = it.k_len = L;
  it.h = bh % H;
  it.q_begin = qt * kBM;
  it.tile_begin = 0;
  it.ntiles = (L + Geo<D>::kBN - 1) / Geo<D>::kBN;
  Out out{o, nullptr, nullptr, nullptr, 0, 0};
  run_item<D, kFinal, kThin>(it, q, k, v, out, H, c, negate_q != 0, smem);
}

// Packed batch: segment s has queries [cu_q[s], cu_q[s+1]) and keys [cu_k[s], cu_k[s+1])
// (cu_k == cu_q for self-attention).  Each (segment, head, query tile) is split into n_split
// items over consecutive ranges of the segment's key tiles (n_split = 1: one item, kFinal).
// plan layout (int32): [0] item count, [1] error flag, then per rank r (most keys first):
// [2 + 2r] segment index, [3 + 2r] first item of that segment.  The items of a segment are
// ordered head-major, then split, then query tile, so consecutive items share K/V ranges.
// plan = null: a batch of one segment, run without a planning kernel.  Its only valid offsets
// are {0, total_q} and {0, total_k}; every workgroup checks them and the call is a no-op
// otherwise, as with a rejected plan.
__device__ __forceinline__ bool one_segment_valid(const int32_t* __restrict__ cu_q,
                                                  const int32_t* __restrict__ cu_k, int total_q,
                                                  int total_k) {
  return cu_q[0] == 0 && cu_q[1] == total_q && cu_k[0] == 0 && cu_k[1] == total_k;
}

template <int D, int kMode>
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
attn_varlen_kernel(const __bf16* __restrict__ q, const __bf16* __restrict__ k,
                   const __bf16* __restrict__ v, Out out, const int32_t* __restrict__ cu_q,
                   const int32_t* __restrict__ cu_k, const int32_t* __restrict__ plan, int nseq,
                   int H, int n_split, int chunk, float c, int negate_q, int total_q,
                   int total_k) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  int s = 0, local;
  if (plan == nullptr) {
    if (!one_segment_valid(cu_q, cu_k, total_q, total_k)) return;
    const int total = H * n_split * ((total_q + kBM - 1) / kBM);
    if ((int)blockIdx.x >= total) return;
    local = remap_block(blockIdx.x, total, chunk);
  } else {
    const int total = plan[0];
    if ((int)blockIdx.x >= total) return;
    const int item = remap_block(blockIdx.x, total, chunk);
    // last rank whose first item is <= item (empty segments share starts with the next rank)
    int lo = 0, hi = nseq;  // plan[3 + 2*lo] <= item < plan[3 + 2*hi] (with hi = nseq as +inf)
    while (hi - lo > 1) {
      int mid = (lo + hi) >> 1;
      if (plan[3 + 2 * mid] <= item) lo = mid; else hi = mid;
    }
    s = plan[2 + 2 * lo];
    local = item - plan[3 + 2 * lo];
  }
  Item it;
  it.q_start = cu_q[s];
  it.q_len = cu_q[s + 1] - cu_q[s];
  it.k_start = cu_k[s];
  it.k_len = cu_k[s + 1] - cu_k[s];
  const int nq = (it.q_len + kBM - 1) / kBM;
  const int per_head = nq * n_split;
  it.h = local / per_head;
  const int split = (local % per_head) / nq;
  it.q_begin = (local % nq) * kBM;
  const int seg_tiles = (it.k_len + Geo<D>::kBN - 1) / Geo<D>::kBN;
  const int per_split = (seg_tiles + n_split - 1) / n_split;
  it.tile_begin = split * per_split;
  it.ntiles = max(0, min(per_split, seg_tiles - it.tile_begin));
  out.split = split;
  run_item<D, kMode>(it, q, k, v, out, H, c, negate_q != 0, smem);
}

// Combines the key ranges of a split call: for every (query row, head) with partial results
// (O_i, lse_i) over disjoint key ranges, O = sum_i exp(lse_i - lse) O_i with
// lse = log sum_i exp(lse_i) -- a softmax-weighted average over the union of the ranges.  One
// thread per 8 channels of a row; rows = Tq * H.
template <int D>
__global__ void __launch_bounds__(kMergeThreads)
attn_merge_kernel(const float* __restrict__ part_o, const float* __restrict__ part_lse,
                  int n_split, int64_t rows, __bf16* __restrict__ o, float* __restrict__ lse,
                  const int32_t* __restrict__ plan, const int32_t* __restrict__ cu_q,
                  const int32_t* __restrict__ cu_k, int total_q, int total_k) {
  constexpr int kChunks = D / 8;
  const int64_t gid = (int64_t)blockIdx.x * kMergeThreads + threadIdx.x;
  const int64_t row = gid / kChunks;
  const int c8 = (int)(gid % kChunks);
  // rejected offsets wrote no partials: O stays as is
  if (row >= rows) return;
  if (plan != nullptr ? plan[1] != 0 : !one_segment_valid(cu_q, cu_k, total_q, total_k)) return;
  float m = -INFINITY;
  for (int i = 0; i < n_split; ++i) m = fmaxf(m, part_lse[i * rows + row]);
  f32x4 a0 = {0.0f, 0.0f, 0.0f, 0.0f}, a1 = a0;
  float wsum = 0.0f;
  if (m != -INFINITY) {
    for (int i = 0; i < n_split; ++i) {
      const float w = expf(part_lse[i * rows + row] - m);  // 0 for a range without keys
      const f32x4* src = (const f32x4*)(part_o + (i * rows + row) * D + c8 * 8);
      a0 += w * src[0];
      a1 += w * src[1];
      wsum += w;
    }
  }
  const float inv = wsum > 0.0f ? 1.0f / wsum : 0.0f;
  f32x4 r0 = a0 * inv, r1 = a1 * inv;
  bf16x4 b0 = __builtin_convertvector(r0, bf16x4), b1 = __builtin_convertvector(r1, bf16x4);
  bf16x8 b = {b0[0], b0[1], b0[2], b0[3], b1[0], b1[1], b1[2], b1[3]};
  *(bf16x8*)(o + row * D + c8 * 8) = b;
  if (lse != nullptr && c8 == 0) lse[row] = wsum > 0.0f ? m + logf(wsum) : -INFINITY;
}

// ---- planning kernel: validate the offsets, order segments by key count (the cost of each of
// their items) longest first, prefix-sum the items.
constexpr int kPlanThreads = 1024;
constexpr int kPlanSortMax = 4096;  // larger batches keep their given order

__global__ void __launch_bounds__(kPlanThreads)
plan_kernel(const int32_t* __restrict__ cu_q, const int32_t* __restrict__ cu_k, int nseq,
            int max_q, int max_k, int total_q, int total_k, int H, int n_split,
            int32_t* __restrict__ plan) {
  __shared__ uint64_t keys[kPlanSortMax];
  __shared__ int32_t scan[kPlanThreads];
  const int tid = threadIdx.x;
  int bad = 0;
  if (tid == 0 && (cu_q[0] != 0 || cu_q[nseq] != total_q || cu_k[0] != 0 || cu_k[nseq] != total_k))
    bad = 1;
  // every offset within [0, total] before any difference is taken: a check of the differences
  // alone could be passed by offsets that wrap around the int32 range
  for (int s = tid; s < nseq; s += kPlanThreads) {
    const int q0 = cu_q[s], q1 = cu_q[s + 1], k0 = cu_k[s], k1 = cu_k[s + 1];
    if (q0 < 0 || q1 > total_q || q1 < q0 || q1 - q0 > max_q || k0 < 0 || k1 > total_k ||
        k1 < k0 || k1 - k0 > max_k)
      bad = 1;
  }
  if (__syncthreads_or(bad)) {
    if (tid == 0) { plan[0] = 0; plan[1] = 1; }
    return;
  }
  const bool sorted = nseq <= kPlanSortMax;
  if (sorted) {
    int n2 = 1;
    while (n2 < nseq) n2 <<= 1;
    // key: (max - keys) in the high word, index in the low word -> ascending = most keys first
    for (int i = tid; i < n2; i += kPlanThreads) {
      if (i < nseq) {
        uint32_t len = (uint32_t)(cu_k[i + 1] - cu_k[i]);
        keys[i] = ((uint64_t)(0x7fffffffu - len) << 32) | (uint32_t)i;
      } else {
        keys[i] = ~0ull;
      }
    }
    __syncthreads();
    for (int size = 2; size <= n2; size <<= 1)
      for (int stride = size >> 1; stride > 0; stride >>= 1) {
        for (int i = tid; i < n2; i += kPlanThreads) {
          int jx = i ^ stride;
          if (jx > i) {
            bool up = (i & size) == 0;
            uint64_t a = keys[i], b = keys[jx];
            if ((a > b) == up) { keys[i] = b; keys[jx] = a; }
          }
        }
        __syncthreads();
      }
  }
  // exclusive prefix sum of H * n_split * ceil(queries / kBM) in rank order, 1024 ranks per pass
  int carry = 0;
  for (int base = 0; base < nseq; base += kPlanThreads) {
    int r = base + tid;
    int seg = 0, cnt = 0;
    if (r < nseq) {
      seg = sorted ? (int)(keys[r] & 0xffffffffu) : r;
      const int lq = cu_q[seg + 1] - cu_q[seg];
      cnt = H * n_split * ((lq + kBM - 1) / kBM);
    }
    scan[tid] = cnt;
    __syncthreads();
    for (int off = 1; off < kPlanThreads; off <<= 1) {
      int add = tid >= off ? scan[tid - off] : 0;
      __syncthreads();
      scan[tid] += add;
      __syncthreads();
    }
    if (r < nseq) {
      plan[2 + 2 * r] = seg;
      plan[3 + 2 * r] = carry + scan[tid] - cnt;
    }
    carry += scan[kPlanThreads - 1];
    __syncthreads();
  }
  if (tid == 0) { plan[0] = carry; plan[1] = 0; }
}

// ---------------------------------------------------------------------------------------------
// host-side launchers

template <int D>
static hipError_t launch_dense_d(const DenseArgs& a, hipStream_t st) {
  const int nq = (a.L + kBM - 1) / kBM;
  const int total = a.B * a.H * nq;
  const float c = fabsf(a.scale) * kLog2e;
  const int tail = a.L % kBM;
  auto kern = tail != 0 && tail <= kThinQueries ? attn_dense_kernel<D, true>
                                                : attn_dense_kernel<D, false>;
  hipLaunchKernelGGL(kern, dim3(total), dim3(kThreads), Geo<D>::kLds, st, (const __bf16*)a.q,
                     (const __bf16*)a.k, (const __bf16*)a.v, (__bf16*)a.o, a.L, a.H, nq,
                     main_query_tiles(a.L), total, a.xcd_chunk, c, a.scale < 0.0f ? 1 : 0);
  return hipGetLastError();
}

template <int D>
static hipError_t launch_packed_d(const PackedArgs& a, hipStream_t st) {
  hipError_t e;
  if (a.plan != nullptr) {
    hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(kPlanThreads), 0, st, a.cu_q, a.cu_k, a.nseq,
                       a.max_q, a.max_k, a.total_q, a.total_k, a.H, a.n_split, a.plan);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const int64_t grid = packed_grid_bound(a.total_q, a.nseq, a.H, a.n_split);
  const float c = fabsf(a.scale) * kLog2e;
  const int neg = a.scale < 0.0f ? 1 : 0;
  Out out{(__bf16*)a.o, a.lse, a.part_o, a.part_lse, a.total_q, 0};
  if (a.n_split == 1) {
    hipLaunchKernelGGL((attn_varlen_kernel<D, kFinal>), dim3((unsigned)grid), dim3(kThreads),
                       Geo<D>::kLds, st, (const __bf16*)a.q, (const __bf16*)a.k,
                       (const __bf16*)a.v, out, a.cu_q, a.cu_k, a.plan, a.nseq, a.H, 1,
                       a.xcd_chunk, c, neg, a.total_q, a.total_k);
    return hipGetLastError();
  }
  hipLaunchKernelGGL((attn_varlen_kernel<D, kPartial>), dim3((unsigned)grid), dim3(kThreads),
                     Geo<D>::kLds, st, (const __bf16*)a.q, (const __bf16*)a.k, (const __bf16*)a.v,
                     out, a.cu_q, a.cu_k, a.plan, a.nseq, a.H, a.n_split, a.xcd_chunk, c, neg,
                     a.total_q, a.total_k);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t rows = (int64_t)a.total_q * a.H;
  const int64_t threads = rows * (D / 8);
  const int64_t blocks = (threads + kMergeThreads - 1) / kMergeThreads;
  hipLaunchKernelGGL((attn_merge_kernel<D>), dim3((unsigned)blocks), dim3(kMergeThreads), 0, st,
                     a.part_o, a.part_lse, a.n_split, rows, (__bf16*)a.o, a.lse, a.plan, a.cu_q,
                     a.cu_k, a.total_q, a.total_k);
  return hipGetLastError();
}

hipError_t configure_kernels() {
  hipError_t e;
  const void* dense[4] = {(const void*)attn_dense_kernel<64, false>,
                          (const void*)attn_dense_kernel<64, true>,
                          (const void*)attn_dense_kernel<128, false>,
                          (const void*)attn_dense_kernel<128, true>};
  for (int i = 0; i < 4; ++i) {
    e = hipFuncSetAttribute(dense[i], hipFuncAttributeMaxDynamicSharedMemorySize,
                            i < 2 ? Geo<64>::kLds : Geo<128>::kLds);
    if (e != hipSuccess) return e;
  }
  const void* packed[4] = {(const void*)attn_varlen_kernel<64, kFinal>,
                           (const void*)attn_varlen_kernel<64, kPartial>,
                           (const void*)attn_varlen_kernel<128, kFinal>,
                           (const void*)attn_varlen_kernel<128, kPartial>};
  for (int i = 0; i < 4; ++i) {
    e = hipFuncSetAttribute(packed[i], hipFuncAttributeMaxDynamicSharedMemorySize,
                            i < 2 ? Geo<64>::kLds : Geo<128>::kLds);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// Scratch of the allocation-free chunk call: its plan and, for split calls, the float32 partial
// results, in one array per device that lives as long as the loaded library.  Host code never
// passes `scratch` itself to a kernel (on the host the name is only a stand-in for the device
// symbol); it looks up the device address once per device and passes that.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

hipError_t scratch_address(void** ptr) {
  return hipGetSymbolAddress(ptr, HIP_SYMBOL(scratch));
}

hipError_t launch_dense(const DenseArgs& a, hipStream_t st) {
  return a.d == 64 ? launch_dense_d<64>(a, st) : launch_dense_d<128>(a, st);
}

hipError_t launch_packed(const PackedArgs& a, hipStream_t st) {
  return a.d == 64 ? launch_packed_d<64>(a, st) : launch_packed_d<128>(a, st);
}

}  // namespace tsattn
