/*
 * ts_attn.h -- C ABI of the MI355X (gfx950) fused attention library libts_attn.so.
 *
 * The operation.  The paper's serving runtime runs one model call per coalesced chunk batch:
 * the ready sessions on a GPU are packed together and the model is invoked once for all of
 * them (Sec. 3.1, "Concurrent chunk execution"); every session keeps its own isolated state
 * region (Sec. 6.1, "Session memory layout").  The dominant per-step cost of such a call in a
 * video diffusion transformer is multi-head self-attention over the flattened
 * frames x height x width latent tokens, whose cost grows quadratically with the number of
 * tokens (Sec. 1).  In a packed batch each session attends only to its own tokens, so the
 * batch is a list of segments and attention is block-diagonal:
 *
 *   for segment s = tokens [cu[s], cu[s+1]), token t in s, head h, channel c:
 *     O[t,h,c] = sum_j softmax_j(scale * <Q[t,h,:], K[j,h,:]>) * V[j,h,c],  j over segment s,
 *
 * non-causal (j ranges over the whole segment).  The library computes this in one fused
 * kernel: Q K^T, an online softmax and P V on bf16 matrix cores with fp32 accumulation.
 *
 * Common conventions of every entry point
 *  - Tensors q, k, v, o: device pointers to bfloat16, contiguous, token-major [T][H][d]
 *    (row stride H*d elements).  For the dense call T = B*L, i.e. [B][L][H][d].
 *    Base pointers must be 16-byte aligned.  d must be 64 or 128.
 *  - o must not overlap q, k or v (they may overlap each other).  For chunk-vs-cache calls
 *    q/o have total_q rows and k/v total_k rows.
 *  - scale: any finite float (0 is allowed: O becomes the segment mean of V).  Typical:
 *    1/sqrt(d) rounded to float.
 *  - stream: a hipStream_t passed as void* (NULL = the legacy default stream).  Calls are
 *    asynchronous: they enqueue work on stream and return without synchronizing (exceptions:
 *    validation mode, the rare growth of the packed calls' workspace, and split partials beyond
 *    its 256 MiB, see ts_attn_fwd_varlen and ts_attn_fwd_kvcache).  Buffers must stay valid
 *    until that work completes.  Device faults surface at the caller's next synchronization.
 *  - Ownership: the caller owns every buffer; the library keeps no pointer after returning.
 *  - Errors: argument checks run on the host before any HIP call and return a ts_status
 *    without touching the device.  Empty problems (B, L, T or nseq equal to 0) are no-ops
 *    returning TS_OK.  A tensor of zero rows is never dereferenced, so its pointer may be
 *    NULL: q, k, v, o when B*L or T is 0; in the chunk call q and o when total_q is 0 and k
 *    and v when total_k is 0.  A device that is not gfx950 gives TS_ERR_UNSUPPORTED.
 *  - Determinism: results are bitwise reproducible for fixed inputs on one device (no atomics
 *    in the arithmetic, fixed reduction order), and a row's result does not depend on the
 *    other segments of the batch.
 *  - Thread safety: all entry points may be called concurrently from several host threads.
 *  - Graph capture: the attention calls only enqueue kernels on a capturing stream, so they are
 *    recorded into the HIP graph and replay with the pointers and sizes they were made with.
 *    On a capturing stream ts_attn_fwd_varlen and ts_attn_fwd_kvcache run as
 *    ts_attn_fwd_kvcache_noalloc does, on its static scratch array and under its rules (the
 *    split count it can hold, replays that overlap other calls on the device race), instead of
 *    the library's workspace, whose event waits and growth do not belong in a graph.
 *    ts_state_copy returns TS_ERR_CAPTURE on a capturing stream (it looks up where its operands
 *    live), and so does any call that would be the first on its device, since the one-time
 *    device set-up must run outside capture.
 *  - Size limits: (L or max_seqlen + 256) * H * d * 2 bytes must stay below 2^31, and the
 *    work items (H * ceil(L / 256) per sequence; H * (ceil(T / 256) + nseq) for packed
 *    batches; 16 * H * (ceil(total_q / 256) + nseq) for chunk-vs-cache calls) below 2^23.
 *    Larger problems return TS_ERR_SHAPE.
 */
#ifndef TS_ATTN_H
#define TS_ATTN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TS_ATTN_ABI_VERSION 6

typedef enum ts_status {
  TS_OK = 0,
  TS_ERR_NULL = 1,        /* a required pointer is NULL */
  TS_ERR_SHAPE = 2,       /* negative or inconsistent sizes, or above the size limit */
  TS_ERR_HEAD_DIM = 3,    /* d is not 64 or 128 */
  TS_ERR_SCALE = 4,       /* scale is NaN or infinite */
  TS_ERR_ALIGN = 5,       /* a tensor pointer is not 16-byte aligned */
  TS_ERR_ALIAS = 6,       /* o overlaps q, k or v */
  TS_ERR_UNSUPPORTED = 7, /* no usable gfx950 device */
  TS_ERR_HIP = 8,         /* a HIP runtime call or kernel launch failed */
  TS_ERR_NOMEM = 9,       /* device scratch allocation failed */
  TS_ERR_SEGMENTS = 10,   /* cu_seqlens contents invalid (reported only in validation mode) */
  TS_ERR_MEMORY = 11,     /* a copy operand is neither current-device memory nor pinned host memory */
  TS_ERR_CAPTURE = 12,    /* the call cannot be recorded into a HIP graph (see "Graph capture") */
  TS_ERR_SCRATCH = 13     /* the call needs more than the static scratch of ts_attn_fwd_kvcache_noalloc */
} ts_status;

/*
 * Dense batch: B independent sequences of L tokens each; q, k, v, o are [B][L][H][d] bf16.
 * Every sequence is one segment; the result equals ts_attn_fwd_varlen with
 * cu_seqlens = {0, L, 2L, ..., B*L}, bit for bit.
 * Returns TS_OK when the work was enqueued on stream.
 */
int ts_attn_fwd(const void* q, const void* k, const void* v, void* o, int32_t B, int32_t L,
                int32_t H, int32_t d, float scale, void* stream);

/*
 * Packed variable-length batch (one coalesced chunk batch of the paper's Sec. 3.1):
 * q, k, v, o are [T][H][d] bf16 with T = total_tokens.
 *  cu_seqlens  DEVICE pointer to nseq+1 int32 offsets: cu[0] = 0, nondecreasing,
 *              cu[nseq] = total_tokens.  Segment s is tokens [cu[s], cu[s+1]); empty
 *              segments are allowed.  Every segment length must be <= max_seqlen.
 *  nseq        number of segments (host value).
 *  max_seqlen  an upper bound of every segment length (host value; sizes the launch).
 * The library reads cu_seqlens on the device only, never synchronizing with the host.  A
 * cu_seqlens that breaks the rules above makes the call a device-side no-op (o is left
 * unwritten); with the environment variable TS_ATTN_VALIDATE=1 the call instead synchronizes
 * on stream and returns TS_ERR_SEGMENTS.
 * Work scheduling: a small planning kernel orders the segments longest first and the
 * attention kernel walks that order, so uneven batches finish with a short tail.  The plan
 * lives in a device workspace the library keeps per device (grown when a call needs more, up to
 * 256 MiB, and held until the process ends; TS_ERR_NOMEM if it cannot be grown).  The calls
 * that use it take it in turn: each one's stream waits on the GPU for an event recorded after
 * the previous one, so the host never waits, calls on one stream keep their order, and such
 * calls on different streams run one after the other.  A batch of one segment (nseq = 1)
 * needs no plan outside validation mode: the attention kernel checks its offsets against
 * {0, T} itself (a mismatch is the same device-side no-op), and a total above max_seqlen
 * returns TS_OK without device work.
 */
int ts_attn_fwd_varlen(const void* q, const void* k, const void* v, void* o,
                       const int32_t* cu_seqlens, int32_t nseq, int32_t max_seqlen,
                       int32_t total_tokens, int32_t H, int32_t d, float scale, void* stream);

/*
 * Chunk queries against per-session key/value caches, with an optional log-sum-exp output.
 * The streaming models the paper serves generate each new chunk of a session conditioned on
 * the cached state of its earlier chunks (Sec. 2, "Streaming video generation workflow"); that
 * state, the KV cache among it, lives in the session's isolated region (Sec. 6.1, "Session
 * memory layout"), and one model call serves the coalesced batch of ready sessions (Sec. 3.1).
 * Segment s of the call has
 *   queries  rows [cu_seqlens_q[s], cu_seqlens_q[s+1]) of q and o   (the session's new chunk)
 *   keys     rows [cu_seqlens_k[s], cu_seqlens_k[s+1]) of k and v   (typically its cached
 *            tokens followed by the chunk's own),
 * and every query attends to every key of its segment:
 *   O[t,h,c] = sum_j softmax_j(scale * <Q[t,h,:], K[j,h,:]>) * V[j,h,c]
 *   lse[t,h] = ln sum_j exp(scale * <Q[t,h,:], K[j,h,:]>)
 * A segment with queries but no keys gets O = 0 and lse = -inf.  With cu_seqlens_q ==
 * cu_seqlens_k (same tensors for q and k rows) it is the packed self-attention above.
 *  q, o            bf16 [total_q][H][d];  k, v  bf16 [total_k][H][d]  (DEVICE, 16-byte aligned)
 *  lse             DEVICE float32 [total_q][H] (4-byte aligned), or NULL to skip it
 *  cu_seqlens_q/k  DEVICE int32, nseq+1 entries each: start at 0, nondecreasing, end at
 *                  total_q / total_k.  Empty segments are allowed on either side.
 *  max_seqlen_q/k  upper bounds of the segment lengths (host values; size the launch)
 *  num_splits      0: chosen by the library.  n in 1..16: every (segment, head, 256-query tile)
 *                  is split into n consecutive key ranges run by separate workgroups, and a
 *                  second kernel merges their results by their log-sum-exp.  Splitting fills
 *                  the GPU when there are few query tiles (short chunks, long caches).  The
 *                  result of a split call agrees with n = 1 to float32 rounding of the partial
 *                  results, not bit for bit; n = 1 is bit-identical to ts_attn_fwd_varlen when
 *                  the offsets coincide.
 * o must not overlap q, k or v, and lse must not overlap any of q, k, v, o (TS_ERR_ALIAS).
 * Device memory: the plan and, for n > 1, float32 partial results (n * total_q * H * (d + 1)
 * floats) come from the workspace of ts_attn_fwd_varlen, or, when they exceed its 256 MiB,
 * from a stream-ordered pool allocation made and released by the call (TS_ERR_NOMEM if it
 * cannot be made; HIP's pool makes the host wait for the stream there); a call of one segment
 * needs no plan, and unsplit no
 * allocation at all (as in ts_attn_fwd_varlen, against {0, total_q} and {0, total_k}).  Bad
 * offsets behave as in ts_attn_fwd_varlen (a device no-op, or TS_ERR_SEGMENTS under
 * TS_ATTN_VALIDATE=1).  num_splits outside 0..16 and the size
 * limits above (for max_seqlen_q and max_seqlen_k each) give TS_ERR_SHAPE.
 */
int ts_attn_fwd_kvcache(const void* q, const void* k, const void* v, void* o, float* lse,
                        const int32_t* cu_seqlens_q, const int32_t* cu_seqlens_k, int32_t nseq,
                        int32_t max_seqlen_q, int32_t max_seqlen_k, int32_t total_q,
                        int32_t total_k, int32_t H, int32_t d, float scale, int32_t num_splits,
                        void* stream);

/*
 * The chunk-vs-cache call of ts_attn_fwd_kvcache without any device memory allocation, for
 * callers that cannot allocate: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc.  Arguments, result and errors are those of ts_attn_fwd_kvcache, except:
 *  - Scratch: the plan and the split partials live in one static device array of 32 MiB per
 *    device (allocated when the library's code is loaded on that device, held until the process
 *    ends), not in a per-call allocation.  A call needs
 *      align256(4 * (2 nseq + 2)) + [n > 1] (align256(4 n total_q H) + 4 n total_q H d)
 *    bytes for n key ranges.  A forced num_splits whose partials do not fit returns
 *    TS_ERR_SCRATCH before any HIP call; num_splits = 0 takes the library's choice, lowered to
 *    the largest n that fits (n = 1 always fits).
 *  - Races: every call on a device shares that device's array, and a call leaves its contents
 *    behind.  Calls on one stream are ordered; calls that may overlap on one device (different
 *    streams, or host threads without ordering between their streams) race on the array and give
 *    unspecified results.  Nothing in the array needs to start at zero: each call writes every
 *    entry it later reads.
 *  - Graph capture: allowed once the device has been set up by an earlier call of any entry
 *    point (the device's first call returns TS_ERR_CAPTURE on a capturing stream).
 *  - TS_ATTN_VALIDATE is ignored: invalid offsets always make the call a device-side no-op.
 * With the same split count n the result equals ts_attn_fwd_kvcache's bit for bit.
 */
int ts_attn_fwd_kvcache_noalloc(const void* q, const void* k, const void* v, void* o, float* lse,
                                const int32_t* cu_seqlens_q, const int32_t* cu_seqlens_k,
                                int32_t nseq, int32_t max_seqlen_q, int32_t max_seqlen_k,
                                int32_t total_q, int32_t total_k, int32_t H, int32_t d,
                                float scale, int32_t num_splits, void* stream);

/*
 * Session-state copy: suspend (device -> host), resume (host -> device) and compaction (device
 * -> device) of session state regions.  The paper's runtime suspends an idle session by copying
 * its persistent state from GPU memory to host memory and resumes it by restoring that state to
 * the GPU chosen for it (Sec. 3.1, "GPU-CPU state offloading"); only the session's isolated
 * state region moves (Sec. 6.1, "Session memory layout").  In a packed token-major batch a
 * session's cached keys (or values) are one contiguous byte range, rows
 * [cu_seqlens_k[s], cu_seqlens_k[s+1]) times H * d * 2 bytes.
 *   for every r < nranges:  dst[ranges[3r+1] .. + ranges[3r+2]) = src[ranges[3r] .. + ranges[3r+2])
 *  src, dst     base pointers: device memory of the current device, or pinned host memory
 *               (page-locked and mapped, e.g. hipHostMalloc or torch pin_memory); 16-byte
 *               aligned.  Pageable, managed or another device's memory gives TS_ERR_MEMORY.
 *  src_bytes,   sizes of the src and dst buffers; every range must lie inside them
 *  dst_bytes    (TS_ERR_SHAPE otherwise).  The two buffers must not overlap (TS_ERR_ALIAS);
 *               ranges whose destinations overlap each other leave those bytes unspecified.
 *  ranges       HOST array of 3 * nranges int64: source offset, destination offset, byte count
 *               of each range, all multiples of 16 (TS_ERR_ALIGN) and non-negative.  Read during
 *               the call only.
 * One kernel launch per 64 ranges on stream, asynchronous like every entry point: host memory
 * written by a suspend is complete once the stream reaches that point (synchronize before
 * reading it).  No device memory is allocated.  nranges = 0 is a no-op.
 */
int ts_state_copy(const void* src, int64_t src_bytes, void* dst, int64_t dst_bytes,
                  const int64_t* ranges, int32_t nranges, void* stream);

/* Human-readable name of a ts_status value (a static string; never NULL). */
const char* ts_attn_status_str(int status);

/* TS_ATTN_ABI_VERSION of the built library. */
int ts_attn_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* TS_ATTN_H */
