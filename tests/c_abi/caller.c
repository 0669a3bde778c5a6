/*
 * caller.c -- a plain C program that drives libts_attn.so through include/ts_attn.h only: HIP
 * runtime calls for memory and a stream, no C++ and no PyTorch.  Test infrastructure for
 * tests/test_gpu_c_abi.py, which writes the inputs, runs this program and compares its output
 * with the oracle.
 *
 * usage: caller IN OUT
 * IN (little-endian): int32 mode (0: ts_attn_fwd_varlen, 1: ts_attn_fwd_kvcache, 2: ts_attn_fwd
 *   with B = nseq equal segments), nseq, H, d, total_q, total_k, max_q, max_k, num_splits;
 *   float32 scale; int32 cu_q[nseq + 1]; int32 cu_k[nseq + 1]; then the bf16 bits (uint16) of
 *   q [total_q][H][d], k [total_k][H][d] and v [total_k][H][d].
 * OUT: the bf16 bits of o [total_q][H][d], then (mode 1 only) float32 lse [total_q][H].
 * Exit status 0 on success; otherwise a message on stderr names the failing call.
 */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include "ts_attn.h"

static int hip_ok(hipError_t e, const char* what) {
  if (e != hipSuccess) {
    fprintf(stderr, "caller: %s: %s\n", what, hipGetErrorString(e));
    return 0;
  }
  return 1;
}

static void* read_all(FILE* f, size_t n) {
  void* p = malloc(n ? n : 1);
  if (p != NULL && n > 0 && fread(p, 1, n, f) != n) {
    free(p);
    return NULL;
  }
  return p;
}

int main(int argc, char** argv) {
  if (argc != 3) {
    fprintf(stderr, "usage: caller IN OUT\n");
    return 2;
  }
  if (ts_attn_abi_version() != TS_ATTN_ABI_VERSION) {
    fprintf(stderr, "caller: library ABI %d, header %d\n", ts_attn_abi_version(), TS_ATTN_ABI_VERSION);
    return 1;
  }
  FILE* in = fopen(argv[1], "rb");
  if (in == NULL) {
    fprintf(stderr, "caller: cannot open %s\n", argv[1]);
    return 1;
  }
  int32_t hd[9];
  float scale;
  if (fread(hd, sizeof hd, 1, in) != 1 || fread(&scale, sizeof scale, 1, in) != 1) {
    fprintf(stderr, "caller: short header\n");
    return 1;
  }
  const int32_t mode = hd[0], nseq = hd[1], H = hd[2], d = hd[3], total_q = hd[4],
                total_k = hd[5], max_q = hd[6], max_k = hd[7], num_splits = hd[8];
  if (nseq < 1 || H < 1 || d < 1 || total_q < 0 || total_k < 0) {
    fprintf(stderr, "caller: bad header\n");
    return 1;
  }
  const size_t nq = (size_t)total_q * H * d, nk = (size_t)total_k * H * d;
  int32_t* cu_q = read_all(in, sizeof(int32_t) * (size_t)(nseq + 1));
  int32_t* cu_k = read_all(in, sizeof(int32_t) * (size_t)(nseq + 1));
  uint16_t* q = read_all(in, 2 * nq);
  uint16_t* k = read_all(in, 2 * nk);
  uint16_t* v = read_all(in, 2 * nk);
  fclose(in);
  if (cu_q == NULL || cu_k == NULL || q == NULL || k == NULL || v == NULL) {
    fprintf(stderr, "caller: short input\n");
    return 1;
  }

  hipStream_t st;
  void *dq, *dk, *dv, *dout, *dcq, *dck;
  float* dlse = NULL;
  if (!hip_ok(hipStreamCreate(&st), "hipStreamCreate") ||
      !hip_ok(hipMalloc(&dq, 2 * nq + 16), "hipMalloc q") ||
      !hip_ok(hipMalloc(&dk, 2 * nk + 16), "hipMalloc k") ||
      !hip_ok(hipMalloc(&dv, 2 * nk + 16), "hipMalloc v") ||
      !hip_ok(hipMalloc(&dout, 2 * nq + 16), "hipMalloc o") ||
      !hip_ok(hipMalloc(&dcq, sizeof(int32_t) * (size_t)(nseq + 1)), "hipMalloc cu_q") ||
      !hip_ok(hipMalloc(&dck, sizeof(int32_t) * (size_t)(nseq + 1)), "hipMalloc cu_k"))
    return 1;
  if (mode == 1 && !hip_ok(hipMalloc((void**)&dlse, sizeof(float) * (size_t)total_q * H + 4), "hipMalloc lse"))
    return 1;
  if (!hip_ok(hipMemcpy(dq, q, 2 * nq, hipMemcpyHostToDevice), "copy q") ||
      !hip_ok(hipMemcpy(dk, k, 2 * nk, hipMemcpyHostToDevice), "copy k") ||
      !hip_ok(hipMemcpy(dv, v, 2 * nk, hipMemcpyHostToDevice), "copy v") ||
      !hip_ok(hipMemcpy(dcq, cu_q, sizeof(int32_t) * (size_t)(nseq + 1), hipMemcpyHostToDevice), "copy cu_q") ||
      !hip_ok(hipMemcpy(dck, cu_k, sizeof(int32_t) * (size_t)(nseq + 1), hipMemcpyHostToDevice), "copy cu_k"))
    return 1;

  int rc;
  if (mode == 0)
    rc = ts_attn_fwd_varlen(dq, dk, dv, dout, dcq, nseq, max_q, total_q, H, d, scale, st);
  else if (mode == 1)
    rc = ts_attn_fwd_kvcache(dq, dk, dv, dout, dlse, dcq, dck, nseq, max_q, max_k, total_q,
                             total_k, H, d, scale, num_splits, st);
  else
    rc = ts_attn_fwd(dq, dk, dv, dout, nseq, total_q / nseq, H, d, scale, st);
  if (rc != TS_OK) {
    fprintf(stderr, "caller: mode %d returned %d (%s)\n", mode, rc, ts_attn_status_str(rc));
    return 1;
  }
  if (!hip_ok(hipStreamSynchronize(st), "hipStreamSynchronize")) return 1;

  uint16_t* o = malloc(2 * nq + 2);
  float* lse = mode == 1 ? malloc(sizeof(float) * (size_t)total_q * H + 4) : NULL;
  if (o == NULL || (mode == 1 && lse == NULL)) return 1;
  if (!hip_ok(hipMemcpy(o, dout, 2 * nq, hipMemcpyDeviceToHost), "copy o")) return 1;
  if (mode == 1 && !hip_ok(hipMemcpy(lse, dlse, sizeof(float) * (size_t)total_q * H,
                                     hipMemcpyDeviceToHost), "copy lse"))
    return 1;
  FILE* out = fopen(argv[2], "wb");
  if (out == NULL || fwrite(o, 2, nq, out) != nq ||
      (mode == 1 && fwrite(lse, sizeof(float), (size_t)total_q * H, out) != (size_t)total_q * H)) {
    fprintf(stderr, "caller: cannot write %s\n", argv[2]);
    return 1;
  }
  fclose(out);
  hipFree(dq); hipFree(dk); hipFree(dv); hipFree(dout); hipFree(dcq); hipFree(dck);
  if (dlse != NULL) hipFree(dlse);
  hipStreamDestroy(st);
  free(cu_q); free(cu_k); free(q); free(k); free(v); free(o); free(lse);
  return 0;
}
