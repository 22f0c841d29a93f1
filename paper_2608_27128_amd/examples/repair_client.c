/*
 * A plain C client of libtwinkv: the repair pass of Sec. 3.4 on one batch, called through the
 * C ABI with device buffers from the HIP runtime (no Python, no torch).
 *
 *   repair_client <input file> <output file>
 *
 * Input (little-endian): int32 n_heads, n_seqs, d, w, n_sink, n_recent; fp32 tau;
 * int64 cu_seqlens[n_seqs + 1]; int64 budget[n_seqs]; bf16 keys[n_heads][T][d] (as uint16);
 * uint8 retained[n_heads][T], where T = cu_seqlens[n_seqs].
 * Output: uint8 s1[n_heads][T]; int32 stats[n_heads * n_seqs][4]; fp32 best_ret[n_heads][T];
 * int32 arg_ret[n_heads][T]; fp32 best_all[n_heads][T]; int32 arg_all[n_heads][T].
 *
 * Exit status 0 on success; on any failure it prints the library's or the runtime's message
 * and exits with 1.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include <hip/hip_runtime_api.h>

#include "twinkv.h"

#define HIP_OK(call)                                                              \
  do {                                                                            \
    hipError_t e_ = (call);                                                       \
    if (e_ != hipSuccess) {                                                       \
      fprintf(stderr, "%s: %s\n", #call, hipGetErrorString(e_));                  \
      exit(1);                                                                    \
    }                                                                             \
  } while (0)

static void read_all(FILE* f, void* dst, size_t bytes) {
  if (bytes && fread(dst, 1, bytes, f) != bytes) {
    fprintf(stderr, "input file too short\n");
    exit(1);
  }
}

static void* host_alloc(size_t bytes) {
  void* p = malloc(bytes ? bytes : 1);
  if (!p) {
    fprintf(stderr, "out of host memory\n");
    exit(1);
  }
  return p;
}

static void* dev_alloc(size_t bytes) {
  void* p = NULL;
  HIP_OK(hipMalloc(&p, bytes ? bytes : 16));
  return p;
}

int main(int argc, char** argv) {
  if (argc != 3) {
    fprintf(stderr, "usage: %s <input file> <output file>\n", argv[0]);
    return 1;
  }
  FILE* in = fopen(argv[1], "rb");
  if (!in) {
    perror(argv[1]);
    return 1;
  }
  int32_t hdr[6];
  float tau;
  read_all(in, hdr, sizeof hdr);
  read_all(in, &tau, sizeof tau);
  const int n_heads = hdr[0], n_seqs = hdr[1], d = hdr[2], w = hdr[3];
  const int n_sink = hdr[4], n_recent = hdr[5];
  if (n_heads < 0 || n_seqs < 0 || n_seqs > (1 << 24)) {
    fprintf(stderr, "bad header\n");
    return 1;
  }
  int64_t* cu = (int64_t*)host_alloc(sizeof(int64_t) * (size_t)(n_seqs + 1));
  int64_t* budget = (int64_t*)host_alloc(sizeof(int64_t) * (size_t)(n_seqs ? n_seqs : 1));
  read_all(in, cu, sizeof(int64_t) * (size_t)(n_seqs + 1));
  read_all(in, budget, sizeof(int64_t) * (size_t)n_seqs);
  /* the library checks the batch description on the host before anything reaches the
     device; the key and mask sizes below rely on it */
  const int64_t ws_bytes = twinkv_workspace_bytes(TWINKV_OP_REPAIR, TWINKV_BF16, d, n_heads,
                                                  n_seqs, cu);
  if (ws_bytes < 0) {
    fprintf(stderr, "twinkv_workspace_bytes: %s\n", twinkv_status_string((int)-ws_bytes));
    return 1;
  }

  const int64_t T = cu[n_seqs];
  if (T < 0 || d <= 0) {
    fprintf(stderr, "bad sequence table\n");
    return 1;
  }
  const size_t n_tok = (size_t)n_heads * (size_t)T;
  const size_t key_bytes = n_tok * (size_t)d * sizeof(uint16_t);
  const size_t n_prob = (size_t)n_heads * (size_t)n_seqs;
  uint16_t* keys = (uint16_t*)host_alloc(key_bytes);
  uint8_t* retained = (uint8_t*)host_alloc(n_tok);
  read_all(in, keys, key_bytes);
  read_all(in, retained, n_tok);
  fclose(in);

  HIP_OK(hipSetDevice(0));
  hipStream_t stream;
  HIP_OK(hipStreamCreate(&stream));
  void* d_keys = dev_alloc(key_bytes);
  uint8_t* d_ret = (uint8_t*)dev_alloc(n_tok);
  uint8_t* d_s1 = (uint8_t*)dev_alloc(n_tok);
  int32_t* d_stats = (int32_t*)dev_alloc(n_prob * 4 * sizeof(int32_t));
  float* d_best_ret = (float*)dev_alloc(n_tok * sizeof(float));
  int32_t* d_arg_ret = (int32_t*)dev_alloc(n_tok * sizeof(int32_t));
  float* d_best_all = (float*)dev_alloc(n_tok * sizeof(float));
  int32_t* d_arg_all = (int32_t*)dev_alloc(n_tok * sizeof(int32_t));
  void* d_ws = dev_alloc((size_t)ws_bytes);
  HIP_OK(hipMemcpy(d_keys, keys, key_bytes, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(d_ret, retained, n_tok, hipMemcpyHostToDevice));

  /* keys [n_heads][T][d] contiguous: strides in elements */
  const int rc = twinkv_repair(d_keys, TWINKV_BF16, d, n_heads, n_seqs, cu, T * d, d, d_ret,
                               d_s1, budget, tau, w, n_sink, n_recent, d_stats, d_best_all,
                               d_arg_all, d_best_ret, d_arg_ret, d_ws, ws_bytes, stream);
  if (rc != TWINKV_OK) {
    fprintf(stderr, "twinkv_repair: %s\n", twinkv_status_string(rc));
    return 1;
  }
  HIP_OK(hipStreamSynchronize(stream));

  uint8_t* s1 = (uint8_t*)host_alloc(n_tok);
  int32_t* stats = (int32_t*)host_alloc(n_prob * 4 * sizeof(int32_t));
  float* best_ret = (float*)host_alloc(n_tok * sizeof(float));
  int32_t* arg_ret = (int32_t*)host_alloc(n_tok * sizeof(int32_t));
  float* best_all = (float*)host_alloc(n_tok * sizeof(float));
  int32_t* arg_all = (int32_t*)host_alloc(n_tok * sizeof(int32_t));
  HIP_OK(hipMemcpy(s1, d_s1, n_tok, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(stats, d_stats, n_prob * 4 * sizeof(int32_t), hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(best_ret, d_best_ret, n_tok * sizeof(float), hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(arg_ret, d_arg_ret, n_tok * sizeof(int32_t), hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(best_all, d_best_all, n_tok * sizeof(float), hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(arg_all, d_arg_all, n_tok * sizeof(int32_t), hipMemcpyDeviceToHost));

  FILE* out = fopen(argv[2], "wb");
  if (!out) {
    perror(argv[2]);
    return 1;
  }
  const int ok = fwrite(s1, 1, n_tok, out) == n_tok &&
                 fwrite(stats, sizeof(int32_t), n_prob * 4, out) == n_prob * 4 &&
                 fwrite(best_ret, sizeof(float), n_tok, out) == n_tok &&
                 fwrite(arg_ret, sizeof(int32_t), n_tok, out) == n_tok &&
                 fwrite(best_all, sizeof(float), n_tok, out) == n_tok &&
                 fwrite(arg_all, sizeof(int32_t), n_tok, out) == n_tok;
  if (fclose(out) != 0 || !ok) {
    fprintf(stderr, "cannot write %s\n", argv[2]);
    return 1;
  }

  HIP_OK(hipFree(d_keys));
  HIP_OK(hipFree(d_ret));
  HIP_OK(hipFree(d_s1));
  HIP_OK(hipFree(d_stats));
  HIP_OK(hipFree(d_best_ret));
  HIP_OK(hipFree(d_arg_ret));
  HIP_OK(hipFree(d_best_all));
  HIP_OK(hipFree(d_arg_all));
  HIP_OK(hipFree(d_ws));
  HIP_OK(hipStreamDestroy(stream));
  free(cu);
  free(budget);
  free(keys);
  free(retained);
  free(s1);
  free(stats);
  free(best_ret);
  free(arg_ret);
  free(best_all);
  free(arg_all);
  printf("repair_client ok: %d heads, %d sequences, %lld tokens\n", n_heads, n_seqs,
         (long long)T);
  return 0;
}
