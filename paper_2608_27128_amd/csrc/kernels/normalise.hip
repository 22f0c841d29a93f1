// K1a: per-key inverse l2 norm (Sec. 3.2: k_hat = k / ||k||_2) and, for fp32 keys, the bf16
//      hi/lo split the similarity kernel multiplies on bf16 MFMA.
// K1b: per-problem stable partition of the positions into [S0 | evicted] column lists (the
//      S0 list padded to a multiple of kGroupAlign columns, the evicted list to whole
//      32-column chunks), carrying the inverse norm of every column.
//
// Both kernels are HBM-bound streams: K1a reads d*esize bytes and writes 4 bytes per key
// (+ 4d bytes of planes for fp32 keys); K1b reads 1 + 4 bytes and writes 8 bytes per key.
#include <hip/hip_runtime.h>

#include "../twinkv_internal.h"

namespace twinkv {
namespace {

__device__ inline uint16_t bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ inline float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// LPT lanes cooperate on one key; each lane owns 16 contiguous bytes of it.
template <int D, bool F32>
__global__ __launch_bounds__(256) void normalise_kernel(const uint8_t* __restrict__ keys,
                                                        int64_t n_tok, int64_t T, int64_t hs_bytes,
                                                        int64_t ts_bytes, float* __restrict__ rinv,
                                                        uint16_t* __restrict__ hilo) {
  constexpr int ESZ = F32 ? 4 : 2;
  constexpr int LPT = D * ESZ / 16;
  constexpr int TPB = 256 / LPT;
  static_assert(LPT <= 64 && (64 % LPT) == 0, "a key must fit inside one wave");
  const int sub = threadIdx.x % LPT;
  const int64_t tok = (int64_t)blockIdx.x * TPB + threadIdx.x / LPT;
  const bool valid = tok < n_tok;
  const int64_t h = valid ? tok / T : 0;
  const int64_t t = valid ? tok - h * T : 0;
  uint4 raw = make_uint4(0, 0, 0, 0);
  if (valid) raw = *reinterpret_cast<const uint4*>(keys + h * hs_bytes + t * ts_bytes + sub * 16);
  double ss = 0.0;
  if constexpr (F32) {
    float v[4] = {__uint_as_float(raw.x), __uint_as_float(raw.y), __uint_as_float(raw.z),
                  __uint_as_float(raw.w)};
    uint16_t hi[4], lo[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      ss += (double)v[e] * (double)v[e];
      hi[e] = bf16_rne(v[e]);
      lo[e] = bf16_rne(v[e] - bf16_to_f32(hi[e]));  // v - hi is exact in fp32
    }
    if (valid) {
      uint16_t* dst = hilo + tok * (2 * D) + sub * 4;
      uint2 phi, plo;
      phi.x = hi[0] | ((uint32_t)hi[1] << 16);
      phi.y = hi[2] | ((uint32_t)hi[3] << 16);
      plo.x = lo[0] | ((uint32_t)lo[1] << 16);
      plo.y = lo[2] | ((uint32_t)lo[3] << 16);
      *reinterpret_cast<uint2*>(dst) = phi;
      *reinterpret_cast<uint2*>(dst + D) = plo;
    }
  } else {
    const uint32_t wds[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const double a = (double)__uint_as_float(wds[e] << 16);
      const double b = (double)__uint_as_float(wds[e] & 0xFFFF0000u);
      ss += a * a + b * b;
    }
  }
#pragma unroll
  for (int off = LPT / 2; off > 0; off >>= 1) ss += __shfl_xor(ss, off, LPT);
  if (valid && sub == 0) {
    float r;
    if (!(ss < 1.0e300)) r = __uint_as_float(0x7FC00000u);  // NaN / Inf key: marker for K1b
    else if (ss > 0.0) r = (float)(1.0 / sqrt(ss));
    else r = 0.0f;                                        // zero key: similarity 0 to all
    rinv[tok] = r;
  }
}

template <int NT>
__device__ inline int block_sum(int v, int* s_red) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  const int wv = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) s_red[wv] = v;
  __syncthreads();
  int tot = 0;
#pragma unroll
  for (int k = 0; k < NT / 64; ++k) tot += s_red[k];
  __syncthreads();
  return tot;
}

constexpr int kPartThreads = 256;

__global__ __launch_bounds__(kPartThreads) void partition_kernel(
    const uint8_t* __restrict__ retained, const float* __restrict__ rinv,
    const SeqInfo* __restrict__ seqtab, int n_seqs, int64_t T, int64_t PT,
    int32_t* __restrict__ pcol, float* __restrict__ rcol, int32_t* __restrict__ prank,
    ProblemMeta* __restrict__ pmeta, int32_t* __restrict__ status) {
  __shared__ int s_red[kPartThreads / 64];
  __shared__ int s_wave[kPartThreads / 64];
  const int q = blockIdx.x;
  const int h = q / n_seqs;
  const int s = q - h * n_seqs;
  const SeqInfo si = seqtab[s];
  const int len = si.len;
  const uint8_t* ret = retained ? retained + h * T + si.start : nullptr;
  const float* rv = rinv + h * T + si.start;
  int32_t* pc = pcol + h * PT + si.perm_off;
  float* rc = rcol + h * PT + si.perm_off;
  int32_t* pr = prank + h * PT + si.perm_off;

  int cnt = 0, bad = 0;
  for (int t = threadIdx.x; t < len; t += kPartThreads) {
    cnt += (ret != nullptr && ret[t] != 0);
    bad |= !(fabsf(rv[t]) <= 3.4e38f);
  }
  const int n_ret = block_sum<kPartThreads>(cnt, s_red);
  const int any_bad = block_sum<kPartThreads>(bad, s_red);
  const int ret_pad = (n_ret + kGroupAlign - 1) / kGroupAlign * kGroupAlign;
  const int n_ev = len - n_ret;
  const int ev_pad = (n_ev + kChunk - 1) / kChunk * kChunk;

  const int lane = threadIdx.x & 63;
  const int wv = threadIdx.x >> 6;
  int ret_before_round = 0;
  for (int t0 = 0; t0 < len; t0 += kPartThreads) {
    const int t = t0 + threadIdx.x;
    const bool in = t < len;
    const bool r = in && ret != nullptr && ret[t] != 0;
    const unsigned long long bal = __ballot(r);
    const int pre = __popcll(bal & ((1ull << lane) - 1ull));
    if (lane == 0) s_wave[wv] = __popcll(bal);
    __syncthreads();
    int wbase = 0, tot = 0;
#pragma unroll
    for (int k = 0; k < kPartThreads / 64; ++k) {
      const int c = s_wave[k];
      wbase += (k < wv) ? c : 0;
      tot += c;
    }
    if (in) {
      const int ret_before = ret_before_round + wbase + pre;
      const int p = r ? ret_before : ret_pad + (t - ret_before);
      pc[p] = t;
      rc[p] = rv[t];
      pr[t] = ret_before;
    }
    ret_before_round += tot;
    __syncthreads();
  }
  for (int k = n_ret + (int)threadIdx.x; k < ret_pad; k += kPartThreads) {
    pc[k] = -1;
    rc[k] = 0.0f;
  }
  for (int k = ret_pad + n_ev + (int)threadIdx.x; k < ret_pad + ev_pad; k += kPartThreads) {
    pc[k] = -1;
    rc[k] = 0.0f;
  }
  if (threadIdx.x == 0) {
    pr[len] = n_ret;
    ProblemMeta m;
    m.n_ret = n_ret;
    m.ret_chunks = ret_pad / kChunk;
    m.total_chunks = (ret_pad + ev_pad) / kChunk;
    m.flags = any_bad ? kFlagNonfinite : 0;
    pmeta[q] = m;
    if (status) status[q] = any_bad ? 2 /* TWINKV_PROBLEM_NONFINITE */ : 0;
  }
}

// K1c: one 16-byte piece per thread; blockIdx.y = problem, blockIdx.x = group of columns.
constexpr int kGatherThreads = 256;

__global__ __launch_bounds__(kGatherThreads) void gather_columns_kernel(
    const uint16_t* __restrict__ src, int64_t src_hs, int64_t src_ts, int dcol,
    const int32_t* __restrict__ pcol, const ProblemMeta* __restrict__ pmeta,
    const SeqInfo* __restrict__ seqtab, int n_seqs, int64_t PT, uint16_t* __restrict__ pkeys) {
  const int q = blockIdx.y;
  const int h = q / n_seqs;
  const int s = q - h * n_seqs;
  const SeqInfo si = seqtab[s];
  const int ncols = pmeta[q].total_chunks * kChunk;
  const int pieces = dcol / 8;                      // 16-byte pieces per column
  const int cols_per_block = kGatherThreads / pieces;
  const int c = blockIdx.x * cols_per_block + threadIdx.x / pieces;
  const int part = threadIdx.x % pieces;
  if (c >= ncols) return;
  const int64_t p = h * PT + si.perm_off + c;
  const int j = pcol[p];
  uint4 v = make_uint4(0, 0, 0, 0);
  if (j >= 0) v = *reinterpret_cast<const uint4*>(src + h * src_hs + (int64_t)(si.start + j) * src_ts + part * 8);
  *reinterpret_cast<uint4*>(pkeys + p * dcol + part * 8) = v;
}

template <int D, bool F32>
hipError_t run_normalise(const void* keys, int n_heads, int64_t T, int64_t hs, int64_t ts,
                         float* rinv, uint16_t* hilo, hipStream_t st) {
  constexpr int ESZ = F32 ? 4 : 2;
  constexpr int LPT = D * ESZ / 16;
  constexpr int TPB = 256 / LPT;
  const int64_t n_tok = (int64_t)n_heads * T;
  if (n_tok == 0) return hipSuccess;
  const int64_t blocks = (n_tok + TPB - 1) / TPB;
  hipLaunchKernelGGL((normalise_kernel<D, F32>), dim3((unsigned)blocks), dim3(256), 0, st,
                     (const uint8_t*)keys, n_tok, T, hs * ESZ, ts * ESZ, rinv, hilo);
  return hipGetLastError();
}

}  // namespace

int launch_normalise(const void* keys, int dtype, int d, int n_heads, int64_t T,
                     int64_t head_stride, int64_t token_stride, float* rinv, uint16_t* hilo,
                     void* stream) {
  hipStream_t st = (hipStream_t)stream;
  if (dtype == 0 && d == 64) return run_normalise<64, false>(keys, n_heads, T, head_stride, token_stride, rinv, hilo, st);
  if (dtype == 0 && d == 128) return run_normalise<128, false>(keys, n_heads, T, head_stride, token_stride, rinv, hilo, st);
  if (dtype == 1 && d == 64) return run_normalise<64, true>(keys, n_heads, T, head_stride, token_stride, rinv, hilo, st);
  if (dtype == 1 && d == 128) return run_normalise<128, true>(keys, n_heads, T, head_stride, token_stride, rinv, hilo, st);
  return hipErrorInvalidValue;
}

int launch_partition(const uint8_t* retained, const float* rinv, const SeqInfo* seqtab,
                     int n_heads, int n_seqs, int64_t T, int64_t PT, int32_t* pcol, float* rcol,
                     int32_t* prank, ProblemMeta* pmeta, int32_t* status, void* stream) {
  const int64_t P = (int64_t)n_heads * n_seqs;
  if (P == 0) return hipSuccess;
  hipLaunchKernelGGL(partition_kernel, dim3((unsigned)P), dim3(kPartThreads), 0,
                     (hipStream_t)stream, retained, rinv, seqtab, n_seqs, T, PT, pcol, rcol,
                     prank, pmeta, status);
  return hipGetLastError();
}

int launch_gather_columns(const uint16_t* src, int64_t src_head_stride, int64_t src_token_stride,
                          int dcol, const int32_t* pcol, const ProblemMeta* pmeta,
                          const SeqInfo* seqtab, int n_heads, int n_seqs, int max_len, int64_t PT,
                          uint16_t* pkeys, void* stream) {
  const int64_t P = (int64_t)n_heads * n_seqs;
  if (P == 0 || max_len == 0) return hipSuccess;
  const int cols_per_block = kGatherThreads / (dcol / 8);
  const int max_cols = max_len + kPermPad;
  const unsigned gx = (unsigned)((max_cols + cols_per_block - 1) / cols_per_block);
  hipLaunchKernelGGL(gather_columns_kernel, dim3(gx, (unsigned)P), dim3(kGatherThreads), 0,
                     (hipStream_t)stream, src, src_head_stride, src_token_stride, dcol, pcol, pmeta,
                     seqtab, n_seqs, PT, pkeys);
  return hipGetLastError();
}

}  // namespace twinkv
