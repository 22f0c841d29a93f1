// K4: the standalone scorer's eviction (Sec. 3.2), a score-based policy's retained set
// (Sec. 3.1 / 3.2) and the twin prevalence statistic (Sec. 2, Fig. 1b), one problem per
// workgroup.
//
// Eviction: the score is s_i = -r_i / n (Eq. 3), the sink and recent regions score highest,
// and the `budget` highest scores are retained; equal scores go to the later position first.
// Ranking by the key  0 for protected positions, r_i + 1 otherwise  (ascending) gives the
// same order.  The budget-th smallest key is found by an MSB-first radix select (11/11/10-bit
// digits, LDS histograms, 1024 or 256 threads); a pass in position order (wave ballots, slab
// by slab) then keeps the last members equal to that key.  Sequences of up to 32768 tokens
// read their counts from HBM once into LDS; longer ones stream them on every pass.
//
// Policy selection (FROM_SCORES): the same with a caller's fp32 scores.  The key is 0 for
// protected positions and otherwise the score's bits mapped to an order-reversing integer
// (higher score, smaller key; -0 as +0; NaN last), and at the cut the first members by
// position are kept.
//
// Prevalence: for each threshold tau_k, the number of tokens whose best similarity outside
// the window exceeds tau_k, i.e. that have at least one twin (Eq. 2).
#include <hip/hip_runtime.h>

#include "../twinkv_internal.h"
#include "block_select.h"

namespace twinkv {
namespace {

constexpr int kEvThreads = 256;  // prevalence

// Ascending key of an unprotected score: decreasing in the score, never 0 (the protected
// key); -0 counts as +0, and NaN takes the largest key.
__device__ inline uint32_t score_key(float f) {
  if (f != f) return 0xFFFFFFFFu;
  uint32_t u = __float_as_uint(f == 0.0f ? 0.0f : f);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);  // increasing in f
  return ~u;
}

// CAP > 0: the problem's counts (keys of its scores) are copied to LDS in the first pass
// (sequences of at most CAP tokens), so HBM is read once; CAP = 0: every pass reads global
// memory.
template <int NT, int CAP, bool FROM_SCORES>
__global__ __launch_bounds__(NT) void evict_kernel(EvictArgs a) {
  static_assert(CAP % NT == 0, "the cache holds whole slabs");
  __shared__ int s_wave[NT / 64];
  __shared__ int s_hist[kSelBins];
  __shared__ int s_pick[3];
  __shared__ int s_nan;
  __shared__ uint32_t s_c[CAP > 0 ? CAP : 1];

  const int q = blockIdx.x;
  const int h = q / a.n_seqs;
  const int s = q - h * a.n_seqs;
  const SeqInfo si = a.seqtab[s];
  const int len = si.len;
  const int64_t base = (int64_t)h * a.T + si.start;
  const int32_t* cnt = FROM_SCORES ? nullptr : a.counts + base;
  const float* psc = FROM_SCORES ? a.in_scores + base : nullptr;
  uint8_t* out = a.retained + base;
  const int rec0 = len - a.n_recent;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int budget = si.budget < len ? si.budget : len;
  const float inv_n = len > 0 ? 1.0f / (float)len : 0.0f;
  // unprotected key: count + 1, or the score's key
  auto free_key = [&](int t) -> uint32_t {
    if constexpr (CAP > 0) return s_c[t];
    else if constexpr (FROM_SCORES) return score_key(psc[t]);
    else return (uint32_t)cnt[t] + 1u;
  };
  auto key_of = [&](int t) -> uint32_t {
    return (t < a.n_sink || t >= rec0) ? 0u : free_key(t);
  };

  // ---- pass 1: the LDS copy, the Eq. 3 scores, the NaN count of the policy scores ----
  if constexpr (FROM_SCORES) {
    if (tid == 0) s_nan = 0;
    __syncthreads();
    int nan = 0;
    for (int t = tid; t < len; t += NT) {
      const float f = psc[t];
      nan += (f != f) ? 1 : 0;
      if constexpr (CAP > 0) s_c[t] = score_key(f);
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) nan += __shfl_xor(nan, off);
    if (lane == 0 && nan) atomicAdd(&s_nan, nan);
  } else if (CAP > 0 || a.scores) {
    for (int t = tid; t < len; t += NT) {
      const int32_t c = cnt[t];
      if constexpr (CAP > 0) s_c[t] = (uint32_t)c + 1u;
      if (a.scores) a.scores[base + t] = -(float)c * inv_n;
    }
  }
  __syncthreads();

  // ---- radix select of the budget-th smallest key ----
  uint32_t key_cut = 0u;
  int take_eq = 0, total_eq = 0;
  const bool cut = budget > 0 && budget < len;
  if (cut) {
    key_cut = block_select<NT>(
        len, budget,
        [&](int t, uint32_t& key) {
          key = key_of(t);
          return true;
        },
        s_hist, s_wave, s_pick, take_eq);
    // the last digit's histogram still holds the number of keys equal to the cut
    total_eq = s_hist[key_cut & 1023u];
  }

  // ---- final pass, slab by slab: the last (policy scores: the first) take_eq keys equal to
  // the cut are kept ----
  const uint64_t below = lane ? (~0ull >> (64 - lane)) : 0ull;
  int eq_before = 0;
  for (int t0 = 0; t0 < len; t0 += NT) {
    const int t = t0 + tid;
    const bool valid = t < len;
    const uint32_t key = valid ? key_of(t) : 0u;
    const bool eq = cut && valid && key == key_cut;
    const uint64_t bal = __ballot(eq);
    if (lane == 0) s_wave[wave] = __popcll(bal);
    __syncthreads();
    int rank = eq_before + __popcll(bal & below);
#pragma unroll
    for (int k = 0; k < NT / 64; ++k) {
      const int c = s_wave[k];
      rank += k < wave ? c : 0;
      eq_before += c;
    }
    __syncthreads();
    uint8_t keep;
    if (!cut) keep = budget > 0 ? 1 : 0;
    else if (key < key_cut) keep = 1;
    else if (key == key_cut) keep = (FROM_SCORES ? rank < take_eq : rank >= total_eq - take_eq) ? 1 : 0;
    else keep = 0;
    if (valid) out[t] = keep;
  }
  if (tid == 0 && a.stats) {
    int32_t* st = a.stats + 4 * (int64_t)q;
    st[0] = budget;
    if constexpr (FROM_SCORES) {
      st[1] = s_nan;
      st[2] = 0;
    } else {
      st[1] = cut ? (key_cut == 0u ? -1 : (int32_t)(key_cut - 1u)) : -1;
      st[2] = (a.pmeta && (a.pmeta[q].flags & kFlagNonfinite)) ? 2 : 0;
    }
    st[3] = 0;
  }
}

__global__ __launch_bounds__(kEvThreads) void prevalence_kernel(PrevalenceArgs a) {
  __shared__ int s_cnt[kMaxTaus];
  const int q = blockIdx.x;
  const int h = q / a.n_seqs;
  const int s = q - h * a.n_seqs;
  const SeqInfo si = a.seqtab[s];
  const float* b = a.best + (int64_t)h * a.T + si.start;
  if (threadIdx.x < kMaxTaus) s_cnt[threadIdx.x] = 0;
  __syncthreads();
  int c[kMaxTaus];
#pragma unroll
  for (int k = 0; k < kMaxTaus; ++k) c[k] = 0;
  for (int t = threadIdx.x; t < si.len; t += kEvThreads) {
    const float x = b[t];
#pragma unroll
    for (int k = 0; k < kMaxTaus; ++k) c[k] += (k < a.n_taus && x > a.taus[k]) ? 1 : 0;
  }
#pragma unroll
  for (int k = 0; k < kMaxTaus; ++k) {
    int v = c[k];
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    if ((threadIdx.x & 63) == 0 && k < a.n_taus) atomicAdd(&s_cnt[k], v);
  }
  __syncthreads();
  if (threadIdx.x < a.n_taus) a.out[(int64_t)q * a.n_taus + threadIdx.x] = s_cnt[threadIdx.x];
}

}  // namespace

template <bool FROM_SCORES>
void launch_evict_mode(const EvictArgs& a, hipStream_t st) {
  const dim3 grid((unsigned)((int64_t)a.n_heads * a.n_seqs));
  if (a.max_len <= 4096)
    hipLaunchKernelGGL((evict_kernel<256, 4096, FROM_SCORES>), grid, dim3(256), 0, st, a);
  else if (a.max_len <= 16384)
    hipLaunchKernelGGL((evict_kernel<1024, 16384, FROM_SCORES>), grid, dim3(1024), 0, st, a);
  else if (a.max_len <= 32768)
    hipLaunchKernelGGL((evict_kernel<1024, 32768, FROM_SCORES>), grid, dim3(1024), 0, st, a);
  else
    hipLaunchKernelGGL((evict_kernel<1024, 0, FROM_SCORES>), grid, dim3(1024), 0, st, a);
}

int launch_evict(const EvictArgs& a, void* stream) {
  const int64_t P = (int64_t)a.n_heads * a.n_seqs;
  if (P == 0) return hipSuccess;
  if (a.in_scores) launch_evict_mode<true>(a, (hipStream_t)stream);
  else launch_evict_mode<false>(a, (hipStream_t)stream);
  return hipGetLastError();
}

int launch_prevalence(const PrevalenceArgs& a, void* stream) {
  const int64_t P = (int64_t)a.n_heads * a.n_seqs;
  if (P == 0) return hipSuccess;
  hipLaunchKernelGGL(prevalence_kernel, dim3((unsigned)P), dim3(kEvThreads), 0,
                     (hipStream_t)stream, a);
  return hipGetLastError();
}

}  // namespace twinkv
