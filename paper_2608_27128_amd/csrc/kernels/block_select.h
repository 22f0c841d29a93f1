// Block-wide building blocks of the per-problem selection kernels (repair, scorer eviction):
// an exclusive scan and an MSB-first radix select over 32-bit keys with 11/11/10-bit digits
// (three passes over the data, LDS histograms of 2048 bins).  NT threads per block: 1024 for
// long sequences, 256 when every sequence is short.
#pragma once

#include <hip/hip_runtime.h>

namespace twinkv {

constexpr int kSelBins = 2048;
constexpr int kSelMaxThreads = 1024;

// Exclusive prefix sum of v over the block of NT threads; `total` receives the block sum.
// s_wave holds NT / 64 ints.
template <int NT>
__device__ inline int sel_exclusive_scan(int v, int* s_wave, int& total) {
  const int lane = threadIdx.x & 63;
  const int wv = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int y = __shfl_up(x, off);
    if (lane >= off) x += y;
  }
  if (lane == 63) s_wave[wv] = x;
  __syncthreads();
  int base = 0;
  total = 0;
#pragma unroll
  for (int k = 0; k < NT / 64; ++k) {
    const int t = s_wave[k];
    base += (k < wv) ? t : 0;
    total += t;
  }
  __syncthreads();
  return base + x - v;
}

// Among the members of [0, len) (member(t, key) returns true and sets key), the rank-th
// smallest key (1-based rank, 1 <= rank <= number of members).  Returns that key; take_eq
// receives how many members equal to it are needed so that exactly `rank` are taken when
// every member below it is taken.  Workspace: s_hist[kSelBins], s_wave[NT / 64], s_pick[2].
// Every thread of the block must call it.
template <int NT, class Member>
__device__ inline uint32_t block_select(int len, int rank, Member member, int* s_hist,
                                        int* s_wave, int* s_pick, int& take_eq) {
  const int tid = threadIdx.x;
  uint32_t prefix = 0u, mask = 0u;
  int kk = rank;
  const int shifts[3] = {21, 10, 0};
  const int widths[3] = {11, 11, 10};
#pragma unroll
  for (int pass = 0; pass < 3; ++pass) {
    const int shift = shifts[pass];
    const uint32_t dmask = (1u << widths[pass]) - 1u;
    for (int b = tid; b < kSelBins; b += NT) s_hist[b] = 0;
    __syncthreads();
    for (int t = tid; t < len; t += NT) {
      uint32_t key;
      if (member(t, key) && (key & mask) == prefix) atomicAdd(&s_hist[(key >> shift) & dmask], 1);
    }
    __syncthreads();
    // thread tid owns the BPT consecutive bins from BPT * tid
    constexpr int BPT = kSelBins / NT;
    int hs[BPT];
    int sum = 0;
#pragma unroll
    for (int k = 0; k < BPT; ++k) {
      hs[k] = s_hist[BPT * tid + k];
      sum += hs[k];
    }
    int dummy;
    int before = sel_exclusive_scan<NT>(sum, s_wave, dummy);
#pragma unroll
    for (int k = 0; k < BPT; ++k) {
      if (before < kk && kk <= before + hs[k]) {
        s_pick[0] = BPT * tid + k;
        s_pick[1] = before;
      }
      before += hs[k];
    }
    __syncthreads();
    kk -= s_pick[1];
    prefix |= (uint32_t)s_pick[0] << shift;
    mask |= dmask << shift;
    __syncthreads();
  }
  take_eq = kk;
  return prefix;
}

}  // namespace twinkv
