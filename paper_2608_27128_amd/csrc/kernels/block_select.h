// Block-wide building blocks of the per-problem selection kernels (repair, scorer eviction):
// an exclusive scan, histogram adds, one wave's pick of a digit's bin and two MSB-first radix
// selects over 32-bit keys (fixed 11/11/10-bit digits; or digits below the leading bits all
// keys share, with an early stop), LDS histograms of up to 2048 bins.  NT threads per block:
// 1024 for long sequences, 256 when every sequence is short.
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

// One histogram increment per lane with mem set.  The lanes that share the bin of the first
// such lane add through that lane alone (keys are often concentrated in a few bins, where
// plain LDS atomics from one instruction would serialise on one address); the others add
// their own.  All lanes of the wave must call it.  (Handling more leaders per call, up to 4
// or 8 distinct bins, measured slower on every selection kernel.)
__device__ inline void hist_add(bool mem, int bin, int* s_hist) {
  const uint64_t act = __ballot(mem);
  if (act == 0ull) return;
  const int leader = __ffsll((long long)act) - 1;
  const int lbin = __builtin_amdgcn_readlane(bin, leader);
  const bool peer = mem && bin == lbin;
  const uint64_t peers = __ballot(peer);
  if ((int)(threadIdx.x & 63) == leader) atomicAdd(&s_hist[lbin], (int)__popcll(peers));
  if (mem && !peer) atomicAdd(&s_hist[bin], 1);
}

// One wave's part of a digit pass over BINS bins (call from one whole wave): the bin that
// holds the rank-th smallest member (1-based), the members in lower bins and the members in
// that bin go to s_pick[0..2].  Lane l sums bins BINS/64 l .. BINS/64 (l + 1) - 1; the lane
// whose range holds the rank-th member walks its bins.
template <int BINS = kSelBins>
__device__ inline void wave_pick_bin(const int* hist, int rank, int* s_pick) {
  constexpr int BPL = BINS / 64;
  static_assert(BPL % 4 == 0, "whole 16-byte reads per lane");
  const int lane = threadIdx.x & 63;
  int hb[BPL];
  int sum = 0;
#pragma unroll
  for (int j = 0; j < BPL / 4; ++j) {
    const int4 h4 = *reinterpret_cast<const int4*>(&hist[BPL * lane + 4 * j]);
    hb[4 * j + 0] = h4.x;
    hb[4 * j + 1] = h4.y;
    hb[4 * j + 2] = h4.z;
    hb[4 * j + 3] = h4.w;
    sum += h4.x + h4.y + h4.z + h4.w;
  }
  int inc = sum;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int y = __shfl_up(inc, off);
    if (lane >= off) inc += y;
  }
  int before = inc - sum;
  if (before < rank && rank <= inc) {
    int bin = -1, c = 0;
#pragma unroll
    for (int e = 0; e < BPL; ++e) {
      if (bin < 0) {
        if (rank <= before + hb[e]) {
          bin = BPL * lane + e;
          c = hb[e];
        } else {
          before += hb[e];
        }
      }
    }
    s_pick[0] = bin;
    s_pick[1] = before;
    s_pick[2] = c;
  }
}

// Zero BINS bins (call from one whole wave).
template <int BINS = kSelBins>
__device__ inline void wave_clear_bins(int* hist) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int j = 0; j < BINS / 256; ++j)
    *reinterpret_cast<int4*>(&hist[BINS / 64 * lane + 4 * j]) = make_int4(0, 0, 0, 0);
}

// Among the members of [0, len) (member(t, key) returns true and sets key), the rank-th
// smallest key (1-based rank, 1 <= rank <= number of members).  Returns that key; take_eq
// receives how many members equal to it are needed so that exactly `rank` are taken when
// every member below it is taken, and eq_total (if non-null) how many members equal it.
// Workspace: s_hist[kSelBins], s_wave[NT / 64], s_pick[3].  Every thread of the block must
// call it.
// Digits: three passes of 11/11/10 bits over kSelBins = 2048 bins, every thread scanning two
// bins (the streaming repair pass of sequences over 32768 tokens: measured faster there than
// block_select_below, whose one-wave pick costs more per pass when all three passes run).
struct SelDigits {
  static constexpr int PASSES = 3, BINS = kSelBins;
  static __device__ constexpr int shift(int p) { return p == 0 ? 21 : (p == 1 ? 10 : 0); }
  static __device__ constexpr int width(int p) { return p == 2 ? 10 : 11; }
};

template <int NT, class Member>
__device__ inline uint32_t block_select(int len, int rank, Member member, int* s_hist,
                                        int* s_wave, int* s_pick, int& take_eq,
                                        int* eq_total = nullptr) {
  using Dg = SelDigits;
  static_assert(Dg::BINS % NT == 0 || NT % Dg::BINS == 0, "bins and threads must tile");
  const int tid = threadIdx.x;
  uint32_t prefix = 0u, mask = 0u;
  int kk = rank;
#pragma unroll
  for (int pass = 0; pass < Dg::PASSES; ++pass) {
    const int shift = Dg::shift(pass);
    const uint32_t dmask = (1u << Dg::width(pass)) - 1u;
    for (int b = tid; b < Dg::BINS; b += NT) s_hist[b] = 0;
    __syncthreads();
    // uniform trip count over the block, so that every lane of a wave takes part in the
    // ballots of hist_add
    for (int t0 = 0; t0 < len; t0 += NT) {
      const int t = t0 + tid;
      uint32_t key = 0u;
      const bool mem = t < len && member(t, key) && (key & mask) == prefix;
      hist_add(mem, (int)((key >> shift) & dmask), s_hist);
    }
    __syncthreads();
    // thread tid owns the BPT consecutive bins from BPT * tid (none past the last bin)
    constexpr int BPT = Dg::BINS >= NT ? Dg::BINS / NT : 1;
    int hs[BPT];
    int sum = 0;
#pragma unroll
    for (int k = 0; k < BPT; ++k) {
      hs[k] = BPT * tid + k < Dg::BINS ? s_hist[BPT * tid + k] : 0;
      sum += hs[k];
    }
    int dummy;
    int before = sel_exclusive_scan<NT>(sum, s_wave, dummy);
#pragma unroll
    for (int k = 0; k < BPT; ++k) {
      if (before < kk && kk <= before + hs[k]) {
        s_pick[0] = BPT * tid + k;
        s_pick[1] = before;
        s_pick[2] = hs[k];
      }
      before += hs[k];
    }
    __syncthreads();
    kk -= s_pick[1];
    prefix |= (uint32_t)s_pick[0] << shift;
    mask |= dmask << shift;
    if (pass == Dg::PASSES - 1 && eq_total != nullptr) *eq_total = s_pick[2];
    __syncthreads();
  }
  take_eq = kk;
  return prefix;
}

// Among the members of [0, len) (member(t, key) returns true and sets key; n_members of them,
// their keys' AND kand and OR kor), the rank-th smallest key (1-based, 1 <= rank <
// n_members): MSB-first digits of up to DBITS bits below the leading bits every member key
// shares, over 2^DBITS LDS bins, each pass reading the members afresh (8 slabs of NT tokens
// per round, their loads in flight together); two barriers per pass, one wave picking the
// bin while another clears the other histogram; the passes stop once the rank-th key's bucket
// is taken whole.  Returns the cut key; take_eq receives how many members equal to it are
// taken and eq_total how many there are (take_eq == eq_total: every member up to the cut is
// taken).  s_hist: two histograms of 2^DBITS ints, the first zero and visible to every thread
// on entry.  Every thread of the block must call it.
template <int NT, int DBITS, class Member>
__device__ inline uint32_t block_select_below(int len, int rank, int n_members, uint32_t kand,
                                              uint32_t kor, Member member, int (*s_hist)[1 << DBITS],
                                              int* s_pick, int& take_eq, int& eq_total) {
  constexpr int BINS = 1 << DBITS;
  constexpr int R = 8;  // slabs per round
  static_assert(NT >= 128, "one wave picks while another clears");
  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const uint32_t diff = kand ^ kor;
  int hi = diff ? 32 - __clz(diff) : 0;
  uint32_t mask = hi >= 32 ? 0u : (~0u << hi);
  uint32_t prefix = kand & mask;
  int kk = rank, cnt = n_members, buf = 0;
#pragma unroll 1
  while (hi > 0 && kk < cnt) {
    const int shift = hi > DBITS ? hi - DBITS : 0;
    const uint32_t dmask = (1u << (hi - shift)) - 1u;
    // uniform trip count over the block, so that every lane of a wave takes part in the
    // ballots of hist_add
#pragma unroll 1
    for (int t0 = 0; t0 < len; t0 += R * NT) {
      uint32_t key[R];
      bool mem[R];
#pragma unroll
      for (int u = 0; u < R; ++u) {
        const int t = t0 + u * NT + tid;
        key[u] = 0u;
        mem[u] = t < len && member(t, key[u]);
      }
#pragma unroll
      for (int u = 0; u < R; ++u)
        hist_add(mem[u] && (key[u] & mask) == prefix, (int)((key[u] >> shift) & dmask),
                 s_hist[buf]);
    }
    __syncthreads();
    if (wave == 0) wave_pick_bin<BINS>(s_hist[buf], kk, s_pick);
    else if (wave == 1) wave_clear_bins<BINS>(s_hist[buf ^ 1]);
    __syncthreads();
    kk -= s_pick[1];
    prefix |= (uint32_t)s_pick[0] << shift;
    mask |= dmask << shift;
    cnt = s_pick[2];
    hi = shift;
    buf ^= 1;
  }
  eq_total = cnt;
  if (kk == cnt) {
    // every member sharing bits [hi, 32) with the rank-th key is taken: cut at the largest
    // key with those bits
    take_eq = cnt;
    return prefix | ~mask;
  }
  take_eq = kk;  // hi == 0: the rank-th key itself; cnt members equal it
  return prefix;
}

}  // namespace twinkv
