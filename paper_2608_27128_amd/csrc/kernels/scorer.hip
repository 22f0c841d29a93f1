// K4: the standalone scorer's eviction (Sec. 3.2), a score-based policy's retained set
// (Sec. 3.1 / 3.2) and the twin prevalence statistic (Sec. 2, Fig. 1b), one problem per
// workgroup.
//
// Eviction: the score is s_i = -r_i / n (Eq. 3), the sink and recent regions score highest,
// and the `budget` highest scores are retained; equal scores go to the later position first.
// Ranking by the key  0 for protected positions, r_i + 1 otherwise  (ascending) gives the
// same order.  The budget-th smallest key is found by an MSB-first radix select (LDS
// histograms of 2048 bins with 1024 threads, of 256 bins with 256 threads), and the last
// members equal to it by position are kept.  Sequences of up to 32768 tokens keep their keys in LDS (evict_lds_kernel: one
// round of loads, digits below the leading bits all keys share, an early stop, the members
// equal to the cut ranked with one count per slab and wave); longer ones stream the counts
// from HBM on every pass (evict_kernel: 11-bit digits below the shared bits, ranking slab by
// slab).
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

// Sequences of any length: every pass streams the counts (scores) from HBM, 8 slabs of NT
// tokens per thread and round with the round's loads in flight together.  The first pass
// writes the Eq. 3 scores and takes the AND and OR of the keys; the selection's digits start
// below the leading bits they share and stop once the cut's bucket is taken whole; the keys
// equal to the cut are ranked slab by slab (two barriers per slab) only when some of them
// must be left out.
template <int NT, bool FROM_SCORES>
__global__ __launch_bounds__(NT) void evict_kernel(EvictArgs a) {
  constexpr int NW = NT / 64;
  constexpr int R = 8;  // slabs per round
  __shared__ int s_wave[NW];
  __shared__ uint32_t s_bits[NW][2];
  __shared__ int s_nan[NW];
  __shared__ int s_hist[2][kSelBins];  // digit histograms, used in turn
  __shared__ int s_pick[3];

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
  // protected positions take the key 0; the others count + 1, or the score's key
  auto key_of = [&](int t) -> uint32_t {
    if (t < a.n_sink || t >= rec0) return 0u;
    if constexpr (FROM_SCORES) return score_key(psc[t]);
    else return (uint32_t)cnt[t] + 1u;
  };

  for (int i = tid; i < kSelBins; i += NT) s_hist[0][i] = 0;  // visible after the next barrier

  // ---- pass 1: the AND and OR of the keys, the Eq. 3 scores, the NaN count of the policy
  // scores ----
  uint32_t kand = ~0u, kor = 0u;
  int nan = 0;
#pragma unroll 1
  for (int t0 = 0; t0 < len; t0 += R * NT) {
    float f[R];
    int32_t c[R];
#pragma unroll
    for (int u = 0; u < R; ++u) {
      const int t = t0 + u * NT + tid;
      if constexpr (FROM_SCORES) f[u] = t < len ? psc[t] : 0.0f;
      else c[u] = t < len ? cnt[t] : 0;
    }
#pragma unroll
    for (int u = 0; u < R; ++u) {
      const int t = t0 + u * NT + tid;
      if (t < len) {
        const bool pr = t < a.n_sink || t >= rec0;
        uint32_t k;
        if constexpr (FROM_SCORES) {
          nan += (f[u] != f[u]) ? 1 : 0;
          k = pr ? 0u : score_key(f[u]);
        } else {
          k = pr ? 0u : (uint32_t)c[u] + 1u;
          if (a.scores) a.scores[base + t] = -(float)c[u] * inv_n;
        }
        kand &= k;
        kor |= k;
      }
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    kand &= __shfl_xor(kand, off);
    kor |= __shfl_xor(kor, off);
    nan += __shfl_xor(nan, off);
  }
  if (lane == 0) {
    s_bits[wave][0] = kand;
    s_bits[wave][1] = kor;
    s_nan[wave] = nan;
  }
  __syncthreads();
  int n_nan = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    kand &= s_bits[w][0];
    kor |= s_bits[w][1];
    n_nan += s_nan[w];
  }

  // ---- radix select of the budget-th smallest key ----
  uint32_t key_cut = 0u;
  int take_eq = 0, total_eq = 0;
  const bool cut = budget > 0 && budget < len;
  if (cut) {
    key_cut = block_select_below<NT, 11>(
        len, budget, len, kand, kor,
        [&](int t, uint32_t& key) {
          key = key_of(t);
          return true;
        },
        s_hist, s_pick, take_eq, total_eq);
  }
  const bool rank_eq = cut && take_eq < total_eq;

  // ---- final pass: keys below the cut are kept, and of those equal to it the last take_eq
  // (policy scores: the first), ranked slab by slab when some of them must be left out ----
  const uint64_t below = lane ? (~0ull >> (64 - lane)) : 0ull;
  int eq_before = 0;
  for (int t0 = 0; t0 < len; t0 += NT) {
    const int t = t0 + tid;
    const bool valid = t < len;
    const uint32_t key = valid ? key_of(t) : 0u;
    const bool eq = cut && valid && key == key_cut;
    int rank = 0;
    if (rank_eq) {
      const uint64_t bal = __ballot(eq);
      if (lane == 0) s_wave[wave] = __popcll(bal);
      __syncthreads();
      rank = eq_before + __popcll(bal & below);
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        const int c = s_wave[w];
        rank += w < wave ? c : 0;
        eq_before += c;
      }
      __syncthreads();
    }
    uint8_t keep;
    if (!cut) keep = budget > 0 ? 1 : 0;
    else if (key < key_cut) keep = 1;
    else if (eq) keep = !rank_eq || (FROM_SCORES ? rank < take_eq : rank >= total_eq - take_eq);
    else keep = 0;
    if (valid) out[t] = keep;
  }
  if (tid == 0 && a.stats) {
    int32_t* st = a.stats + 4 * (int64_t)q;
    st[0] = budget;
    if constexpr (FROM_SCORES) {
      st[1] = n_nan;
      st[2] = 0;
    } else {
      st[1] = cut ? (key_cut == 0u ? -1 : (int32_t)(key_cut - 1u)) : -1;
      st[2] = (a.pmeta && (a.pmeta[q].flags & kFlagNonfinite)) ? 2 : 0;
    }
    st[3] = 0;
  }
}

// Sequences of at most CAP tokens: the problem's keys stay in LDS (token t at s_c[t], slab u
// of thread tid holding token u NT + tid), loaded in one round with all of a thread's loads
// in flight.  The AND and OR of the keys give the leading bits they all share; the digit
// passes of the selection (up to 11 bits over 2048 bins with 1024 threads, up to 8 over 256
// with 256, so that short problems keep more workgroups per CU; two barriers each: one wave
// picks the bin while another clears the next pass's histogram) start below those bits and
// stop once the cut's bucket is taken whole.  The keys equal to the cut are ranked by position
// only when some of them must be left out: one count per slab and wave, one scan by one wave.
template <int NT, int CAP, bool FROM_SCORES>
__global__ __launch_bounds__(NT) void evict_lds_kernel(EvictArgs a) {
  constexpr int NW = NT / 64;
  constexpr int U = CAP / NT;  // slabs
  constexpr int DBITS = NT >= 1024 ? 11 : 8;  // bits per digit
  constexpr int BINS = 1 << DBITS;
  static_assert(CAP % NT == 0 && NW >= 2, "whole slabs; one wave picks while another clears");
  __shared__ uint32_t s_c[CAP];
  __shared__ int s_hist[2][BINS];  // digit histograms, used in turn
  __shared__ int s_slab[U * NW];       // keys equal to the cut per (slab, wave), then their
                                       // exclusive prefix in position order
  __shared__ uint32_t s_bits[NW][2];   // per wave: AND and OR of its keys
  __shared__ int s_nan[NW];
  __shared__ int s_pick[3];

  const int q = blockIdx.x;
  const int h = q / a.n_seqs;
  const int s = q - h * a.n_seqs;
  const SeqInfo si = a.seqtab[s];
  const int len = si.len;
  const int64_t base = (int64_t)h * a.T + si.start;
  uint8_t* out = a.retained + base;
  const int rec0 = len - a.n_recent;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const uint64_t below = lane ? (~0ull >> (64 - lane)) : 0ull;
  const int budget = si.budget < len ? si.budget : len;
  const float inv_n = len > 0 ? 1.0f / (float)len : 0.0f;
  auto prot = [&](int t) { return t < a.n_sink || t >= rec0; };

  for (int i = tid; i < BINS; i += NT) s_hist[0][i] = 0;

  // ---- load: the keys (0 for protected positions), the Eq. 3 scores, the NaN count ----
  uint32_t kand = ~0u, kor = 0u;
  int nan = 0;
  if constexpr (FROM_SCORES) {
    float f[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int t = u * NT + tid;
      f[u] = t < len ? a.in_scores[base + t] : 0.0f;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int t = u * NT + tid;
      if (t < len) {
        nan += (f[u] != f[u]) ? 1 : 0;
        const uint32_t k = prot(t) ? 0u : score_key(f[u]);
        s_c[t] = k;
        kand &= k;
        kor |= k;
      }
    }
  } else {
    int32_t c[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int t = u * NT + tid;
      c[u] = t < len ? a.counts[base + t] : 0;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int t = u * NT + tid;
      if (t < len) {
        const uint32_t k = prot(t) ? 0u : (uint32_t)c[u] + 1u;
        s_c[t] = k;
        kand &= k;
        kor |= k;
        if (a.scores) a.scores[base + t] = -(float)c[u] * inv_n;
      }
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    kand &= __shfl_xor(kand, off);
    kor |= __shfl_xor(kor, off);
    nan += __shfl_xor(nan, off);
  }
  if (lane == 0) {
    s_bits[wave][0] = kand;
    s_bits[wave][1] = kor;
    s_nan[wave] = nan;
  }
  __syncthreads();
  int n_nan = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    kand &= s_bits[w][0];
    kor |= s_bits[w][1];
    n_nan += s_nan[w];
  }

  // ---- radix select of the budget-th smallest key: after each pass bits [hi, 32) of it are
  // known (prefix) and cnt keys share them ----
  const bool cut = budget > 0 && budget < len;
  uint32_t key_cut = 0u;
  int take_eq = 0, eq_total = 0;
  if (cut) {
    const uint32_t diff = kand ^ kor;
    int hi = diff ? 32 - __clz(diff) : 0;
    uint32_t mask = hi >= 32 ? 0u : (~0u << hi);
    uint32_t prefix = kand & mask;
    int kk = budget;
    int cnt = len;
    int buf = 0;
#pragma unroll 1
    while (hi > 0 && kk < cnt) {
      const int shift = hi > DBITS ? hi - DBITS : 0;
      const uint32_t dmask = (1u << (hi - shift)) - 1u;
#pragma unroll 4
      for (int u = 0; u < U; ++u) {
        const int t = u * NT + tid;
        const uint32_t key = t < len ? s_c[t] : 0u;
        // twin counts crowd into few bins: hist_add adds through one lane per bin
        hist_add(t < len && (key & mask) == prefix, (int)((key >> shift) & dmask), s_hist[buf]);
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
    if (kk == cnt) {
      // every key sharing bits [hi, 32) with the budget-th is kept: cut at the largest key
      // with those bits, all keys equal to it kept
      key_cut = prefix | ~mask;
      take_eq = cnt;
    } else {
      key_cut = prefix;  // hi == 0: the budget-th key itself; cnt keys equal it
      take_eq = kk;
    }
    eq_total = cnt;
  }

  // ---- keys equal to the cut, ranked by position (slab, then wave, then lane) when some of
  // them must be left out ----
  const bool rank_eq = cut && take_eq < eq_total;
  if (rank_eq) {
#pragma unroll 4
    for (int u = 0; u < U; ++u) {
      const int t = u * NT + tid;
      const uint64_t bal = __ballot(t < len && s_c[t] == key_cut);
      if (lane == 0) s_slab[u * NW + wave] = (int)__popcll(bal);
    }
    __syncthreads();
    if (wave == 0) {
      constexpr int E = U * NW;
      constexpr int EPL = (E + 63) / 64;
      int v[EPL];
      int sum = 0;
#pragma unroll
      for (int j = 0; j < EPL; ++j) {
        const int e = lane * EPL + j;
        v[j] = e < E ? s_slab[e] : 0;
        sum += v[j];
      }
      int inc = sum;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const int y = __shfl_up(inc, off);
        if (lane >= off) inc += y;
      }
      int run = inc - sum;
#pragma unroll
      for (int j = 0; j < EPL; ++j) {
        const int e = lane * EPL + j;
        if (e < E) s_slab[e] = run;
        run += v[j];
      }
    }
    __syncthreads();
  }

  // ---- final pass: keys below the cut are kept, and of those equal to it the last take_eq
  // (policy scores: the first) ----
#pragma unroll 4
  for (int u = 0; u < U; ++u) {
    const int t = u * NT + tid;
    const uint32_t key = t < len ? s_c[t] : 0u;
    const bool eq = cut && t < len && key == key_cut;
    int rank = 0;
    if (rank_eq) rank = s_slab[u * NW + wave] + (int)__popcll(__ballot(eq) & below);
    uint8_t keep;
    if (!cut) keep = budget > 0 ? 1 : 0;
    else if (key < key_cut) keep = 1;
    else if (eq) keep = !rank_eq || (FROM_SCORES ? rank < take_eq : rank >= eq_total - take_eq);
    else keep = 0;
    if (t < len) out[t] = keep;
  }
  if (tid == 0 && a.stats) {
    int32_t* st = a.stats + 4 * (int64_t)q;
    st[0] = budget;
    if constexpr (FROM_SCORES) {
      st[1] = n_nan;
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
    hipLaunchKernelGGL((evict_lds_kernel<256, 4096, FROM_SCORES>), grid, dim3(256), 0, st, a);
  else if (a.max_len <= 16384)
    hipLaunchKernelGGL((evict_lds_kernel<1024, 16384, FROM_SCORES>), grid, dim3(1024), 0, st, a);
  else if (a.max_len <= 32768)
    hipLaunchKernelGGL((evict_lds_kernel<1024, 32768, FROM_SCORES>), grid, dim3(1024), 0, st, a);
  else
    hipLaunchKernelGGL((evict_kernel<1024, FROM_SCORES>), grid, dim3(1024), 0, st, a);
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
