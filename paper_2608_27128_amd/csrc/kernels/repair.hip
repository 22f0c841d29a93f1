// K3: the composable repair pass of Sec. 3.4 for one problem per workgroup.
//
//   orphan  i not in S0, b_i < tau
//   donor   j in S0, outside [0, n_sink) and [len - n_recent, len), b_j >= tau
//   m = min(|O|, |D|); admit the m orphans of lowest (b, position), evict the m donors of
//   highest b (ties: lowest position first); S1 has exactly |S0| members.
//
// Since m = min(|O|, |D|), at least one side is taken whole; the other side needs the
// m-th smallest key, found by an MSB-first radix select on order-preserving float keys, then
// a pass in position order that takes exactly the remaining members equal to that key
// (ranked by wave ballots) when some of them must be left out.
//  * Up to 4096 tokens per sequence (repair_short_kernel, 256 threads): the tokens stay in
//    registers, the cut side's keys are compacted into LDS and selected with 8-bit digit
//    passes below the leading bits they all share.
//  * 4097 to 32768 tokens (repair_reg_kernel, 1024 threads): b and S0 are read from HBM
//    once, in one round of loads, into 16 or 32 slots per thread (the keys of b in registers
//    up to 16384 tokens, in LDS beyond); digit passes of up to 11 bits over 2048 LDS bins,
//    below the leading bits the cut side's keys share, read the slots.
//  * Longer sequences (repair_kernel, 1024 threads): fixed 11/11/10-bit digits over the whole
//    key, every pass streaming b and S0 from global memory.
#include <hip/hip_runtime.h>

#include "../twinkv_internal.h"
#include "block_select.h"

// Threads per problem of the short-sequence path (build-time tuning; 256 measured best
// against 128 and 512 on 1k-4k-token sequences).
// Keys of sequences of up to 16384 tokens in LDS instead of registers (build-time tuning;
// registers measured faster: 64 against 68 us on the 36x8x16k cache).
#ifndef TWINKV_K3_16K_LDS_KEYS
#define TWINKV_K3_16K_LDS_KEYS false
#endif
#ifndef TWINKV_K3_SHORT_THREADS
#define TWINKV_K3_SHORT_THREADS 256
#endif

namespace twinkv {
namespace {

// Order-preserving map of fp32 onto uint32 (+0 and -0 map to the same key).
__device__ inline uint32_t ord_key(float x) {
  const uint32_t u = __float_as_uint(x == 0.0f ? 0.0f : x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Sequences of any length: every pass reads b and S0 from global memory.
//
// Latency: the count pass and the final pass take U tokens per thread per round, with all of
// a round's loads issued before any is used; the counts are summed per wave from ballots and
// reduced across the block once; the position-ordered ranking of members equal to the cut
// key (two barriers per slab) only runs when some of them must be left out.
template <int NT>
__global__ __launch_bounds__(NT) void repair_kernel(RepairArgs a) {
  constexpr int U = 8;
  constexpr int NW = NT / 64;
  __shared__ int s_wave[NW];
  __shared__ int s_red[4][NW];
  __shared__ int s_hist[kSelBins];
  __shared__ int s_pick[3];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int q = blockIdx.x;
  const int h = q / a.n_seqs;
  const int s = q - h * a.n_seqs;
  const SeqInfo si = a.seqtab[s];
  const int len = si.len;
  const int64_t base = (int64_t)h * a.T + si.start;
  const float* b = a.b + base;
  const uint8_t* s0 = a.s0 + base;
  uint8_t* s1 = a.s1 + base;
  const float tau = a.tau;
  const int rec0 = len - a.n_recent;  // first recent-window position
  auto is_orphan = [&](int t, float x, bool r) { return !r && x < tau; };
  auto is_donor = [&](int t, float x, bool r) {
    return r && !(t < a.n_sink || t >= rec0) && x >= tau;
  };
  auto bval = [&](int t) -> float { return b[t]; };
  auto rbit = [&](int t) -> bool { return s0[t] != 0; };

#ifdef TWINKV_DEBUG
  // Debug build: the histogram starts as poison.
  for (int i = tid; i < kSelBins; i += NT) s_hist[i] = -1;
  __syncthreads();
#endif
  // ---- pass 1: counts, U slabs of NT tokens per round ----
  // per-wave counts from ballots (wave-uniform scalars)
  int c_ret = 0, c_o = 0, c_d = 0, bad = 0;
  for (int t0 = 0; t0 < len; t0 += U * NT) {
    float x[U];
    bool r[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int t = t0 + u * NT + tid;
      x[u] = t < len ? b[t] : 0.0f;
      r[u] = t < len && s0[t] != 0;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int slab = t0 + u * NT;
      if (slab >= len) break;  // uniform over the block
      const int t = slab + tid;
      const bool valid = t < len;
      const uint64_t rb = __ballot(r[u]);
      c_ret += (int)__popcll(rb);
      c_o += (int)__popcll(__ballot(valid && is_orphan(t, x[u], r[u])));
      c_d += (int)__popcll(__ballot(valid && is_donor(t, x[u], r[u])));
      bad |= (int)(__ballot(valid && !(fabsf(x[u]) <= 3.4e38f)) != 0ull);
    }
  }
  if (lane == 0) {
    s_red[0][wave] = c_ret;
    s_red[1][wave] = c_o;
    s_red[2][wave] = c_d;
    s_red[3][wave] = bad;
  }
  __syncthreads();
  int tot_ret = 0, tot_o = 0, tot_d = 0, tot_bad = 0;
#pragma unroll
  for (int k = 0; k < NW; ++k) {
    tot_ret += s_red[0][k];
    tot_o += s_red[1][k];
    tot_d += s_red[2][k];
    tot_bad |= s_red[3][k];
  }

  int status = 0;
  if (tot_bad || (a.pmeta && (a.pmeta[q].flags & kFlagNonfinite))) status = 2;
  else if (si.budget >= 0 && tot_ret != si.budget) status = 1;
  const int m = status == 0 ? min(tot_o, tot_d) : 0;
  const bool sel_o = m > 0 && tot_o > m;  // orphans must be cut at the m-th
  const bool sel_d = m > 0 && tot_d > m;  // donors must be cut at the m-th

  // ---- radix select of the m-th smallest key on the side that is cut ----
  uint32_t key_cut = 0xFFFFFFFFu;
  int take_eq = 0, eq_total = 0;
  if (sel_o || sel_d) {
    auto member = [&](int t, uint32_t& key) {
      const float x = bval(t);
      const bool r = rbit(t);
      if (sel_o) {
        key = ord_key(x);
        return is_orphan(t, x, r);
      }
      key = ~ord_key(x);
      return is_donor(t, x, r);
    };
    key_cut = block_select<NT>(len, m, member, s_hist, s_wave, s_pick, take_eq, &eq_total);
  }
  // every member equal to the cut key is taken unless some must be left out
  const bool rank_eq = (sel_o || sel_d) && take_eq < eq_total;

  // the decision for one token, given the rank of an equal-to-cut member among its peers
  auto decide = [&](int t, float x, bool r, int rank) -> uint8_t {
    uint8_t out = r ? 1 : 0;
    if (m > 0) {
      if (is_orphan(t, x, r)) {
        bool admit = true;
        if (sel_o) {
          const uint32_t key = ord_key(x);
          admit = key < key_cut || (key == key_cut && rank < take_eq);
        }
        if (admit) out = 1;
      } else if (is_donor(t, x, r)) {
        bool evict = true;
        if (sel_d) {
          const uint32_t key = ~ord_key(x);
          evict = key < key_cut || (key == key_cut && rank < take_eq);
        }
        if (evict) out = 0;
      }
    }
    return out;
  };

  if (!rank_eq) {
    // ---- final pass without ranking: U tokens per thread per round, no barriers ----
    for (int t0 = 0; t0 < len; t0 += U * NT) {
      float x[U];
      bool r[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int t = t0 + u * NT + tid;
        x[u] = t < len ? bval(t) : 0.0f;
        r[u] = t < len && rbit(t);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int t = t0 + u * NT + tid;
        if (t < len) s1[t] = decide(t, x[u], r[u], 0);
      }
    }
  } else {
    // ---- final pass, slab by slab: members equal to the cut key are ranked by position ----
    const uint64_t below = lane ? (~0ull >> (64 - lane)) : 0ull;
    int eq_before = 0;
    for (int t0 = 0; t0 < len; t0 += NT) {
      const int t = t0 + tid;
      const bool valid = t < len;
      const float x = valid ? bval(t) : 0.0f;
      const bool r = valid && rbit(t);
      bool eq = false;
      if (valid) {
        if (sel_o) eq = is_orphan(t, x, r) && ord_key(x) == key_cut;
        else eq = is_donor(t, x, r) && ~ord_key(x) == key_cut;
      }
      const uint64_t bal = __ballot(eq);
      if (lane == 0) s_wave[wave] = __popcll(bal);
      __syncthreads();
      int rank = eq_before + __popcll(bal & below);
#pragma unroll
      for (int k = 0; k < NW; ++k) {
        const int c = s_wave[k];
        rank += k < wave ? c : 0;
        eq_before += c;
      }
      __syncthreads();
      if (valid) s1[t] = decide(t, x, r, rank);
    }
  }
  if (tid == 0) {
    int32_t* st = a.stats + 4 * (int64_t)q;
    st[0] = status == 0 ? tot_o : 0;
    st[1] = status == 0 ? tot_d : 0;
    st[2] = m;
    st[3] = status;
  }
}

// Raw buffer loads whose range check returns 0 past the last byte of the sequence: the loads
// of a thread's slots need no branches.
constexpr int kRawBufferFlags = 0x00020000;  // 32-bit data format, gfx9 family
__device__ inline __amdgpu_buffer_rsrc_t seq_rsrc(const void* base, int nbytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, nbytes,
                                           kRawBufferFlags);
}

// Short sequences (at most kShortLen tokens): every thread keeps its kShortLen / NT tokens
// (token u * NT + tid in slot u) in registers for the whole problem as order-preserving keys
// and orphan / donor / S0 bits, so b and S0 are read from HBM once, in one round of branch-
// free loads, and no LDS copy is needed.  The counts are popcounts reduced once.  When one
// side is cut, each wave compacts its members' keys into its own part of LDS (ballots, no
// atomics); the AND and OR of all of them give the leading bits they share, and the
// selection runs 8-bit digit passes over the bits below those only, each with two barriers
// (one wave scans the histogram while another clears the next one), stopping once the
// bucket of the m-th key is taken whole.  The final pass decides every token from the
// registers; members equal to the cut key are ranked by position (slot-major, then thread)
// only when some must be left out.  At most 64 VGPRs, so that 8 workgroups share a CU.
// (Layouts with runs of 4 or 16 consecutive tokens per thread, read with 16-byte loads,
// measured slower: a problem's rows are rarely 16-byte aligned.)
constexpr int kShortLen = 4096;

template <int NT>
__global__ __launch_bounds__(NT, 8) void repair_short_kernel(RepairArgs a) {
  constexpr int U = kShortLen / NT;
  constexpr int NW = NT / 64;
  constexpr int WCAP = 64 * U;  // members one wave can hold
  static_assert(U <= 32, "the S0 and member bits of a thread's slots fit one word each");
  static_assert(NW >= 2, "one wave scans the histogram while another clears the next one");
  // wave w's members of the cut side at s_key[w * WCAP, w * WCAP + its count)
  __shared__ uint32_t s_key[kShortLen];
  __shared__ int s_hist[2][256];  // digit histograms, used in turn
  __shared__ uint64_t s_red[NW];
  __shared__ uint32_t s_bits[NW][2];  // per wave: AND and OR of its members' keys
  __shared__ int s_wave[NW];
  __shared__ int s_pick[3];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const uint64_t below = lane ? (~0ull >> (64 - lane)) : 0ull;
  const int q = blockIdx.x;
  const int h = q / a.n_seqs;
  const int s = q - h * a.n_seqs;
  const SeqInfo si = a.seqtab[s];
  const int len = si.len;
  const int64_t base = (int64_t)h * a.T + si.start;
  const float* b = a.b + base;
  const uint8_t* s0 = a.s0 + base;
  uint8_t* s1 = a.s1 + base;
  const float tau = a.tau;
  const int rec0 = len - a.n_recent;
  auto is_orphan = [&](int t, float x, bool r) { return !r && x < tau; };
  auto is_donor = [&](int t, float x, bool r) {
    return r && !(t < a.n_sink || t >= rec0) && x >= tau;
  };

#ifdef TWINKV_DEBUG
  for (int i = tid; i < kShortLen; i += NT) s_key[i] = ~0u;
  for (int i = tid; i < 256; i += NT) s_hist[1][i] = -1;
#endif
  for (int i = tid; i < 256; i += NT) s_hist[0][i] = 0;  // visible after the count barrier

  // ---- load (all loads of a thread in flight together, none past the sequence; raw buffer
  // loads return 0 there, so no branches) and count ----
  float x[U];
  uint32_t rb = 0u;  // bit u: token u * NT + tid is in S0
  {
    const __amdgpu_buffer_rsrc_t rs_b = seq_rsrc(b, 4 * len);
    const __amdgpu_buffer_rsrc_t rs_r = seq_rsrc(s0, len);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int t = u * NT + tid;
      x[u] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rs_b, 4 * t, 0, 0));
      rb |= (uint32_t)(__builtin_amdgcn_raw_buffer_load_b8(rs_r, t, 0, 0) != 0) << u;
    }
  }
  uint32_t orph = 0u, don = 0u;  // bit u: the token of slot u is an orphan / a donor
  int bad = 0;
  uint32_t k[U];  // order-preserving keys of b (the floats are not kept)
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int t = u * NT + tid;
    const bool valid = t < len;
    const bool r = (rb >> u) & 1u;
    orph |= (uint32_t)(valid && is_orphan(t, x[u], r)) << u;
    don |= (uint32_t)(valid && is_donor(t, x[u], r)) << u;
    bad |= valid && !(fabsf(x[u]) <= 3.4e38f);
    k[u] = ord_key(x[u]);
  }
  const int c_ret = __builtin_popcount(rb), c_o = __builtin_popcount(orph);
  const int c_d = __builtin_popcount(don);
  // one 64-bit word per thread (16 bits a count: a block sums at most kShortLen), summed
  // over the wave and then over the waves
  uint64_t pk = (uint64_t)c_ret | ((uint64_t)c_o << 16) | ((uint64_t)c_d << 32) |
                ((uint64_t)bad << 48);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) pk += __shfl_xor(pk, off);
  if (lane == 0) s_red[wave] = pk;
  __syncthreads();
  uint64_t tot = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) tot += s_red[w];
  const int tot_ret = (int)(tot & 0xFFFFu), tot_o = (int)((tot >> 16) & 0xFFFFu);
  const int tot_d = (int)((tot >> 32) & 0xFFFFu);
  const bool tot_bad = ((tot >> 48) & 0xFFFFu) != 0;

  int status = 0;
  if (tot_bad || (a.pmeta && (a.pmeta[q].flags & kFlagNonfinite))) status = 2;
  else if (si.budget >= 0 && tot_ret != si.budget) status = 1;
  const int m = status == 0 ? min(tot_o, tot_d) : 0;
  const bool sel_o = m > 0 && tot_o > m;
  const bool sel_d = m > 0 && tot_d > m;

  uint32_t key_cut = 0xFFFFFFFFu;
  int take_eq = 0, eq_total = 0;
  if (sel_o || sel_d) {
    // ---- the cut side's keys (descending donors as complemented keys), compacted per wave
    // into the wave's own part of LDS, in no particular order; the AND and the OR of all of
    // them give the leading bits they share, which no digit pass needs to look at ----
    const uint32_t mbits = sel_o ? orph : don;  // bit u: the token of slot u is a member
    const uint32_t flip = sel_o ? 0u : ~0u;
    uint32_t* wkeys = s_key + wave * WCAP;
    int nmem = 0;  // members of this wave so far (uniform over the wave)
    uint32_t kand = ~0u, kor = 0u;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const bool mem = (mbits >> u) & 1u;
      const uint64_t bal = __ballot(mem);
      const uint32_t key = k[u] ^ flip;
      if (mem) {
        wkeys[nmem + (int)__popcll(bal & below)] = key;
        kand &= key;
        kor |= key;
      }
      nmem += (int)__popcll(bal);
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      kand &= __shfl_xor(kand, off);
      kor |= __shfl_xor(kor, off);
    }
    if (lane == 0) {
      s_bits[wave][0] = kand;
      s_bits[wave][1] = kor;
    }
    __syncthreads();
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      kand &= s_bits[w][0];
      kor |= s_bits[w][1];
    }
    // ---- radix select, MSB first, in digits of up to 8 bits below the shared bits: after
    // each pass, bits [hi, 32) of the kk-th smallest key are known (prefix) and cnt members
    // share them.  The passes stop early once every one of those cnt is taken. ----
    const uint32_t diff = kand ^ kor;
    int hi = diff ? 32 - __clz(diff) : 0;
    uint32_t mask = hi >= 32 ? 0u : (~0u << hi);
    uint32_t prefix = kand & mask;
    int kk = m;
    int cnt = sel_o ? tot_o : tot_d;
    int buf = 0;
#pragma unroll 1
    while (hi > 0 && kk < cnt) {
      const int shift = hi > 8 ? hi - 8 : 0;
      const uint32_t dmask = (1u << (hi - shift)) - 1u;
      for (int i0 = 0; i0 < nmem; i0 += 64) {
        const int i = i0 + lane;
        if (i < nmem) {
          const uint32_t key = wkeys[i];
          if ((key & mask) == prefix) atomicAdd(&s_hist[buf][(key >> shift) & dmask], 1);
        }
      }
      __syncthreads();
      if (wave == 0) {
        // bins 4 lane .. 4 lane + 3; the lane whose range holds the kk-th key picks its bin
        const int4 h4 = *reinterpret_cast<const int4*>(&s_hist[buf][4 * lane]);
        const int sum = h4.x + h4.y + h4.z + h4.w;
        int inc = sum;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
          const int y = __shfl_up(inc, off);
          if (lane >= off) inc += y;
        }
        int before = inc - sum;
        if (before < kk && kk <= inc) {
          int bin = 4 * lane, c = h4.x;
          if (kk > before + c) { before += c; ++bin; c = h4.y; }
          if (kk > before + c) { before += c; ++bin; c = h4.z; }
          if (kk > before + c) { before += c; ++bin; c = h4.w; }
          s_pick[0] = bin;
          s_pick[1] = before;
          s_pick[2] = c;
        }
      } else if (wave == 1) {
        // the next pass's histogram
        *reinterpret_cast<int4*>(&s_hist[buf ^ 1][4 * lane]) = make_int4(0, 0, 0, 0);
      }
      __syncthreads();
      kk -= s_pick[1];
      prefix |= (uint32_t)s_pick[0] << shift;
      mask |= dmask << shift;
      cnt = s_pick[2];
      hi = shift;
      buf ^= 1;
    }
    if (kk == cnt) {
      // every member sharing bits [hi, 32) with the kk-th key is taken: cut at the largest
      // key with those bits, all members equal to it taken
      key_cut = prefix | ~mask;
      take_eq = cnt;
    } else {
      key_cut = prefix;  // hi == 0: the kk-th key itself; cnt members equal it
      take_eq = kk;
    }
    eq_total = cnt;
  }
  const bool rank_eq = (sel_o || sel_d) && take_eq < eq_total;

  // ---- final pass from the registers ----
  // (opaque: the slots' bits are read back from the three words, instead of the compiler
  // keeping the per-slot predicates of the load phase alive, and spilled, until here)
  asm volatile("" : "+v"(rb), "+v"(orph), "+v"(don));
  const uint32_t memb = sel_o ? orph : don;  // the cut side (when one side is cut)
  const uint32_t flip = sel_o ? 0u : ~0u;
  int eq_before = 0;
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int t = u * NT + tid;
    const bool r = (rb >> u) & 1u;
    const bool orphan = (orph >> u) & 1u;
    const bool donor = (don >> u) & 1u;
    const uint32_t key = k[u] ^ flip;
    int rank = 0;
    if (rank_eq) {
      // position order: slot u, then thread; uniform over the block
      const bool eq = ((memb >> u) & 1u) && key == key_cut;
      const uint64_t bal = __ballot(eq);
      if (lane == 0) s_wave[wave] = (int)__popcll(bal);
      __syncthreads();
      rank = eq_before + (int)__popcll(bal & below);
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        const int c = s_wave[w];
        rank += w < wave ? c : 0;
        eq_before += c;
      }
      __syncthreads();
    }
    // a member of the cut side is taken when its key is below the cut, or equal to it and
    // among the first take_eq of those by position; the other side is taken whole
    const bool cut_side = sel_o ? orphan : (sel_d ? donor : false);
    const bool taken = !cut_side || key < key_cut || (key == key_cut && rank < take_eq);
    uint8_t out = r ? 1 : 0;
    if (m > 0 && taken) {
      if (orphan) out = 1;
      else if (donor) out = 0;
    }
    if (t < len) s1[t] = out;
  }
  if (tid == 0) {
    int32_t* st = a.stats + 4 * (int64_t)q;
    st[0] = status == 0 ? tot_o : 0;
    st[1] = status == 0 ? tot_d : 0;
    st[2] = m;
    st[3] = status;
  }
}


// Sequences of up to NT * U tokens with every token in a slot of its own thread (token
// u * NT + tid in slot u of thread tid): in registers, or (KL) in an LDS array that b is
// loaded into directly.  A slot keeps the order-preserving key of b_t (orphan: b_t < tau, i.e.
// key < key(tau); donor: key >= key(tau)), never the float itself.  When one side is cut, the
// AND and OR of its keys give the leading bits they all share, and the selection's digit
// passes (up to 11 bits, 2048 LDS bins, two barriers each: one wave scans the histogram while
// another clears the next one) start below those bits and stop once the bucket of the m-th
// key is taken whole.  When m = 0 the final pass copies S0.
template <int NT, int U, bool KL>
__global__ __launch_bounds__(NT) void repair_reg_kernel(RepairArgs a) {
  constexpr int NW = NT / 64;
  static_assert(U <= 32, "the S0 and member bits of a thread's slots fit one word each");
  static_assert((int64_t)NT * U < 65536, "the packed 16-bit counts hold a problem's sums");
  static_assert(NW >= 2, "one wave scans the histogram while another clears the next one");
  __shared__ int s_hist[2][kSelBins];  // digit histograms, used in turn
  // keys in LDS (KL) instead of registers: slot u of thread tid at s_key[u * NT + tid]
  __shared__ uint32_t s_key[KL ? NT * U : 1];
  __shared__ uint64_t s_red[NW];
  __shared__ uint32_t s_bits[NW][2];  // per wave: AND and OR of its members' keys
  __shared__ int s_wave[NW];
  __shared__ int s_pick[3];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const uint64_t below = lane ? (~0ull >> (64 - lane)) : 0ull;
  const int q = blockIdx.x;
  const int h = q / a.n_seqs;
  const int s = q - h * a.n_seqs;
  const SeqInfo si = a.seqtab[s];
  const int len = si.len;
  const int64_t base = (int64_t)h * a.T + si.start;
  uint8_t* s1 = a.s1 + base;
  const uint32_t ktau = ord_key(a.tau);
  const int rec0 = len - a.n_recent;
  auto prot = [&](int t) { return t < a.n_sink || t >= rec0; };

#ifdef TWINKV_DEBUG
  for (int i = tid; i < kSelBins; i += NT) s_hist[1][i] = -1;
#endif
  for (int i = tid; i < kSelBins; i += NT) s_hist[0][i] = 0;  // visible after the count barrier

  // ---- load (all loads of a thread in flight together, none past the sequence) and count.
  // With the keys in LDS, b goes straight into s_key by 4-byte direct loads (no registers,
  // one round with the S0 bytes) and is turned into keys in place; a slot index then need not
  // be a constant, so the slot loops unroll partially (UR slots at a time).
  constexpr int UR = KL ? 4 : U;
  uint32_t kr[KL ? 1 : U];  // order-preserving keys of b (in registers unless KL)
  auto key_of = [&](int u) -> uint32_t {
    if constexpr (KL) return s_key[u * NT + tid];
    else return kr[u];
  };
  uint32_t rb = 0u;  // bit u: token u * NT + tid is in S0
  uint32_t orph = 0u, don = 0u;  // bit u: the token of slot u is an orphan / a donor
  int bad = 0;
  {
    const __amdgpu_buffer_rsrc_t rs_b = seq_rsrc(a.b + base, 4 * len);
    const __amdgpu_buffer_rsrc_t rs_r = seq_rsrc(a.s0 + base, len);
    float x[KL ? 1 : U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int t = u * NT + tid;
      if constexpr (KL) {
        // lane l of the wave lands at s_key[u * NT + 64 wave + l], its own slot u
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            rs_b, (void __attribute__((address_space(3)))*)(s_key + u * NT + 64 * wave), 4,
            4 * t, 0, 0, 0);
      } else {
        x[u] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rs_b, 4 * t, 0, 0));
      }
      rb |= (uint32_t)(__builtin_amdgcn_raw_buffer_load_b8(rs_r, t, 0, 0) != 0) << u;
    }
    if constexpr (KL) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
#pragma unroll UR
    for (int u = 0; u < U; ++u) {
      const int t = u * NT + tid;
      const bool valid = t < len;
      const bool r = (rb >> u) & 1u;
      float xv;
      if constexpr (KL) xv = __uint_as_float(s_key[u * NT + tid]);
      else xv = x[u];
      const uint32_t ku = ord_key(xv);
      bad |= !(fabsf(xv) <= 3.4e38f);  // slots past the end hold 0
      orph |= (uint32_t)(valid && !r && ku < ktau) << u;
      don |= (uint32_t)(valid && r && !prot(t) && ku >= ktau) << u;
      if constexpr (KL) s_key[u * NT + tid] = ku;
      else kr[u] = ku;
    }
  }
  const int c_ret = __builtin_popcount(rb), c_o = __builtin_popcount(orph);
  const int c_d = __builtin_popcount(don);
  uint64_t pk = (uint64_t)c_ret | ((uint64_t)c_o << 16) | ((uint64_t)c_d << 32) |
                ((uint64_t)bad << 48);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) pk += __shfl_xor(pk, off);
  if (lane == 0) s_red[wave] = pk;
  __syncthreads();
  uint64_t tot = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) tot += s_red[w];
  const int tot_ret = (int)(tot & 0xFFFFu), tot_o = (int)((tot >> 16) & 0xFFFFu);
  const int tot_d = (int)((tot >> 32) & 0xFFFFu);
  const bool tot_bad = ((tot >> 48) & 0xFFFFu) != 0;

  int status = 0;
  if (tot_bad || (a.pmeta && (a.pmeta[q].flags & kFlagNonfinite))) status = 2;
  else if (si.budget >= 0 && tot_ret != si.budget) status = 1;
  const int m = status == 0 ? min(tot_o, tot_d) : 0;
  const bool sel_o = m > 0 && tot_o > m;
  const bool sel_d = m > 0 && tot_d > m;
  // the cut side's members and their selection keys: ascending b for orphans, descending b
  // for donors (the key complemented)
  const uint32_t memb = sel_o ? orph : don;
  const uint32_t flip = sel_o ? 0u : ~0u;

  uint32_t key_cut = 0xFFFFFFFFu;
  int take_eq = 0, eq_total = 0;
  if (sel_o || sel_d) {
    // ---- the AND and OR of the cut side's keys: the leading bits they all share ----
    uint32_t kand = ~0u, kor = 0u;
    {
      // opaque: the slots' keys and member tests are made in each loop over the slots, not
      // hoisted out of it into registers held for all slots
      uint32_t fl = flip, mb = memb;
      asm volatile("" : "+v"(fl), "+v"(mb));
#pragma unroll UR
      for (int u = 0; u < U; ++u) {
        const uint32_t key = key_of(u) ^ fl;
        const bool mem = (mb >> u) & 1u;
        kand &= mem ? key : ~0u;
        kor |= mem ? key : 0u;
      }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      kand &= __shfl_xor(kand, off);
      kor |= __shfl_xor(kor, off);
    }
    if (lane == 0) {
      s_bits[wave][0] = kand;
      s_bits[wave][1] = kor;
    }
    __syncthreads();
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      kand &= s_bits[w][0];
      kor |= s_bits[w][1];
    }
    // ---- MSB-first radix select in digits of up to 11 bits below the shared bits, over the
    // slots: after each pass bits [hi, 32) of the kk-th smallest key are known (prefix) and
    // cnt members share them; the passes stop once every one of those cnt is taken ----
    const uint32_t diff = kand ^ kor;
    int hi = diff ? 32 - __clz(diff) : 0;
    uint32_t mask = hi >= 32 ? 0u : (~0u << hi);
    uint32_t prefix = kand & mask;
    int kk = m;
    int cnt = sel_o ? tot_o : tot_d;
    int buf = 0;
#pragma unroll 1
    while (hi > 0 && kk < cnt) {
      const int shift = hi > 11 ? hi - 11 : 0;
      const uint32_t dmask = (1u << (hi - shift)) - 1u;
      uint32_t fl = flip, mb = memb;
      asm volatile("" : "+v"(fl), "+v"(mb));
#pragma unroll UR
      for (int u = 0; u < U; ++u) {
        const uint32_t key = key_of(u) ^ fl;
        if (((mb >> u) & 1u) && (key & mask) == prefix)
          atomicAdd(&s_hist[buf][(key >> shift) & dmask], 1);
      }
      __syncthreads();
      if (wave == 0) {
        // bins 32 lane .. 32 lane + 31; the lane whose range holds the kk-th key picks its bin
        constexpr int BPL = kSelBins / 64;
        int hb[BPL];
        int sum = 0;
#pragma unroll
        for (int j = 0; j < BPL / 4; ++j) {
          const int4 h4 = *reinterpret_cast<const int4*>(&s_hist[buf][BPL * lane + 4 * j]);
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
        if (before < kk && kk <= inc) {
          int bin = -1, c = 0;
#pragma unroll
          for (int e = 0; e < BPL; ++e) {
            if (bin < 0) {
              if (kk <= before + hb[e]) {
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
      } else if (wave == 1) {
        // the next pass's histogram
#pragma unroll
        for (int j = 0; j < kSelBins / 256; ++j)
          *reinterpret_cast<int4*>(&s_hist[buf ^ 1][kSelBins / 64 * lane + 4 * j]) =
              make_int4(0, 0, 0, 0);
      }
      __syncthreads();
      kk -= s_pick[1];
      prefix |= (uint32_t)s_pick[0] << shift;
      mask |= dmask << shift;
      cnt = s_pick[2];
      hi = shift;
      buf ^= 1;
    }
    if (kk == cnt) {
      // every member sharing bits [hi, 32) with the kk-th key is taken: cut at the largest
      // key with those bits, all members equal to it taken
      key_cut = prefix | ~mask;
      take_eq = cnt;
    } else {
      key_cut = prefix;  // hi == 0: the kk-th key itself; cnt members equal it
      take_eq = kk;
    }
    eq_total = cnt;
  }
  const bool rank_eq = (sel_o || sel_d) && take_eq < eq_total;

  if (m == 0) {
    // ---- nothing moves: S1 is S0 ----
#pragma unroll UR
    for (int u = 0; u < U; ++u) {
      const int t = u * NT + tid;
      if (t < len) s1[t] = (uint8_t)((rb >> u) & 1u);
    }
  } else {
  // ---- final pass from the registers ----
  int eq_before = 0;
#pragma unroll UR
  for (int u = 0; u < U; ++u) {
    const int t = u * NT + tid;
    const bool r = (rb >> u) & 1u;
    const bool orphan = (orph >> u) & 1u;
    const bool donor = (don >> u) & 1u;
    const uint32_t key = key_of(u) ^ flip;
    int rank = 0;
    if (rank_eq) {
      // position order: slot u, then thread; uniform over the block
      const bool eq = ((memb >> u) & 1u) && key == key_cut;
      const uint64_t bal = __ballot(eq);
      if (lane == 0) s_wave[wave] = (int)__popcll(bal);
      __syncthreads();
      rank = eq_before + (int)__popcll(bal & below);
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        const int c = s_wave[w];
        rank += w < wave ? c : 0;
        eq_before += c;
      }
      __syncthreads();
    }
    // a member of the cut side is taken when its key is below the cut, or equal to it and
    // among the first take_eq of those by position; the other side is taken whole
    const bool cut_side = sel_o ? orphan : (sel_d ? donor : false);
    const bool taken = !cut_side || key < key_cut || (key == key_cut && rank < take_eq);
    uint8_t out = r ? 1 : 0;
    if (m > 0 && taken) {
      if (orphan) out = 1;
      else if (donor) out = 0;
    }
    if (t < len) s1[t] = out;
  }
  }
  if (tid == 0) {
    int32_t* st = a.stats + 4 * (int64_t)q;
    st[0] = status == 0 ? tot_o : 0;
    st[1] = status == 0 ? tot_d : 0;
    st[2] = m;
    st[3] = status;
  }
}

}  // namespace

int launch_repair(const RepairArgs& a, void* stream) {
  const int64_t P = (int64_t)a.n_heads * a.n_seqs;
  if (P == 0) return hipSuccess;
  hipStream_t st = (hipStream_t)stream;
  const dim3 grid((unsigned)P);
  // the smallest kernel whose slots hold the longest sequence; beyond 32768 tokens, streaming
  if (a.max_len <= kShortLen)
    hipLaunchKernelGGL((repair_short_kernel<TWINKV_K3_SHORT_THREADS>), grid,
                       dim3(TWINKV_K3_SHORT_THREADS), 0, st, a);
  else if (a.max_len <= 16384)
    hipLaunchKernelGGL((repair_reg_kernel<1024, 16, TWINKV_K3_16K_LDS_KEYS>), grid, dim3(1024),
                       0, st, a);
  else if (a.max_len <= 32768)
    hipLaunchKernelGGL((repair_reg_kernel<1024, 32, true>), grid, dim3(1024), 0, st, a);
  else
    hipLaunchKernelGGL((repair_kernel<1024>), grid, dim3(1024), 0, st, a);
  return hipGetLastError();
}

}  // namespace twinkv
