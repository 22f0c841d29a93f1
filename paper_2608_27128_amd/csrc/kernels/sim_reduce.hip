// K2: fused cosine-similarity contraction with two masked row max / argmax reductions.
//
// For every problem (head, sequence) and token i it computes, without materialising the
// N x N matrix (Sec. 3.2 Eq. 1 and the twin window; Sec. 3.4 Eq. 4):
//   best over all j with |i-j| > w of sim(i, j)        -> best_all / arg_all
//   best over j in S0 with |i-j| > w of sim(i, j)      -> best_ret / arg_ret  (= b_i(S0))
// with sim(i, j) = (k_i . k_j) * r_i * r_j, r = 1 / ||k||.
//
// Mapping onto gfx950:
//  * One workgroup owns RB = NWAVES * NSUB * 32 consecutive rows of one problem; each wave
//    holds NSUB 32-row blocks of its row keys as MFMA B operands in registers for the whole
//    sweep (d <= 128 makes this a short-K contraction).
//  * Column keys stream through LDS in tiles of TN = 32 * CPT columns, double buffered, from
//    the contiguous copy in partitioned order [S0 | evicted] (K1b, K1c), so every 32-column
//    chunk belongs to exactly one of the two reductions and tile loads are plain streams.
//  * v_mfma_f32_32x32x16_bf16 with A = 32 column keys, B = 32 row keys gives each lane one
//    row i (lane % 32) and 16 columns: register v holds column 8*(v/4) + 4*(lane/32) + v%4.
//  * Row keys are pre-scaled by an exact power of two g_i so that ||g_i k_i|| is in (0.5, 1];
//    x = dot * r_j + 3 then lies in [2, 4), where the fp32 bit pattern is monotone and the
//    low 4 mantissa bits can carry the register slot: one v_max_u32 reduces value and
//    argmax together (quantum 2^-18 of the scaled similarity, far below the 1e-3 tolerance).
//    The chunk index of a lane's running maximum is kept beside it.
//  * Products of bf16 values are exact in fp32; accumulation is fp32.  fp32 keys use the
//    split k = hi + lo (bf16 each) and the three products hi.hi + lo.hi + hi.lo, laid out
//    as a contraction over 3d.
//  * Pairs inside the window and padding columns only occur in a few chunks per wave, found
//    by scalar range tests; those take a masked epilogue, all others a 2.5-instruction-per-
//    element epilogue (v_fmaak, v_and_or, half a v_max3).
#include <hip/hip_runtime.h>

#include <type_traits>

#include "../twinkv_internal.h"

namespace twinkv {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

template <int D, bool SPLIT, int NSUB, int NWAVES, int CPT>
struct Cfg {
  static constexpr int KSTEPS = SPLIT ? 3 * D / 16 : D / 16;
  static constexpr int DCOL = SPLIT ? 2 * D : D;      // bf16 elements per column in LDS
  static constexpr int PPC = DCOL / 8;                // 16-byte pieces per column
  static constexpr int SWZ = (PPC < 16 ? PPC : 16) - 1;  // piece-index XOR swizzle mask
  static constexpr int TN = CPT * kChunk;             // columns per LDS tile
  static constexpr int NT = NWAVES * 64;
  static constexpr int RB = NWAVES * NSUB * 32;       // rows per workgroup
  static constexpr int KEY_BYTES = TN * DCOL * 2;
  static constexpr int STAGE = KEY_BYTES + TN * 8;    // keys + inverse norms + positions
  static constexpr int RETIRED = NWAVES * NSUB * 64 * 8;  // S0 results parked in LDS
  static constexpr int LOADS_PER_WAVE = TN * PPC / (NWAVES * 64);  // 1-KB direct loads
  static constexpr int VALU_PER_MFMA = (52 + KSTEPS - 1) / KSTEPS;
  static_assert((TN * PPC) % (NWAVES * 64) == 0, "tile copy must divide evenly");
  static_assert(TN <= NT, "one thread per tile column for the column tables");
};

// Element offset of k-step t inside a column (A operand) / a row (B operand).
// bf16 keys: plain. fp32 keys: columns hold [hi | lo], rows hold [hi | lo]; the three
// k-step groups pair (col hi, row hi), (col lo, row hi), (col hi, row lo).
template <int D, bool SPLIT>
__device__ constexpr int col_off(int t) {
  if constexpr (!SPLIT) {
    return t * 16;
  } else {
    constexpr int G = D / 16;
    return t < G ? t * 16 : (t < 2 * G ? D + (t - G) * 16 : (t - 2 * G) * 16);
  }
}
template <int D, bool SPLIT>
__device__ constexpr int row_off(int t) {
  if constexpr (!SPLIT) {
    return t * 16;
  } else {
    constexpr int G = D / 16;
    return t < G ? t * 16 : (t < 2 * G ? (t - G) * 16 : D + (t - 2 * G) * 16);
  }
}

// Power of two g with ||g k|| in (0.5, 1] given r = 1/||k|| (1 for zero or bad keys).
__device__ inline float row_scale(float r) {
  if (!(r > 0.0f) || !(r < 3.0e38f)) return 1.0f;
  int e;
  (void)frexpf(r, &e);
  return ldexpf(1.0f, e - 1);
}

// Multiply 8 bf16 values by a power of two.  Exact unless a value leaves the normal range.
__device__ inline bf16x8 scale8(uint4 raw, float g) {
  uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
  uint32_t o[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const float lo = __uint_as_float(w[k] << 16) * g;
    const float hi = __uint_as_float(w[k] & 0xFFFF0000u) * g;
    o[k] = (__float_as_uint(lo) >> 16) | (__float_as_uint(hi) & 0xFFFF0000u);
  }
  uint4 r = make_uint4(o[0], o[1], o[2], o[3]);
  return __builtin_bit_cast(bf16x8, r);
}

// Column (0..31 inside a chunk) held by register v of a lane in half `half`.
__device__ inline int slot_col(int v, int half) { return 8 * (v >> 2) + 4 * half + (v & 3); }

constexpr uint32_t kValidMin = 0x3F800000u;  // packed values >= 1.0f are real candidates

// Scheduling-group masks for __builtin_amdgcn_sched_group_barrier.
constexpr int kSchedValu = 0x002;
constexpr int kSchedMfma = 0x008;
constexpr int kSchedDsRead = 0x100;

// Value + slot of the best column of one lane's 16 accumulators (unmasked chunk).
__device__ inline uint32_t chunk_best(const f32x16& acc, const float (&rv)[16]) {
  uint32_t b = 0u;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const float x = fmaf(acc[v], rv[v], 3.0f);
    b = max(b, (__float_as_uint(x) & 0xFFFFFFF0u) | (uint32_t)(15 - v));
  }
  return b;
}

// Branch-free running update: a strictly larger value (slot bits ignored) replaces the
// running best, so an earlier chunk keeps exact ties.
__device__ inline void run_update(uint32_t best, int gc, uint32_t& run, int& cid) {
  const bool upd = (best >> 4) > (run >> 4);
  run = upd ? best : run;
  cid = upd ? gc : cid;
}

template <int D, bool SPLIT, int NSUB, int NWAVES, int CPT>
__global__ __launch_bounds__(NWAVES * 64, 2) void sim_reduce_kernel(SimArgs a) {
  using C = Cfg<D, SPLIT, NSUB, NWAVES, CPT>;
  __shared__ __attribute__((aligned(1024))) char smem[2 * C::STAGE + C::RETIRED];

  // ---- which (head, sequence, row block) this workgroup owns --------------------------
  // With >= 8 heads, heads h = x (mod 8) go to the XCD x the hardware dispatches block
  // b = x (mod 8) to, so one problem's row blocks share that XCD's L2; inside an XCD the
  // sequences run longest first.
  int k, hx, h0, hstep;
  if (a.n_heads >= 8) {
    const int x = blockIdx.x & 7;
    k = blockIdx.x >> 3;
    hx = (a.n_heads - x + 7) >> 3;
    h0 = x;
    hstep = 8;
  } else {
    k = blockIdx.x;
    hx = a.n_heads;
    h0 = 0;
    hstep = 1;
  }
  if (k >= hx * a.total_tiles) return;
  int lo = 0, hi = a.n_seqs - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (hx * a.seqtab[mid].tile_cum <= k) lo = mid; else hi = mid - 1;
  }
  const int nb = a.seqtab[lo].nb;
  const int local = k - hx * a.seqtab[lo].tile_cum;
  const int head = h0 + hstep * (local / nb);
  const int rb = local - (local / nb) * nb;
  const int seq = a.seqtab[lo].sorted_seq;
  const SeqInfo si = a.seqtab[seq];
  const int q = head * a.n_seqs + seq;
  const ProblemMeta pm = a.pmeta[q];
  const int len = si.len;
  const int nchunks = a.want_all ? pm.total_chunks : pm.ret_chunks;
  const int ncols = nchunks * kChunk;
  const int ntiles = (nchunks + CPT - 1) / CPT;

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  uint2* retired = reinterpret_cast<uint2*>(smem + 2 * C::STAGE) + wave * NSUB * 64;
  const int lane = threadIdx.x & 63;
  const int half = lane >> 5;
  const int l32 = lane & 31;
  const int wrow0 = rb * C::RB + wave * NSUB * 32;

  const int64_t colbase = (int64_t)head * a.PT + si.perm_off;
  const uint16_t* kb = (const uint16_t*)a.keys + (int64_t)head * a.head_stride +
                       (int64_t)si.start * a.token_stride;
  const uint16_t* pk = a.pkeys + colbase * C::DCOL;
  const int32_t* pc = a.pcol + colbase;
  const float* rc = a.rcol + colbase;
  const float* rinv = a.rinv + (int64_t)head * a.T + si.start;

  // ---- chunks that need the masked epilogue: the window band of this wave's rows and the
  // padding at the end of each group.  In the [S0 | evicted] order the columns j with
  // x0 <= j < x1 occupy one contiguous range per group, read off the S0 prefix counts.
  int cr_lo, cr_hi, ce_lo, ce_hi, pad_r, pad_e;
  {
    const int32_t* prk = a.prank + colbase;
    const int x0 = min(max(wrow0 - a.w, 0), len);
    const int x1 = min(max(wrow0 + NSUB * 32 + a.w, 0), len);
    const int r0 = prk[x0], r1 = prk[x1];
    const int ret_pad = pm.ret_chunks * kChunk;
    const int e0 = ret_pad + (x0 - r0), e1 = ret_pad + (x1 - r1);
    cr_lo = r0 < r1 ? r0 / kChunk : 1;
    cr_hi = r0 < r1 ? (r1 - 1) / kChunk : 0;
    ce_lo = e0 < e1 ? e0 / kChunk : 1;
    ce_hi = e0 < e1 ? (e1 - 1) / kChunk : 0;
    const int n_ev = len - pm.n_ret;
    pad_r = (pm.n_ret % kChunk) ? pm.n_ret / kChunk : -1;
    pad_e = (n_ev % kChunk) ? (ret_pad + n_ev) / kChunk : -1;
    cr_lo = __builtin_amdgcn_readfirstlane(cr_lo);
    cr_hi = __builtin_amdgcn_readfirstlane(cr_hi);
    ce_lo = __builtin_amdgcn_readfirstlane(ce_lo);
    ce_hi = __builtin_amdgcn_readfirstlane(ce_hi);
    pad_r = __builtin_amdgcn_readfirstlane(pad_r);
    pad_e = __builtin_amdgcn_readfirstlane(pad_e);
  }

  // ---- row keys: MFMA B operands, resident for the whole sweep ------------------------
  bf16x8 bfrag[NSUB][C::KSTEPS];
#pragma unroll
  for (int s = 0; s < NSUB; ++s) {
    const int i = wrow0 + s * 32 + l32;
    const bool ok = i < len;
    const float g = row_scale(ok ? rinv[i] : 0.0f);
#pragma unroll
    for (int t = 0; t < C::KSTEPS; ++t) {
      uint4 raw = make_uint4(0, 0, 0, 0);
      if (ok) raw = *reinterpret_cast<const uint4*>(kb + (int64_t)i * a.token_stride +
                                                     row_off<D, SPLIT>(t) + half * 8);
      bfrag[s][t] = scale8(raw, g);
      // Row keys are only ever MFMA operands: keep them in accumulation registers so the
      // architectural VGPRs stay free for the epilogue (MFMA reads srcB from AGPRs).
      asm volatile("" : "+a"(bfrag[s][t]));
    }
  }

  // One running maximum per row block: S0 columns are swept first, and their results are
  // parked in LDS (``retire``) when the sweep reaches the evicted columns.
  uint32_t run[NSUB];
  int cid[NSUB];
#pragma unroll
  for (int s = 0; s < NSUB; ++s) {
    run[s] = 0u;
    cid[s] = 0;
  }
  bool retired_done = false;
  auto retire = [&]() {
#pragma unroll
    for (int s = 0; s < NSUB; ++s) {
      retired[s * 64 + lane] = make_uint2(run[s], (uint32_t)cid[s]);
      run[s] = 0u;
      cid[s] = 0;
    }
    retired_done = true;
  };

  // ---- column tiles: global -> LDS by direct (asynchronous) loads, double buffered ------
  // Each wave moves LOADS_PER_WAVE blocks of 1 KB; lane l of a block lands at byte 16*l.
  // A column's 16-byte piece p is stored in slot p ^ (column & SWZ) of its row, so the
  // 32 lanes that read one piece of 32 consecutive columns hit distinct banks.
  int nxt_p = -1;
  float nxt_r = 0.0f;
  auto issue_tile = [&](int tile, int buf) {
    char* st = smem + buf * C::STAGE;
#pragma unroll
    for (int kk = 0; kk < C::LOADS_PER_WAVE; ++kk) {
      const int blk = wave * C::LOADS_PER_WAVE + kk;
      const int e = blk * 64 + lane;
      const int col = e / C::PPC;
      const int slot = e - col * C::PPC;
      const int part = slot ^ (col & C::SWZ);
      int gcol = tile * C::TN + col;
      gcol = gcol < ncols ? gcol : 0;            // beyond the last chunk: any valid column
      __builtin_amdgcn_global_load_lds(
          (const void*)(pk + (int64_t)gcol * C::DCOL + part * 8),
          (void __attribute__((address_space(3)))*)(st + blk * 1024), 16, 0, 0);
    }
    if (threadIdx.x < C::TN) {
      const int col = tile * C::TN + threadIdx.x;
      nxt_p = col < ncols ? pc[col] : -1;
      nxt_r = col < ncols ? rc[col] : 0.0f;
    }
  };
  auto finish_tile = [&](int buf) {  // column tables of the issued tile, then wait for all
    char* st = smem + buf * C::STAGE;
    if (threadIdx.x < C::TN) {
      reinterpret_cast<float*>(st + C::KEY_BYTES)[threadIdx.x] = nxt_r;
      reinterpret_cast<int*>(st + C::KEY_BYTES + C::TN * 4)[threadIdx.x] = nxt_p;
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  };

  if (ntiles > 0) {
    issue_tile(0, 0);
    finish_tile(0);
  }
  __syncthreads();

  for (int tile = 0; tile < ntiles; ++tile) {
    if (tile + 1 < ntiles) issue_tile(tile + 1, (tile + 1) & 1);
    const char* st = smem + (tile & 1) * C::STAGE;
    const uint16_t* lk = reinterpret_cast<const uint16_t*>(st);
    const float* lr = reinterpret_cast<const float*>(st + C::KEY_BYTES);
    const int* lp = reinterpret_cast<const int*>(st + C::KEY_BYTES + C::TN * 4);

    // One 32-column chunk: the MFMA chain of 32-row block s runs while the VALU reduces
    // block s - 1.  RET picks the running maximum, MASKED applies the window / padding test.
    auto chunk = [&](int c, int gc, auto mask_tag) {
      constexpr bool MASKED = decltype(mask_tag)::value;
      const int col = c * kChunk + l32;
      bf16x8 af[C::KSTEPS];
#pragma unroll
      for (int t = 0; t < C::KSTEPS; ++t) {
        const int part = (col_off<D, SPLIT>(t) >> 3) + half;
        af[t] = *reinterpret_cast<const bf16x8*>(lk + col * C::DCOL + ((part ^ (col & C::SWZ)) << 3));
      }
      float rv[16];
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const float4 x = *reinterpret_cast<const float4*>(lr + c * kChunk + 8 * g4 + 4 * half);
        rv[4 * g4 + 0] = x.x;
        rv[4 * g4 + 1] = x.y;
        rv[4 * g4 + 2] = x.z;
        rv[4 * g4 + 3] = x.w;
      }
      auto reduce = [&](const f32x16& acc, int s) {
        uint32_t best;
        if constexpr (MASKED) {
          // column positions read here (rare path) so they are not live across the chunk
          const int i = wrow0 + s * 32 + l32;
          best = 0u;
#pragma unroll
          for (int g4 = 0; g4 < 4; ++g4) {
            const int4 jq = *reinterpret_cast<const int4*>(lp + c * kChunk + 8 * g4 + 4 * half);
            const int jv[4] = {jq.x, jq.y, jq.z, jq.w};
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const int v = 4 * g4 + q;
              const float y = fmaf(acc[v], rv[v], 3.0f);
              const uint32_t u = (__float_as_uint(y) & 0xFFFFFFF0u) | (uint32_t)(15 - v);
              const bool ok = (jv[q] >= 0) && (abs(i - jv[q]) > a.w);
              best = max(best, ok ? u : 0u);
            }
          }
        } else {
          best = chunk_best(acc, rv);
        }
        run_update(best, gc, run[s], cid[s]);
      };
      f32x16 prev;
#pragma unroll
      for (int s = 0; s < NSUB; ++s) {
        f32x16 x = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int t = 0; t < C::KSTEPS; ++t)
          x = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[t], bfrag[s][t], x, 0, 0, 0);
        if (s > 0) reduce(prev, s - 1);
        prev = x;
        if (s > 0) {
#pragma unroll
          for (int i = 0; i < C::KSTEPS; ++i) {
            __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 0);
            __builtin_amdgcn_sched_group_barrier(kSchedValu, C::VALU_PER_MFMA, 0);
          }
        }
      }
      reduce(prev, NSUB - 1);
    };

#pragma unroll 1
    for (int c = 0; c < CPT; ++c) {
      const int gc = tile * CPT + c;
      if (gc >= nchunks) break;
      if (gc == pm.ret_chunks) retire();
      const bool masked = (gc >= cr_lo && gc <= cr_hi) || (gc >= ce_lo && gc <= ce_hi) ||
                          gc == pad_r || gc == pad_e;
      if (!masked) chunk(c, gc, std::false_type{});
      else chunk(c, gc, std::true_type{});
    }
    if (tile + 1 < ntiles) finish_tile((tile + 1) & 1);
    __syncthreads();
  }

  if (!retired_done) retire();          // no evicted columns were swept

  // ---- resolve: lanes l and l+32 hold the same row over disjoint column halves ----------
#pragma unroll
  for (int s = 0; s < NSUB; ++s) {
    const int i = wrow0 + s * 32 + l32;
    const float ri = (i < len) ? rinv[i] : 0.0f;
    const float g = row_scale(ri);
    uint32_t val[2];
    int pos[2];
    const uint2 rr = retired[s * 64 + lane];
    const uint32_t runs[2] = {rr.x, run[s]};
    const int cids[2] = {(int)rr.y, cid[s]};
#pragma unroll
    for (int grp = 0; grp < 2; ++grp) {
      uint32_t v = runs[grp] & 0xFFFFFFF0u;
      int p = cids[grp] * kChunk + slot_col(15 - (int)(runs[grp] & 15u), half);
      const uint32_t v2 = __shfl_xor(v, 32);
      const int p2 = __shfl_xor(p, 32);
      if (v2 > v || (v2 == v && p2 < p)) { v = v2; p = p2; }
      val[grp] = v;
      pos[grp] = p;
    }
    if (half == 0 && i < len) {
      const int64_t o = (int64_t)head * a.T + si.start + i;
      const bool vr = val[0] >= kValidMin;
      const bool ve = val[1] >= kValidMin;
      const int jr = vr ? pc[pos[0]] : -1;
      const int je = ve ? pc[pos[1]] : -1;
      const float sr = vr ? (__uint_as_float(val[0]) - 3.0f) * ri / g : -1.0f;
      const float se = ve ? (__uint_as_float(val[1]) - 3.0f) * ri / g : -1.0f;
      if (a.best_ret) a.best_ret[o] = sr;
      if (a.arg_ret) a.arg_ret[o] = jr;
      if (a.best_all || a.arg_all) {
        bool take_r;
        if (!vr) take_r = false;
        else if (!ve) take_r = true;
        else take_r = (val[0] > val[1]) || (val[0] == val[1] && jr < je);
        const bool any = vr || ve;
        if (a.best_all) a.best_all[o] = any ? (take_r ? sr : se) : -1.0f;
        if (a.arg_all) a.arg_all[o] = any ? (take_r ? jr : je) : -1;
      }
    }
  }
}

template <int D, bool SPLIT, int NSUB, int NWAVES, int CPT>
hipError_t run(const SimArgs& a, hipStream_t st) {
  using C = Cfg<D, SPLIT, NSUB, NWAVES, CPT>;
  const int64_t groups = a.n_heads >= 8 ? 8LL * ((a.n_heads + 7) / 8) : (int64_t)a.n_heads;
  const int64_t blocks = groups * a.total_tiles;
  if (blocks == 0) return hipSuccess;
  hipLaunchKernelGGL((sim_reduce_kernel<D, SPLIT, NSUB, NWAVES, CPT>), dim3((unsigned)blocks),
                     dim3(C::NT), 0, st, a);
  return hipGetLastError();
}

}  // namespace

// Tile shapes: (NSUB 32-row blocks per wave, waves per workgroup, 32-column chunks per tile).
#define TWINKV_CFG_BF16_128 128, false, 3, 4, 4
#define TWINKV_CFG_BF16_64 64, false, 4, 4, 4
#define TWINKV_CFG_F32_64 64, true, 2, 4, 4
#define TWINKV_CFG_F32_128 128, true, 1, 4, 2

int sim_rows_per_block(int dtype, int d) {
  if (dtype == 0 && d == 128) return Cfg<TWINKV_CFG_BF16_128>::RB;
  if (dtype == 0 && d == 64) return Cfg<TWINKV_CFG_BF16_64>::RB;
  if (dtype == 1 && d == 64) return Cfg<TWINKV_CFG_F32_64>::RB;
  if (dtype == 1 && d == 128) return Cfg<TWINKV_CFG_F32_128>::RB;
  return 0;
}

int launch_sim_reduce(const SimArgs& a, int dtype, int d, void* stream) {
  hipStream_t st = (hipStream_t)stream;
  if (dtype == 0 && d == 128) return run<TWINKV_CFG_BF16_128>(a, st);
  if (dtype == 0 && d == 64) return run<TWINKV_CFG_BF16_64>(a, st);
  if (dtype == 1 && d == 64) return run<TWINKV_CFG_F32_64>(a, st);
  if (dtype == 1 && d == 128) return run<TWINKV_CFG_F32_128>(a, st);
  return hipErrorInvalidValue;
}

}  // namespace twinkv
