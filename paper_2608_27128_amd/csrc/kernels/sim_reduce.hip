// K2: fused cosine-similarity contraction with two masked row max / argmax reductions.
//
// For every problem (head, sequence) and token i it computes, without materialising the
// N x N matrix (Sec. 3.2 Eq. 1 and the twin window; Sec. 3.4 Eq. 4):
//   best over all j with |i-j| > w of sim(i, j)        -> best_all / arg_all
//   best over j in S0 with |i-j| > w of sim(i, j)      -> best_ret / arg_ret  (= b_i(S0))
// with sim(i, j) = (k_i . k_j) * r_i * r_j, r = 1 / ||k||.  In count mode (Sec. 3.2 Eq. 2)
// the same sweep instead counts, per token, the j with |i-j| > w and sim(i, j) > tau.
//
// Mapping onto gfx950:
//  * One workgroup owns RB = NWAVES * NSUB * 32 consecutive rows of one problem; each wave
//    holds NSUB 32-row blocks of its row keys as MFMA B operands in registers for the whole
//    sweep (d <= 128 makes this a short-K contraction).
//  * Column keys stream through LDS in tiles of TN = 32 * CPT columns, double buffered, from
//    the contiguous copy in partitioned order [S0 | evicted] written by the key preparation,
//    so every 32-column chunk belongs to exactly one of the two reductions and tile loads
//    are plain streams.
//  * v_mfma_f32_32x32x16_bf16 with A = 32 column keys, B = 32 row keys gives each lane one
//    row i (lane % 32) and 16 columns: register v holds column 8*(v/4) + 4*(lane/32) + v%4.
//  * Row keys are pre-scaled by an exact power of two g_i so that ||g_i k_i|| is in (0.5, 1];
//    x = dot * r_j + 3 then lies in [2, 4), where the fp32 bit pattern is monotone and the
//    low mantissa bits can carry a column code: one v_max_u32 reduces value and argmax
//    together.  With a running update per chunk the code is the register slot (4 bits,
//    quantum 2^-18 of the scaled similarity); with one per tile of 4 chunks it also holds
//    the chunk's place in the tile (6 bits, quantum 2^-16), so the compare-and-select of the
//    running maximum runs once per tile instead of once per chunk.  Either quantum is far
//    below the 1e-3 tolerance.  The first chunk of the running maximum's chunk (or tile) is
//    kept beside it.
//  * Products of bf16 values are exact in fp32; accumulation is fp32.  fp32 keys use the
//    split k = hi + lo (bf16 each) and the three products hi.hi + lo.hi + hi.lo, laid out
//    as a contraction over 3d.
//  * Pairs inside the window and padding columns only occur in a few chunks per wave, found
//    by scalar range tests; the sweep drops their results and a masked pass redoes them at
//    the end (with the tile merge, per 32-row block, and the padding of a group's last
//    chunk holds copies of its last column, so that chunk is only redone when counting).
//    All other chunks take a 2.5-instruction-per-element epilogue (v_fmaak, v_and_or, half
//    a v_max3).
#include <hip/hip_runtime.h>

#include <type_traits>

#include "../twinkv_internal.h"

namespace twinkv {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

template <int D, bool SPLIT, int NSUB, int NWAVES, int CPT, int OCC, int FG>
struct Cfg {
  static_assert(FG == 1 || FG == CPT, "results merge per chunk or per tile");
  static constexpr int WG_PER_CU = OCC * 4 / NWAVES;  // OCC waves per SIMD
  // count mode's epilogue holds more registers: at most 2 waves per SIMD
  static constexpr int WG_PER_CU_COUNT = (OCC < 2 ? OCC : 2) * 4 / NWAVES;
  static constexpr int KSTEPS = SPLIT ? 3 * D / 16 : D / 16;
  static constexpr int DCOL = SPLIT ? 2 * D : D;      // bf16 elements per column in LDS
  static constexpr int PPC = DCOL / 8;                // 16-byte pieces per column
  static constexpr int SWZ = (PPC < 16 ? PPC : 16) - 1;  // piece-index XOR swizzle mask
  // columns sharing one 256-byte LDS bank row (2 at d = 64 bf16), and the period in
  // columns of the swizzle ((column / CPR) & SWZ)
  static constexpr int CPR = DCOL * 2 < 256 ? 256 / (DCOL * 2) : 1;
  static constexpr int SWZ_PERIOD = (SWZ + 1) * CPR;
  static_assert(kChunk % SWZ_PERIOD == 0, "a chunk's columns repeat the swizzle");
  static constexpr int TN = CPT * kChunk;             // columns per LDS tile
  static constexpr int NT = NWAVES * 64;
  static constexpr int RB = NWAVES * NSUB * 32;       // rows per workgroup
  static constexpr int CHUNK_BYTES = kChunk * DCOL * 2;  // keys of one 32-column chunk
  static constexpr int KEY_BYTES = TN * DCOL * 2;
  static constexpr int STAGE = KEY_BYTES + TN * 8;    // keys + inverse norms + positions
  static constexpr int RETIRED = NWAVES * NSUB * 64 * 8;  // S0 results parked in LDS
  static constexpr int LOADS_PER_WAVE = TN * PPC / (NWAVES * 64);  // 1-KB direct loads
  // VALU instructions the schedule places beside each MFMA: one chunk's epilogue (about 40
  // with the tile merge, 48 with a running update per chunk) over its KSTEPS MFMAs
  static constexpr int VALU_PER_MFMA = ((FG > 1 ? 40 : 48) + KSTEPS - 1) / KSTEPS;
  static_assert((TN * PPC) % (NWAVES * 64) == 0, "tile copy must divide evenly");
  static_assert(TN % 64 == 0, "the column tables move in 64-column (256-byte) pieces");
  static_assert(2 * (KEY_BYTES + TN * 8) + RETIRED <= 160 * 1024 / WG_PER_CU,
                "LDS of WG_PER_CU workgroups must fit one CU");
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

// Longest sequence whose row keys the similarity sweep reads from the partitioned column copy.
constexpr int kRowsFromCopyMaxLen = 8192;

// Fourth dword of a raw buffer resource on gfx9-family parts (32-bit data format).
constexpr int kBufferFlags = 0x00020000;

// BYTES (4 or 16) per lane from base + voff straight into LDS at lds + BYTES * lane, through
// a raw buffer resource of nbytes: lanes whose offset is past the end read nothing (zeros).
__device__ inline void load_block_lds16(const void* base, int nbytes, int voff, char* lds) {
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, nbytes, kBufferFlags);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (void __attribute__((address_space(3)))*)lds, 16,
                                           voff, 0, 0, 0);
}
__device__ inline void load_block_lds4(const void* base, int nbytes, int voff, char* lds) {
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, nbytes, kBufferFlags);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (void __attribute__((address_space(3)))*)lds, 4,
                                           voff, 0, 0, 0);
}

// Scheduling-group masks for __builtin_amdgcn_sched_group_barrier.
constexpr int kSchedValu = 0x002;
constexpr int kSchedMfma = 0x008;
constexpr int kSchedDsRead = 0x100;

// Low bits of a packed candidate when the chunks of a group of FG chunks are merged before
// the running update: register slot v (4 bits) and the chunk's place kc in the group,
// coded as LOW - (16 kc + v), so that among equal values the smaller column has the larger
// code.  FG = 1 leaves the plain slot code 15 - v.
template <int FG>
struct Slots {
  static_assert(FG == 1 || FG == 2 || FG == 4, "1, 2 or 4 chunks per group");
  static constexpr int BITS = 4 + (FG >= 2) + (FG >= 4);
  static constexpr uint32_t LOW = (1u << BITS) - 1u;
};

// Value + code of the best column of one lane's 16 accumulators of chunk kc of its group.
template <int FG>
__device__ inline uint32_t chunk_best(const f32x16& acc, const float (&rv)[16], int kc) {
  constexpr uint32_t LOW = Slots<FG>::LOW;
  uint32_t b = 0u;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const float x = fmaf(acc[v], rv[v], 3.0f);
    b = max(b, (__float_as_uint(x) & ~LOW) | (LOW - (uint32_t)(16 * kc + v)));
  }
  return b;
}

// Number of a lane's 16 similarities above the row's threshold (count mode, Eq. 2):
// y = dot * r_j + c_i with c_i = -tau * g_i / r_i is positive exactly when sim(i, j) > tau
// (a y of exactly +0, sim equal to tau up to fp32 rounding, counts as above).  Each sign
// bit is shifted into a mask with one v_alignbit (a serial chain the compiler cannot
// reassociate into a wide tree), and one v_bcnt counts them.
__device__ inline uint32_t chunk_count(const f32x16& acc, const float (&rv)[16], float c_row) {
  uint32_t neg = 0u;
#pragma unroll
  for (int v = 0; v < 16; ++v)
    neg = __builtin_amdgcn_alignbit(neg, __float_as_uint(fmaf(acc[v], rv[v], c_row)), 31);
  return 16u - (uint32_t)__builtin_popcount(neg);
}

// Branch-free running update: a strictly larger value (code bits ignored) replaces the
// running best, so an earlier chunk (group) keeps exact ties.  c: its first chunk.
template <int FG>
__device__ inline void run_update(uint32_t best, int c, uint32_t& run, int& cid) {
  constexpr int B = Slots<FG>::BITS;
  const bool upd = (best >> B) > (run >> B);
  run = upd ? best : run;
  cid = upd ? c : cid;
}

// A running best in the per-chunk form: value, slot code 15 - v, chunk index.
template <int FG>
__device__ inline void to_chunk_form(uint32_t& run, int& cid) {
  constexpr uint32_t LOW = Slots<FG>::LOW;
  const uint32_t q = LOW - (run & LOW);
  cid += (int)(q >> 4);
  run = (run & ~LOW) | (15u - (q & 15u));
}

template <int D, bool SPLIT, int NSUB, int NWAVES, int CPT, int OCC, int FG, bool COUNT>
__global__ __launch_bounds__(NWAVES * 64,
                             (COUNT ? Cfg<D, SPLIT, NSUB, NWAVES, CPT, OCC, FG>::WG_PER_CU_COUNT
                                    : Cfg<D, SPLIT, NSUB, NWAVES, CPT, OCC, FG>::WG_PER_CU))
void sim_reduce_kernel(SimArgs a) {
  using C = Cfg<D, SPLIT, NSUB, NWAVES, CPT, OCC, FG>;
  constexpr uint32_t LOW = Slots<FG>::LOW;
  static_assert(kGroupAlign % C::TN == 0, "the evicted group must start on a tile boundary");
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
  const int ret_chunks = pm.ret_chunks;                      // a multiple of CPT
  const int ret_real = (pm.n_ret + kChunk - 1) / kChunk;     // S0 chunks with a real column
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
  // partly padded last chunk of each group.  In the [S0 | evicted] order the columns j with
  // x0 <= j < x1 occupy one contiguous range per group, read off the S0 prefix counts.
  int cr_lo, cr_hi, ce_lo, ce_hi, pad_r, pad_e;
  {
    const int32_t* prk = a.prank + colbase;
    const int x0 = min(max(wrow0 - a.w, 0), len);
    const int x1 = min(max(wrow0 + NSUB * 32 + a.w, 0), len);
    const int r0 = prk[x0], r1 = prk[x1];
    const int ret_pad = ret_chunks * kChunk;
    const int e0 = ret_pad + (x0 - r0), e1 = ret_pad + (x1 - r1);
    cr_lo = r0 < r1 ? r0 / kChunk : 1;
    cr_hi = r0 < r1 ? (r1 - 1) / kChunk : 0;
    ce_lo = e0 < e1 ? e0 / kChunk : 1;
    ce_hi = e0 < e1 ? (e1 - 1) / kChunk : 0;
    const int n_ev = len - pm.n_ret;
    pad_r = (pm.n_ret % kChunk) ? pm.n_ret / kChunk : -1;
    pad_e = (n_ev % kChunk) ? (ret_pad + n_ev) / kChunk : -1;
    if constexpr (!COUNT && FG > 1) {
      // the key preparation fills a group's partial last chunk with copies of its last
      // column (exact ties), so the maximum needs no padding test there; counting does,
      // and the per-chunk configurations keep the test (it is still correct: the masked
      // pass skips the copies by their position -1)
      pad_r = -1;
      pad_e = -1;
    }
    cr_lo = __builtin_amdgcn_readfirstlane(cr_lo);
    cr_hi = __builtin_amdgcn_readfirstlane(cr_hi);
    ce_lo = __builtin_amdgcn_readfirstlane(ce_lo);
    ce_hi = __builtin_amdgcn_readfirstlane(ce_hi);
    pad_r = __builtin_amdgcn_readfirstlane(pad_r);
    pad_e = __builtin_amdgcn_readfirstlane(pad_e);
  }
  // With the tile merge, the band is also kept per 32-row block: a chunk is dropped and
  // redone only for the row blocks whose own band holds it (the sweep's chunk mask is one
  // scalar operand per chunk and row block either way).
  constexpr bool SUB_BANDS = FG > 1;
  int sr_lo[NSUB], sr_hi[NSUB], se_lo[NSUB], se_hi[NSUB];
  if constexpr (SUB_BANDS) {
    const int32_t* prk = a.prank + colbase;
    const int ret_pad = ret_chunks * kChunk;
#pragma unroll
    for (int s = 0; s < NSUB; ++s) {
      const int x0 = min(max(wrow0 + 32 * s - a.w, 0), len);
      const int x1 = min(max(wrow0 + 32 * s + 32 + a.w, 0), len);
      const int r0 = prk[x0], r1 = prk[x1];
      const int e0 = ret_pad + (x0 - r0), e1 = ret_pad + (x1 - r1);
      sr_lo[s] = __builtin_amdgcn_readfirstlane(r0 < r1 ? r0 / kChunk : 1);
      sr_hi[s] = __builtin_amdgcn_readfirstlane(r0 < r1 ? (r1 - 1) / kChunk : 0);
      se_lo[s] = __builtin_amdgcn_readfirstlane(e0 < e1 ? e0 / kChunk : 1);
      se_hi[s] = __builtin_amdgcn_readfirstlane(e0 < e1 ? (e1 - 1) / kChunk : 0);
    }
  }
  // Result bits of the CPT chunks of a tile in the main sweep (bit k: keep chunk c0 + k).
  // Dropped: chunks the masked pass redoes, the padding-only chunks that align the S0 group,
  // and chunks past the last one.  Branch-free scalar arithmetic, so the tile body stays
  // one straight-line block.
  auto keep_bits = [&](int c0) -> uint32_t {
    // most tiles drop nothing: one range test over the whole tile
    const int c1 = c0 + CPT - 1;
    const bool clean = (c1 < nchunks) && !(c1 >= ret_real && c0 < ret_chunks) &&
                       !(c1 >= cr_lo && c0 <= cr_hi) && !(c1 >= ce_lo && c0 <= ce_hi) &&
                       !(pad_r >= c0 && pad_r <= c1) && !(pad_e >= c0 && pad_e <= c1);
    if (clean) return SUB_BANDS ? (1u << (CPT * NSUB)) - 1u : (1u << CPT) - 1u;
    uint32_t bits = 0u;
    if constexpr (SUB_BANDS) {
#pragma unroll
      for (int kc = 0; kc < CPT; ++kc) {
        const int gc = c0 + kc;
        const int common = (int)(gc >= nchunks) |
                           ((int)(gc >= ret_real) & (int)(gc < ret_chunks)) |
                           (int)(gc == pad_r) | (int)(gc == pad_e);
#pragma unroll
        for (int sb = 0; sb < NSUB; ++sb) {
          const int drop = common | ((int)(gc >= sr_lo[sb]) & (int)(gc <= sr_hi[sb])) |
                           ((int)(gc >= se_lo[sb]) & (int)(gc <= se_hi[sb]));
          bits |= (uint32_t)(drop ^ 1) << (kc * NSUB + sb);
        }
      }
      return bits;
    }
#pragma unroll
    for (int kc = 0; kc < CPT; ++kc) {
      const int gc = c0 + kc;
      const int drop = (int)(gc >= nchunks) | ((int)(gc >= ret_real) & (int)(gc < ret_chunks)) |
                       ((int)(gc >= cr_lo) & (int)(gc <= cr_hi)) |
                       ((int)(gc >= ce_lo) & (int)(gc <= ce_hi)) | (int)(gc == pad_r) |
                       (int)(gc == pad_e);
      bits |= (uint32_t)(drop ^ 1) << kc;
    }
    return bits;
  };

  // ---- row keys: MFMA B operands, resident for the whole sweep ------------------------
  bf16x8 bfrag[NSUB][C::KSTEPS];
  // Count mode: sim(i, j) > tau  <=>  dot * r_j - tau * g_i / r_i > 0  (per row; a zero key
  // has similarity 0 to every key, so it counts every candidate exactly when tau < 0).
  float thr[NSUB];
  {
    // All of a wave's row loads are issued before any of them is used (one memory round
    // trip).  A row past the end of the sequence reads the last row instead: the results of
    // its lane are never written.
    // With every column copied (all-keys sweeps) and a short sequence, row i is read from its
    // own column in the partitioned copy, which the problem's other row blocks are streaming
    // through this XCD's L2, rather than from the key rows: the same bits, and no fresh lines
    // pushed into L2 (measured about 1% faster on 1k-4k-token sequences, 0.2-0.5% slower at
    // 16k-32k tokens, where the row keys are a small part of the traffic).
    float ri[NSUB];
    const uint16_t* src[NSUB];
    if (!COUNT && a.want_all && len <= kRowsFromCopyMaxLen) {
      const int32_t* prk = a.prank + colbase;
#pragma unroll
      for (int s = 0; s < NSUB; ++s) {
        const int i = min(wrow0 + s * 32 + l32, len - 1);
        const int r0 = prk[i], r1 = prk[i + 1];
        const int col = r1 > r0 ? r0 : ret_chunks * kChunk + (i - r0);
        src[s] = pk + (int64_t)col * C::DCOL;
      }
    } else {
#pragma unroll
      for (int s = 0; s < NSUB; ++s) {
        const int i = min(wrow0 + s * 32 + l32, len - 1);
        src[s] = kb + (int64_t)i * a.token_stride;
      }
    }
#pragma unroll
    for (int s = 0; s < NSUB; ++s) {
      const int i = min(wrow0 + s * 32 + l32, len - 1);
      ri[s] = rinv[i];
#pragma unroll
      for (int t = 0; t < C::KSTEPS; ++t)
        bfrag[s][t] = *reinterpret_cast<const bf16x8*>(src[s] + row_off<D, SPLIT>(t) + half * 8);
    }
#pragma unroll
    for (int s = 0; s < NSUB; ++s) {
      const float g = row_scale(ri[s]);
      thr[s] = ri[s] > 0.0f ? -a.tau * g / ri[s] : (a.tau < 0.0f ? INFINITY : -INFINITY);
#pragma unroll
      for (int t = 0; t < C::KSTEPS; ++t)
        bfrag[s][t] = scale8(__builtin_bit_cast(uint4, bfrag[s][t]), g);
    }
  }

  // One running maximum per row block: S0 columns are swept first, and their results are
  // parked in LDS (``retire``) when the sweep reaches the evicted columns.
  // tb: with FG = CPT, the best of the current tile's chunks so far.
  uint32_t run[NSUB], tb[NSUB];
  int cid[NSUB];
#pragma unroll
  for (int s = 0; s < NSUB; ++s) {
    run[s] = 0u;
    tb[s] = 0u;
    cid[s] = 0;
  }
  bool retired_done = false;
  auto retire = [&]() {
#pragma unroll
    for (int s = 0; s < NSUB; ++s) {
      if constexpr (!COUNT) to_chunk_form<FG>(run[s], cid[s]);
      retired[s * 64 + lane] = make_uint2(run[s], (uint32_t)cid[s]);
      run[s] = 0u;
      cid[s] = 0;
    }
    retired_done = true;
  };

  // ---- LDS addressing ------------------------------------------------------------------
  // A column's 16-byte piece p is stored in slot p ^ ((column / CPR) & SWZ) of its row, so
  // the lanes that read one piece of consecutive columns in one LDS pass hit distinct banks
  // (with two 128-byte columns per 256-byte bank row at d = 64, the even and the odd columns
  // take the two halves of the row and the swizzle changes every second column).  The
  // swizzle repeats every SWZ_PERIOD columns, which divides 32, so for column c*32 + l32 it
  // only depends on l32: the byte offset of k-step t of a lane's column is a lane constant
  // plus c * (chunk bytes) plus the stage offset.
  int aoff[C::KSTEPS];
#pragma unroll
  for (int t = 0; t < C::KSTEPS; ++t) {
    const int part = (col_off<D, SPLIT>(t) >> 3) + half;
    aoff[t] = l32 * (C::DCOL * 2) + ((part ^ ((l32 / C::CPR) & C::SWZ)) << 4);
  }
  const int roff = C::KEY_BYTES + 16 * half;  // this lane's inverse norms inside a chunk

  auto load_rv = [&](const char* st, int c, float (&rv)[16]) {
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      const float4 x = *reinterpret_cast<const float4*>(st + roff + c * kChunk * 4 + 32 * g4);
      rv[4 * g4 + 0] = x.x;
      rv[4 * g4 + 1] = x.y;
      rv[4 * g4 + 2] = x.z;
      rv[4 * g4 + 3] = x.w;
    }
  };

  // ---- column tiles: global -> LDS by direct (asynchronous) loads, double buffered ------
  // Each wave moves LOADS_PER_WAVE blocks of 1 KB with buffer loads; lane l of a block lands
  // at byte 16*l.  Block blk holds columns blk*B .. blk*B+B-1 (B = 64 / PPC), lane l piece
  // l % PPC of column blk*B + l / PPC, stored in slot piece ^ ((column / CPR) & SWZ).  The
  // buffer resource of a tile ends at the problem's last column, so the hardware range check
  // turns loads past it into zeros instead of reads (those columns are never used).
  constexpr int B = 64 / C::PPC;
  constexpr int NV = C::SWZ_PERIOD / B;  // distinct lane offsets over a wave's blocks
  static_assert(C::SWZ_PERIOD % B == 0 && ((C::LOADS_PER_WAVE * B) % C::SWZ_PERIOD) == 0,
                "the swizzle of a block's columns must repeat with the block index");
  const int lcol = lane / C::PPC;
  int vlane[NV];
#pragma unroll
  for (int r = 0; r < NV; ++r)
    vlane[r] = lcol * (C::DCOL * 2) + 16 * ((lane % C::PPC) ^ (((r * B + lcol) / C::CPR) & C::SWZ));
  auto issue_tile = [&](int tile, int buf) {
    char* st = smem + buf * C::STAGE;
    const int64_t first = (int64_t)tile * C::TN;
    const int left = ncols - (int)first;                // > 0 for every issued tile
    const int nbytes = (left < C::TN ? left : C::TN) * C::DCOL * 2;
#pragma unroll
    for (int kk = 0; kk < C::LOADS_PER_WAVE; ++kk) {
      // one resource per 1-KB block, based at the block: the range check sees the whole
      // offset of every lane
      const int blk = wave * C::LOADS_PER_WAVE + kk;
      const int rem = nbytes - blk * 1024;
      load_block_lds16(pk + (first * C::DCOL + blk * 512), rem > 0 ? rem : 0,
                       vlane[kk % NV], st + blk * 1024);
    }
    // The column tables (inverse norms, then positions) in 256-byte pieces, 4 bytes a lane.
    const int tbytes = (left < C::TN ? left : C::TN) * 4;
#pragma unroll
    for (int pc4 = wave; pc4 < C::TN / 32; pc4 += NWAVES) {
      const int part = pc4 % (C::TN / 64);
      const int rem = tbytes - part * 256;
      const void* src = pc4 < C::TN / 64 ? (const void*)(rc + first + part * 64)
                                          : (const void*)(pc + first + part * 64);
      load_block_lds4(src, rem > 0 ? rem : 0, 4 * lane, st + C::KEY_BYTES + pc4 * 256);
    }
  };
  auto finish_tile = [&]() {  // wait for this wave's direct loads of the issued tile
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  };

  // ---- the pending reduction: the last 32-row block of the previous chunk is reduced
  // while the first MFMA chain of the next chunk runs (software pipelining across chunks).
  f32x16 pacc = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  float prv[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) prv[v] = 0.0f;
  int pgc = 0;
  uint32_t pmask = 0u;  // result mask of the pending chunk (zero: dropped)

  // Chunk gc (chunk kc of its tile) into row block s.  With FG = CPT the chunks of a tile
  // are merged in tb first and the tile enters the running best at ``flush``.
  auto reduce_into = [&](const f32x16& acc, const float (&rv)[16], int gc, int kc, int s,
                         uint32_t m) {
    if constexpr (COUNT) {
      run[s] += chunk_count(acc, rv, thr[s]) & m;
    } else if constexpr (FG == 1) {
      const uint32_t best = chunk_best<1>(acc, rv, 0) & m;
      run_update<1>(best, gc, run[s], cid[s]);
    } else {
      tb[s] = max(tb[s], chunk_best<FG>(acc, rv, kc) & m);
    }
  };
  auto flush = [&](int s, int c0) {
    if constexpr (!COUNT && FG > 1) {
      run_update<FG>(tb[s], c0, run[s], cid[s]);
      tb[s] = 0u;
    }
  };

  // One tile: each chain's epilogue runs beside the following chain's MFMAs, and the last
  // chain's epilogue is left pending for the next chunk.  During the last chain, k-step t of
  // the next chunk's A fragments is read into the registers that MFMA t has just consumed.
  auto sweep_tile = [&](auto buf_tag, int c0, uint32_t keep) {
    constexpr int BUF = decltype(buf_tag)::value;
    const char* st = smem + BUF * C::STAGE;
    bf16x8 fc[C::KSTEPS];
#pragma unroll
    for (int t = 0; t < C::KSTEPS; ++t)
      fc[t] = *reinterpret_cast<const bf16x8*>(st + aoff[t]);
#pragma unroll
    for (int kc = 0; kc < CPT; ++kc) {
      const int gc = c0 + kc;
      const uint32_t m = 0u - ((keep >> kc) & 1u);
      // with bands per row block, the result mask of row block sb for this chunk
      auto mask_of = [&](int sb) -> uint32_t {
        if constexpr (SUB_BANDS) return 0u - ((keep >> (kc * NSUB + sb)) & 1u);
        else return m;
      };
      float rcur[16];
      // with a single row block, chain 0 is also the last chain and carries the prefetch
      const bool pre0 = (NSUB == 1) && (kc + 1 < CPT);
      f32x16 x = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int t = 0; t < C::KSTEPS; ++t) {
        x = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fc[t], bfrag[0][t], x, 0, 0, 0);
        if (pre0)
          fc[t] = *reinterpret_cast<const bf16x8*>(st + (kc + 1) * C::CHUNK_BYTES + aoff[t]);
      }
      // the pending chunk: the previous chunk of this tile, or the last of the previous tile
      reduce_into(pacc, prv, pgc, kc == 0 ? CPT - 1 : kc - 1, NSUB - 1, pmask);
      if (kc == 0) flush(NSUB - 1, c0 - CPT);
      load_rv(st, kc, rcur);
#pragma unroll
      for (int i = 0; i < C::KSTEPS; ++i) {
        __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 0);
        if (i < 4 || pre0) __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 1, 0);
        __builtin_amdgcn_sched_group_barrier(kSchedValu, C::VALU_PER_MFMA, 0);
      }
#pragma unroll
      for (int s = 1; s < NSUB; ++s) {
        f32x16 y = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
        const bool pre = (s == NSUB - 1) && (kc + 1 < CPT);
#pragma unroll
        for (int t = 0; t < C::KSTEPS; ++t) {
          y = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fc[t], bfrag[s][t], y, 0, 0, 0);
          if (pre)
            fc[t] = *reinterpret_cast<const bf16x8*>(st + (kc + 1) * C::CHUNK_BYTES + aoff[t]);
        }
        reduce_into(x, rcur, gc, kc, s - 1, mask_of(s - 1));
        if (kc == CPT - 1) flush(s - 1, c0);
#pragma unroll
        for (int i = 0; i < C::KSTEPS; ++i) {
          __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 0);
          if (pre) __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 1, 0);
          __builtin_amdgcn_sched_group_barrier(kSchedValu, C::VALU_PER_MFMA, 0);
        }
        x = y;
      }
      pacc = x;
#pragma unroll
      for (int v = 0; v < 16; ++v) prv[v] = rcur[v];
      pgc = gc;
      pmask = mask_of(NSUB - 1);
    }
  };

  // A wave whose rows all lie past the end of the sequence (in the last row block of a
  // sequence) only takes its share of the tile loads; its SIMD's MFMA pipe is left to the
  // other workgroup's wave.
  const bool active = wrow0 < len;
#ifdef TWINKV_DEBUG
  // Debug build: both stages and the parked results start as poison.
  {
    uint4* all = reinterpret_cast<uint4*>(smem);
    for (int i = threadIdx.x; i < (2 * C::STAGE + C::RETIRED) / 16; i += C::NT)
      all[i] = make_uint4(~0u, ~0u, ~0u, ~0u);
  }
  __syncthreads();
#endif
  if (ntiles > 0) issue_tile(0, 0);
#pragma unroll 1
  for (int tile = 0; tile < ntiles; ++tile) {
    const int buf = tile & 1;
    finish_tile();
    __syncthreads();
    if (tile + 1 < ntiles) issue_tile(tile + 1, buf ^ 1);
    const int c0 = tile * CPT;
    if (c0 == ret_chunks) {
      // First evicted chunk: finish the pending S0 reduction here and park the S0 results.
      // The opaque copy keeps the compiler from moving the tile body's own pending
      // reduction out of the body to share it with this rare path.
      f32x16 pa = pacc;
      asm volatile("" : "+v"(pa));
      reduce_into(pa, prv, pgc, CPT - 1, NSUB - 1, pmask);
      flush(NSUB - 1, c0 - CPT);
      pmask = 0u;
      retire();
    }
    const uint32_t keep = __builtin_amdgcn_readfirstlane(keep_bits(c0));
    if (active) {
      if (buf == 0) sweep_tile(std::integral_constant<int, 0>{}, c0, keep);
      else sweep_tile(std::integral_constant<int, 1>{}, c0, keep);
    }
#ifdef TWINKV_DEBUG
    // Debug build: once every wave has swept this stage, fill it with 0xFF bytes (NaN keys
    // and inverse norms, position -1) before the next tile's loads refill it.  A read of a
    // stage outside its tile's lifetime then sees the poison, and the results differ from
    // the normal build's.
    __syncthreads();
    {
      uint4* stg = reinterpret_cast<uint4*>(smem + buf * C::STAGE);
      for (int i = threadIdx.x; i < C::STAGE / 16; i += C::NT)
        stg[i] = make_uint4(~0u, ~0u, ~0u, ~0u);
    }
    __syncthreads();
#endif
  }
  reduce_into(pacc, prv, pgc, CPT - 1, NSUB - 1, pmask);
  flush(NSUB - 1, (ntiles - 1) * CPT);
  if (!retired_done) retire();          // no evicted columns were swept
  if constexpr (!COUNT) {
#pragma unroll
    for (int s = 0; s < NSUB; ++s) to_chunk_form<FG>(run[s], cid[s]);
  }

  // ---- masked pass: the chunks holding window pairs or padding next to real columns, read
  // straight from the column copy, with the window / padding test per element.  Chunks are
  // visited out of order here, so equal values keep the smaller chunk index explicitly.
  //
  // Maximum with the tile merge: in each group the columns whose positions lie within w of a
  // lane's row form one contiguous range of column indices, read off the S0 prefix counts,
  // so the test per element is one unsigned range compare and the position list is not read.
  // The copies of a group's last column in its partly filled last chunk are excluded with
  // that column (and otherwise only tie with it).
  constexpr bool RANGE_TEST = !COUNT && FG > 1;
  // S0 prefix counts at the two ends of each row's window (loaded here, used once the first
  // chunks' loads are in flight)
  int wrx[NSUB], wry[NSUB];
  if constexpr (RANGE_TEST) {
    const int32_t* prk = a.prank + colbase;
#pragma unroll
    for (int s = 0; s < NSUB; ++s) {
      const int i = min(wrow0 + s * 32 + l32, len - 1);
      wrx[s] = prk[max(i - a.w, 0)];
      wry[s] = prk[min(i + a.w + 1, len)];
    }
  }
  // First excluded column and number of excluded columns of row block s's lane row in group
  // grp.
  auto excluded_range = [&](int grp, int s, int& lo, int& num) {
    // opaque copies: computed here, in each chunk's step, not hoisted ahead of the chunk loads
    int rx = wrx[s], ry = wry[s];
    asm volatile("" : "+v"(rx), "+v"(ry));
    const int i = min(wrow0 + s * 32 + l32, len - 1);
    const int x = max(i - a.w, 0), y = min(i + a.w + 1, len);
    const int ret_pad = ret_chunks * kChunk;
    if (grp == 0) {
      lo = rx;
      num = (ry == pm.n_ret ? ret_pad : ry) - lo;
    } else {
      lo = ret_pad + x - rx;
      const int e = ret_pad + y - ry;
      num = (e == ret_pad + (len - pm.n_ret) ? pm.total_chunks * kChunk : e) - lo;
    }
  };
  struct MaskedChunk {  // one chunk's A fragments and column tables, in registers (two
                        // chunks per memory round trip measured slower)
    bf16x8 af[C::KSTEPS];
    float rv[16];
    int jv[16];
  };
  auto masked_load = [&](int gc, MaskedChunk& mc) {
    const int col = gc * kChunk + l32;
#pragma unroll
    for (int t = 0; t < C::KSTEPS; ++t)
      mc.af[t] = *reinterpret_cast<const bf16x8*>(pk + (int64_t)col * C::DCOL +
                                                  col_off<D, SPLIT>(t) + 8 * half);
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int cc = gc * kChunk + slot_col(v, half);
      mc.rv[v] = rc[cc];
      mc.jv[v] = RANGE_TEST ? 0 : pc[cc];
    }
  };
  auto masked_compute = [&](int gc, int grp, const MaskedChunk& mc, uint32_t (&rs)[NSUB],
                            int (&cs)[NSUB]) {
    const bf16x8 (&af)[C::KSTEPS] = mc.af;
    const float (&rv)[16] = mc.rv;
    const int (&jv)[16] = mc.jv;
#pragma unroll
    for (int s = 0; s < NSUB; ++s) {
      if constexpr (SUB_BANDS) {
        // only the row blocks that dropped this chunk in the sweep
        const bool need = grp == 0 ? (gc == pad_r || (gc >= sr_lo[s] && gc <= sr_hi[s]))
                                   : (gc == pad_e || (gc >= se_lo[s] && gc <= se_hi[s]));
        if (!need) continue;
      }
      f32x16 x = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int t = 0; t < C::KSTEPS; ++t)
        x = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[t], bfrag[s][t], x, 0, 0, 0);
      const int i = wrow0 + s * 32 + l32;
      if constexpr (COUNT) {
        uint32_t c = 0u;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const uint32_t ok = (uint32_t)(jv[v] >= 0) & (uint32_t)(abs(i - jv[v]) > a.w);
          c += ok & ((~__float_as_uint(fmaf(x[v], rv[v], thr[s]))) >> 31);
        }
        rs[s] += c;
      } else {
        uint32_t best = 0u;
        // column of slot v, relative to the first excluded column of this row's range
        int xlo = 0, xnum = 0;
        if constexpr (RANGE_TEST) excluded_range(grp, s, xlo, xnum);
        const uint32_t rel = (uint32_t)(gc * kChunk + 4 * half - xlo);
        const uint32_t nex = (uint32_t)xnum;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const float y = fmaf(x[v], rv[v], 3.0f);
          const uint32_t u = (__float_as_uint(y) & ~LOW) | (uint32_t)(15 - v);
          bool ok;
          if constexpr (RANGE_TEST) ok = rel + (uint32_t)(8 * (v >> 2) + (v & 3)) >= nex;
          else ok = (jv[v] >= 0) & (abs(i - jv[v]) > a.w);
          best = max(best, ok ? u : 0u);
        }
        const bool upd = (best >> 4) > (rs[s] >> 4) ||
                         ((best >> 4) == (rs[s] >> 4) && best >= kValidMin && gc < cs[s]);
        rs[s] = upd ? best : rs[s];
        cs[s] = upd ? gc : cs[s];
      }
    }
  };
  auto masked_range = [&](int l, int h, int grp, uint32_t (&rs)[NSUB], int (&cs)[NSUB]) {
#pragma unroll 1
    for (int gc = l; gc <= h; ++gc) {
      if (gc < nchunks) {
        MaskedChunk mc;
        masked_load(gc, mc);
        masked_compute(gc, grp, mc, rs, cs);
      }
    }
  };
  // evicted group: the live registers
  if (active && a.want_all) {
    masked_range(ce_lo, ce_hi, 1, run, cid);
    if (pad_e >= 0 && !(pad_e >= ce_lo && pad_e <= ce_hi)) masked_range(pad_e, pad_e, 1, run, cid);
  }
  // S0 group: the parked results
  {
    uint32_t rr[NSUB];
    int rcid[NSUB];
#pragma unroll
    for (int s = 0; s < NSUB; ++s) {
      const uint2 v = retired[s * 64 + lane];
      rr[s] = v.x;
      rcid[s] = (int)v.y;
    }
    if (active) {
      masked_range(cr_lo, cr_hi, 0, rr, rcid);
      if (pad_r >= 0 && !(pad_r >= cr_lo && pad_r <= cr_hi)) masked_range(pad_r, pad_r, 0, rr, rcid);
    }
#pragma unroll
    for (int s = 0; s < NSUB; ++s) retired[s * 64 + lane] = make_uint2(rr[s], (uint32_t)rcid[s]);
  }

  // ---- resolve: lanes l and l+32 hold the same row over disjoint column halves ----------
  if constexpr (COUNT) {
    // the S0 group is empty in count mode: every column was swept as an evicted column
#pragma unroll
    for (int s = 0; s < NSUB; ++s) {
      const int i = wrow0 + s * 32 + l32;
      const uint32_t total = run[s] + __shfl_xor(run[s], 32);
      if (half == 0 && i < len) a.counts[(int64_t)head * a.T + si.start + i] = (int32_t)total;
    }
    return;
  }
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
      uint32_t v = runs[grp] & ~LOW;
      int p = cids[grp] * kChunk + slot_col(15 - (int)(runs[grp] & 15u), half);
      // a slot past the group's last column holds a copy of that column
      if constexpr (FG > 1)
        p = min(p, grp == 0 ? pm.n_ret - 1 : ret_chunks * kChunk + (len - pm.n_ret) - 1);
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

template <int D, bool SPLIT, int NSUB, int NWAVES, int CPT, int OCC, int FG>
hipError_t run(const SimArgs& a, hipStream_t st) {
  using C = Cfg<D, SPLIT, NSUB, NWAVES, CPT, OCC, FG>;
  const int64_t groups = a.n_heads >= 8 ? 8LL * ((a.n_heads + 7) / 8) : (int64_t)a.n_heads;
  const int64_t blocks = groups * a.total_tiles;
  if (blocks == 0) return hipSuccess;
  if (a.counts != nullptr)
    hipLaunchKernelGGL((sim_reduce_kernel<D, SPLIT, NSUB, NWAVES, CPT, OCC, FG, true>),
                       dim3((unsigned)blocks), dim3(C::NT), 0, st, a);
  else
    hipLaunchKernelGGL((sim_reduce_kernel<D, SPLIT, NSUB, NWAVES, CPT, OCC, FG, false>),
                       dim3((unsigned)blocks), dim3(C::NT), 0, st, a);
  return hipGetLastError();
}

}  // namespace

// Tile shapes: (d, fp32 split, NSUB 32-row blocks per wave, waves per workgroup, 32-column
// chunks per LDS tile, waves per SIMD, chunks merged before each running update: 1 or the
// chunks per tile).  Overridable at build time for tuning sweeps.
#ifndef TWINKV_CFG_BF16_128
#define TWINKV_CFG_BF16_128 128, false, 3, 4, 4, 2, 4
#endif
#ifndef TWINKV_CFG_BF16_64
#define TWINKV_CFG_BF16_64 64, false, 4, 4, 2, 3, 1
#endif
#ifndef TWINKV_CFG_F32_64
#define TWINKV_CFG_F32_64 64, true, 1, 4, 4, 2, 1
#endif
#ifndef TWINKV_CFG_F32_128
#define TWINKV_CFG_F32_128 128, true, 1, 4, 2, 2, 1
#endif

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
