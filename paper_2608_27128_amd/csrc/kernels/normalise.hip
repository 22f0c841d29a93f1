// K1a: per-problem stable partition of the positions into [S0 | evicted] column lists (the
//      S0 list padded to a multiple of kGroupAlign columns, the evicted list to whole
//      32-column chunks), from the retained mask alone.
// K1b: one pass over the keys: per-key inverse l2 norm (Sec. 3.2: k_hat = k / ||k||_2), and
//      the key itself copied to its slot of the partitioned column list (bf16; for fp32 keys
//      the bf16 hi/lo split the similarity kernel multiplies on bf16 MFMA, which also goes
//      to a row-ordered plane for the kernel's row operands).
//
// K1a reads 1 byte and writes 8 bytes per key.  K1b is an HBM stream: it reads d*esize bytes
// (+5 bytes of mask and rank) and writes d*2 (+4d for fp32) + 8 bytes per key.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "../twinkv_internal.h"

namespace twinkv {
namespace {

__device__ inline uint16_t bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ inline float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

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

// One workgroup of NT threads per (head, sequence) problem (1024 for long sequences).
template <int NT>
__global__ __launch_bounds__(NT) void partition_kernel(
    const uint8_t* __restrict__ retained, const SeqInfo* __restrict__ seqtab, int n_seqs,
    int64_t T, int64_t PT, int32_t* __restrict__ pcol, float* __restrict__ rcol,
    int32_t* __restrict__ prank, ProblemMeta* __restrict__ pmeta, int32_t* __restrict__ status) {
  __shared__ int s_red[NT / 64];
  __shared__ int s_wave[NT / 64];
  const int q = blockIdx.x;
  const int h = q / n_seqs;
  const int s = q - h * n_seqs;
  const SeqInfo si = seqtab[s];
  const int len = si.len;
  const uint8_t* ret = retained ? retained + h * T + si.start : nullptr;
  int32_t* pc = pcol + h * PT + si.perm_off;
  float* rc = rcol + h * PT + si.perm_off;
  int32_t* pr = prank + h * PT + si.perm_off;

  int cnt = 0;
  if (ret != nullptr)
    for (int t = threadIdx.x; t < len; t += NT) cnt += (ret[t] != 0);
  const int n_ret = block_sum<NT>(cnt, s_red);
  const int ret_pad = (n_ret + kGroupAlign - 1) / kGroupAlign * kGroupAlign;
  const int n_ev = len - n_ret;
  const int ev_pad = (n_ev + kChunk - 1) / kChunk * kChunk;

  const int lane = threadIdx.x & 63;
  const int wv = threadIdx.x >> 6;
  int ret_before_round = 0;
  for (int t0 = 0; t0 < len; t0 += NT) {
    const int t = t0 + threadIdx.x;
    const bool in = t < len;
    const bool r = in && ret != nullptr && ret[t] != 0;
    const unsigned long long bal = __ballot(r);
    const int pre = __popcll(bal & ((1ull << lane) - 1ull));
    if (lane == 0) s_wave[wv] = __popcll(bal);
    __syncthreads();
    int wbase = 0, tot = 0;
#pragma unroll
    for (int k = 0; k < NT / 64; ++k) {
      const int c = s_wave[k];
      wbase += (k < wv) ? c : 0;
      tot += c;
    }
    if (in) {
      const int ret_before = ret_before_round + wbase + pre;
      pc[r ? ret_before : ret_pad + (t - ret_before)] = t;
      pr[t] = ret_before;
    }
    ret_before_round += tot;
    __syncthreads();
  }
  // padding columns: no position, inverse norm 0 (their keys are never used)
  for (int k = n_ret + (int)threadIdx.x; k < ret_pad; k += NT) {
    pc[k] = -1;
    rc[k] = 0.0f;
  }
  for (int k = ret_pad + n_ev + (int)threadIdx.x; k < ret_pad + ev_pad; k += NT) {
    pc[k] = -1;
    rc[k] = 0.0f;
  }
  if (threadIdx.x == 0) {
    pr[len] = n_ret;
    ProblemMeta m;
    m.n_ret = n_ret;
    m.ret_chunks = ret_pad / kChunk;
    m.total_chunks = (ret_pad + ev_pad) / kChunk;
    m.flags = 0;
    pmeta[q] = m;
    if (status) status[q] = 0;
  }
}

// LPT lanes cooperate on one key; each lane owns 16 contiguous bytes of it.  A workgroup
// takes kPrepIter groups of TPB consecutive tokens of one (head, sequence) problem, all their
// loads issued before any is used.  blockIdx.y is the head; blockIdx.x runs over the
// workgroups of all sequences (seqtab[s].prep_blk0 = the first one of sequence s), so no
// workgroup is launched past the end of a short sequence.  Key reads and column-copy writes
// are nontemporal: each byte is touched once here, and the copy of a long or ragged batch is
// far larger than the caches (ragged batch of 64 sequences of 1k-4k tokens: this kernel
// 5.49 -> 5.14 ms; the reads alone nontemporal were slower).
constexpr int kPrepIter = 4;

typedef unsigned int prep_u32x4 __attribute__((ext_vector_type(4)));

// p moved by a byte offset (one level group's array from group 0's)
template <typename T>
__device__ inline T* byte_offset(T* p, int64_t bytes) {
  using C = typename std::conditional<std::is_const<T>::value, const char, char>::type;
  return reinterpret_cast<T*>(reinterpret_cast<C*>(p) + bytes);
}

__device__ inline uint4 prep_load16(const uint8_t* p) {
  const prep_u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const prep_u32x4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ inline void prep_store16(uint16_t* p, uint4 x) {
  const prep_u32x4 v = {x.x, x.y, x.z, x.w};
  __builtin_nontemporal_store(v, reinterpret_cast<prep_u32x4*>(p));
}

// LEVELS: the groups of nested retained sets in one pass (PrepLevels): each token goes to
// the column list of its own group, whose arrays lie group_stride bytes after the previous
// group's; rinv (and the fp32 row plane) is written once for all groups.  Without LEVELS,
// `retained` splits the positions into the one S0 list and the evicted list.
template <int D, bool F32, bool LEVELS>
__global__ __launch_bounds__(256) void prepare_keys_kernel(
    const uint8_t* __restrict__ keys, int64_t T, int64_t hs_bytes, int64_t ts_bytes, int64_t PT,
    const uint8_t* __restrict__ retained, const int32_t* __restrict__ prank,
    ProblemMeta* __restrict__ pmeta, const SeqInfo* __restrict__ seqtab, int n_seqs,
    float* __restrict__ rinv, float* __restrict__ rcol, uint16_t* __restrict__ hilo,
    uint16_t* __restrict__ pkeys, int32_t* __restrict__ status, int h0, int copy_evicted,
    PrepLevels lv) {
  constexpr int ESZ = F32 ? 4 : 2;
  constexpr int LPT = D * ESZ / 16;
  constexpr int TPB = 256 / LPT;
  constexpr int DCOL = F32 ? 2 * D : D;
  static_assert(LPT <= 64 && (64 % LPT) == 0, "a key must fit inside one wave");
  const int64_t h = h0 + (int64_t)blockIdx.y;
  const int bx = (int)blockIdx.x;
  int lo = 0, hi = n_seqs - 1;  // the last sequence whose first workgroup is <= bx
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (seqtab[mid].prep_blk0 <= bx) lo = mid; else hi = mid - 1;
  }
  const int s = lo;
  const int q = (int)h * n_seqs + s;
  const SeqInfo si = seqtab[s];
  const int sub = threadIdx.x % LPT;
  const int tfirst = (bx - si.prep_blk0) * (TPB * kPrepIter) + threadIdx.x / LPT;
  const int64_t base = h * PT + si.perm_off;
  const int ret_cols = LEVELS ? 0 : pmeta[q].ret_chunks * kChunk;
  const int n_ret0 = LEVELS ? 0 : pmeta[q].n_ret;

  uint4 raw[kPrepIter];
#pragma unroll
  for (int it = 0; it < kPrepIter; ++it) {
    const int tl = tfirst + it * TPB;
    raw[it] = make_uint4(0, 0, 0, 0);
    if (tl < si.len)
      raw[it] = prep_load16(keys + h * hs_bytes + (si.start + tl) * ts_bytes + sub * 16);
  }
#pragma unroll
  for (int it = 0; it < kPrepIter; ++it) {
    const int tl = tfirst + it * TPB;
    const bool valid = tl < si.len;
    const int64_t tt = si.start + (valid ? tl : 0);
    // this token's column list: its group's (LEVELS) or the single split's
    int64_t goff = 0;
    bool r;
    int n_ret = n_ret0;
    if constexpr (LEVELS) {
      const int l = lv.level[h * T + tt];
      const int g = (l >= 1 && l <= lv.n_levels) ? l - 1
                    : (lv.n_groups > lv.n_levels ? lv.n_levels : -1);
      r = g >= 0;                      // a member of its group's list; else copied nowhere
      goff = (int64_t)(r ? g : 0) * lv.group_stride;
      n_ret = byte_offset(pmeta, goff)[q].n_ret;
    } else {
      r = retained != nullptr && retained[h * T + tt] != 0;
    }
    const int pr = byte_offset(prank, goff)[base + (valid ? tl : 0)];
    const int p = r ? pr : ret_cols + ((valid ? tl : 0) - pr);
    const bool copy = valid && (r || copy_evicted);  // evicted columns only for all-keys sweeps
    // The last column of a group fills the rest of its 32-column chunk with copies of itself
    // (key and inverse norm; the position list keeps -1 there), so that chunk holds only
    // exact ties of a real column and the similarity sweep needs no padding test for it.
    const int last = r ? n_ret - 1 : ret_cols + (si.len - n_ret) - 1;
    const int fill_end = (p == last && copy) ? (p / kChunk + 1) * kChunk : p + 1;
    uint16_t* const gkeys = byte_offset(pkeys, goff);
    float* const grcol = byte_offset(rcol, goff);

    double ss = 0.0;
    if constexpr (F32) {
      float v[4] = {__uint_as_float(raw[it].x), __uint_as_float(raw[it].y),
                    __uint_as_float(raw[it].z), __uint_as_float(raw[it].w)};
      uint16_t hs[4], ls[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        ss += (double)v[e] * (double)v[e];
        hs[e] = bf16_rne(v[e]);
        ls[e] = bf16_rne(v[e] - bf16_to_f32(hs[e]));  // v - hi is exact in fp32
      }
      if (valid) {
        uint2 phi, plo;
        phi.x = hs[0] | ((uint32_t)hs[1] << 16);
        phi.y = hs[2] | ((uint32_t)hs[3] << 16);
        plo.x = ls[0] | ((uint32_t)ls[1] << 16);
        plo.y = ls[2] | ((uint32_t)ls[3] << 16);
        uint16_t* row = hilo + (h * T + tt) * (2 * D) + sub * 4;
        *reinterpret_cast<uint2*>(row) = phi;
        *reinterpret_cast<uint2*>(row + D) = plo;
        for (int k = p; copy && k < fill_end; ++k) {
          uint16_t* dk = gkeys + (base + k) * DCOL;
          *reinterpret_cast<uint2*>(dk + sub * 4) = phi;
          *reinterpret_cast<uint2*>(dk + D + sub * 4) = plo;
        }
      }
    } else {
      const uint32_t wds[4] = {raw[it].x, raw[it].y, raw[it].z, raw[it].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const double x0 = (double)__uint_as_float(wds[e] << 16);
        const double x1 = (double)__uint_as_float(wds[e] & 0xFFFF0000u);
        ss += x0 * x0 + x1 * x1;
      }
      for (int k = p; copy && k < fill_end; ++k)
        prep_store16(gkeys + (base + k) * DCOL + sub * 8, raw[it]);
    }
#pragma unroll
    for (int off = LPT / 2; off > 0; off >>= 1) ss += __shfl_xor(ss, off, LPT);
    if (valid && sub == 0) {
      float rv;
      const bool bad = !(ss < 1.0e300);                    // NaN or Inf in the key
      if (bad) rv = __uint_as_float(0x7FC00000u);
      else if (ss > 0.0) rv = (float)(1.0 / sqrt(ss));
      else rv = 0.0f;                                       // zero key: similarity 0 to all
      rinv[h * T + tt] = rv;
      // (a token in no group of the LEVELS pass has no column anywhere)
      for (int k = p; (copy || !LEVELS) && k < fill_end; ++k) grcol[base + k] = rv;
      if (bad) {
        for (int g = 0; g < (LEVELS ? lv.n_groups : 1); ++g)  // every list of the problem
          atomicOr(&byte_offset(pmeta, (int64_t)g * lv.group_stride)[q].flags, kFlagNonfinite);
        if (status) status[q] = 2;  // TWINKV_PROBLEM_NONFINITE
      }
    }
  }
}

template <int D, bool F32>
constexpr int prep_tokens_per_block() {
  return 256 / (D * (F32 ? 4 : 2) / 16) * kPrepIter;
}

template <int D, bool F32, bool LEVELS>
hipError_t run_prepare(const void* keys, int n_heads, int64_t T, int64_t hs, int64_t ts,
                       int64_t PT, int total_blocks, const uint8_t* retained, const int32_t* prank,
                       ProblemMeta* pmeta, const SeqInfo* seqtab, int n_seqs, float* rinv,
                       float* rcol, uint16_t* hilo, uint16_t* pkeys, int32_t* status,
                       int copy_evicted, const PrepLevels& lv, hipStream_t st) {
  constexpr int ESZ = F32 ? 4 : 2;
  if (total_blocks == 0 || n_heads == 0) return hipSuccess;
  for (int h0 = 0; h0 < n_heads; h0 += 65535) {  // heads along y, in slices the grid holds
    const int by = n_heads - h0 < 65535 ? n_heads - h0 : 65535;
    hipLaunchKernelGGL((prepare_keys_kernel<D, F32, LEVELS>),
                       dim3((unsigned)total_blocks, (unsigned)by), dim3(256), 0, st,
                       (const uint8_t*)keys, T, hs * ESZ, ts * ESZ, PT, retained, prank, pmeta,
                       seqtab, n_seqs, rinv, rcol, hilo, pkeys, status, h0, copy_evicted, lv);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

template <bool LEVELS>
int prepare_dispatch(const void* keys, int dtype, int d, int n_heads, int64_t T,
                     int64_t head_stride, int64_t token_stride, int64_t PT, int total_blocks,
                     const uint8_t* retained, const int32_t* prank, ProblemMeta* pmeta,
                     const SeqInfo* seqtab, int n_seqs, float* rinv, float* rcol, uint16_t* hilo,
                     uint16_t* pkeys, int32_t* status, int copy_evicted, const PrepLevels& lv,
                     void* stream) {
  hipStream_t st = (hipStream_t)stream;
  if (dtype == 0 && d == 64)
    return run_prepare<64, false, LEVELS>(keys, n_heads, T, head_stride, token_stride, PT,
                                          total_blocks, retained, prank, pmeta, seqtab, n_seqs,
                                          rinv, rcol, hilo, pkeys, status, copy_evicted, lv, st);
  if (dtype == 0 && d == 128)
    return run_prepare<128, false, LEVELS>(keys, n_heads, T, head_stride, token_stride, PT,
                                           total_blocks, retained, prank, pmeta, seqtab, n_seqs,
                                           rinv, rcol, hilo, pkeys, status, copy_evicted, lv, st);
  if (dtype == 1 && d == 64)
    return run_prepare<64, true, LEVELS>(keys, n_heads, T, head_stride, token_stride, PT,
                                         total_blocks, retained, prank, pmeta, seqtab, n_seqs,
                                         rinv, rcol, hilo, pkeys, status, copy_evicted, lv, st);
  if (dtype == 1 && d == 128)
    return run_prepare<128, true, LEVELS>(keys, n_heads, T, head_stride, token_stride, PT,
                                          total_blocks, retained, prank, pmeta, seqtab, n_seqs,
                                          rinv, rcol, hilo, pkeys, status, copy_evicted, lv, st);
  return hipErrorInvalidValue;
}

}  // namespace

int launch_partition(const uint8_t* retained, const SeqInfo* seqtab, int n_heads, int n_seqs,
                     int64_t T, int64_t PT, int max_len, int32_t* pcol, float* rcol,
                     int32_t* prank, ProblemMeta* pmeta, int32_t* status, void* stream) {
  const int64_t P = (int64_t)n_heads * n_seqs;
  if (P == 0) return hipSuccess;
  if (max_len > 4096)
    hipLaunchKernelGGL(partition_kernel<1024>, dim3((unsigned)P), dim3(1024), 0,
                       (hipStream_t)stream, retained, seqtab, n_seqs, T, PT, pcol, rcol, prank,
                       pmeta, status);
  else
    hipLaunchKernelGGL(partition_kernel<256>, dim3((unsigned)P), dim3(256), 0,
                       (hipStream_t)stream, retained, seqtab, n_seqs, T, PT, pcol, rcol, prank,
                       pmeta, status);
  return hipGetLastError();
}

int prepare_tokens_per_block(int dtype, int d) {
  if (dtype == 0 && d == 64) return prep_tokens_per_block<64, false>();
  if (dtype == 0 && d == 128) return prep_tokens_per_block<128, false>();
  if (dtype == 1 && d == 64) return prep_tokens_per_block<64, true>();
  if (dtype == 1 && d == 128) return prep_tokens_per_block<128, true>();
  return 0;
}

int launch_prepare_keys(const void* keys, int dtype, int d, int n_heads, int64_t T,
                        int64_t head_stride, int64_t token_stride, int64_t PT, int total_blocks,
                        const uint8_t* retained, const int32_t* prank, ProblemMeta* pmeta,
                        const SeqInfo* seqtab, int n_seqs, float* rinv, float* rcol,
                        uint16_t* hilo, uint16_t* pkeys, int32_t* status, int copy_evicted,
                        void* stream) {
  const PrepLevels none{nullptr, 0, 1, 0};
  return prepare_dispatch<false>(keys, dtype, d, n_heads, T, head_stride, token_stride, PT,
                                 total_blocks, retained, prank, pmeta, seqtab, n_seqs, rinv, rcol,
                                 hilo, pkeys, status, copy_evicted, none, stream);
}

int launch_prepare_keys_levels(const void* keys, int dtype, int d, int n_heads, int64_t T,
                               int64_t head_stride, int64_t token_stride, int64_t PT,
                               int total_blocks, const PrepLevels& lv, const int32_t* prank,
                               ProblemMeta* pmeta, const SeqInfo* seqtab, int n_seqs, float* rinv,
                               float* rcol, uint16_t* hilo, uint16_t* pkeys, int32_t* status,
                               void* stream) {
  return prepare_dispatch<true>(keys, dtype, d, n_heads, T, head_stride, token_stride, PT,
                                total_blocks, nullptr, prank, pmeta, seqtab, n_seqs, rinv, rcol,
                                hilo, pkeys, status, /*copy_evicted=*/0, lv, stream);
}

}  // namespace twinkv
