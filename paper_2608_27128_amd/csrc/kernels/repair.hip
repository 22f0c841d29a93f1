// K3: the composable repair pass of Sec. 3.4 for one problem per workgroup.
//
//   orphan  i not in S0, b_i < tau
//   donor   j in S0, outside [0, n_sink) and [len - n_recent, len), b_j >= tau
//   m = min(|O|, |D|); admit the m orphans of lowest (b, position), evict the m donors of
//   highest b (ties: lowest position first); S1 has exactly |S0| members.
//
// Since m = min(|O|, |D|), at least one side is taken whole; the other side needs the
// m-th smallest key, found by an MSB-first 8-bit radix select on order-preserving float
// keys (histograms in LDS), then a block-wide scan in position order to take exactly the
// remaining members equal to that key.  Every pass streams b and S0 (5 bytes per token).
#include <hip/hip_runtime.h>

#include "../twinkv_internal.h"

namespace twinkv {
namespace {

constexpr int kRepThreads = 256;

// Order-preserving map of fp32 onto uint32 (+0 and -0 map to the same key).
__device__ inline uint32_t ord_key(float x) {
  const uint32_t u = __float_as_uint(x == 0.0f ? 0.0f : x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Exclusive prefix sum over the block; `total` receives the block sum.
__device__ inline int block_exclusive_scan(int v, int* s_wave, int& total) {
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
  for (int k = 0; k < kRepThreads / 64; ++k) {
    const int t = s_wave[k];
    base += (k < wv) ? t : 0;
    total += t;
  }
  __syncthreads();
  return base + x - v;
}

__global__ __launch_bounds__(kRepThreads) void repair_kernel(RepairArgs a) {
  __shared__ int s_wave[kRepThreads / 64];
  __shared__ int s_hist[256];
  __shared__ int s_digit, s_before;

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
  const int tid = threadIdx.x;

  // ---- pass 1: counts ----
  int c_ret = 0, c_o = 0, c_d = 0, bad = 0;
  for (int t = tid; t < len; t += kRepThreads) {
    const float x = b[t];
    const bool r = s0[t] != 0;
    const bool prot = t < a.n_sink || t >= rec0;
    bad |= !(fabsf(x) <= 3.4e38f);
    c_ret += r;
    c_o += (!r && x < tau);
    c_d += (r && !prot && x >= tau);
  }
  int tot_ret, tot_o, tot_d, tot_bad;
  (void)block_exclusive_scan(c_ret, s_wave, tot_ret);
  (void)block_exclusive_scan(c_o, s_wave, tot_o);
  (void)block_exclusive_scan(c_d, s_wave, tot_d);
  (void)block_exclusive_scan(bad, s_wave, tot_bad);

  int status = 0;
  if (tot_bad || (a.pmeta && (a.pmeta[q].flags & kFlagNonfinite))) status = 2;
  else if (si.budget >= 0 && tot_ret != si.budget) status = 1;
  const int m = status == 0 ? min(tot_o, tot_d) : 0;
  const bool sel_o = m > 0 && tot_o > m;  // orphans must be cut at the m-th
  const bool sel_d = m > 0 && tot_d > m;  // donors must be cut at the m-th

  // ---- radix select of the m-th smallest key on the side that is cut ----
  uint32_t key_cut = 0xFFFFFFFFu;
  int take_eq = 0;
  if (sel_o || sel_d) {
    uint32_t prefix = 0, mask = 0;
    int kk = m;  // 1-based rank still to find among candidates matching `prefix`
    for (int shift = 24; shift >= 0; shift -= 8) {
      s_hist[tid] = 0;
      __syncthreads();
      for (int t = tid; t < len; t += kRepThreads) {
        const float x = b[t];
        const bool r = s0[t] != 0;
        bool member;
        uint32_t key;
        if (sel_o) {
          member = !r && x < tau;
          key = ord_key(x);
        } else {
          member = r && !(t < a.n_sink || t >= rec0) && x >= tau;
          key = ~ord_key(x);
        }
        if (member && (key & mask) == prefix) atomicAdd(&s_hist[(key >> shift) & 255u], 1);
      }
      __syncthreads();
      const int hcount = s_hist[tid];
      int dummy;
      const int before = block_exclusive_scan(hcount, s_wave, dummy);
      if (before < kk && kk <= before + hcount) {
        s_digit = tid;
        s_before = before;
      }
      __syncthreads();
      kk -= s_before;
      prefix |= (uint32_t)s_digit << shift;
      mask |= 0xFFu << shift;
      __syncthreads();
    }
    key_cut = prefix;
    take_eq = kk;  // members with key == key_cut to take, in position order
  }

  // ---- final pass: contiguous ranges per thread so equal keys are ranked by position ----
  const int chunk = (len + kRepThreads - 1) / kRepThreads;
  const int t0 = min(len, tid * chunk);
  const int t1 = min(len, t0 + chunk);
  int eq_here = 0;
  if (sel_o || sel_d) {
    for (int t = t0; t < t1; ++t) {
      const float x = b[t];
      const bool r = s0[t] != 0;
      if (sel_o) eq_here += (!r && x < tau && ord_key(x) == key_cut);
      else eq_here += (r && !(t < a.n_sink || t >= rec0) && x >= tau && ~ord_key(x) == key_cut);
    }
  }
  int dummy;
  int eq_rank = block_exclusive_scan(eq_here, s_wave, dummy);
  for (int t = t0; t < t1; ++t) {
    const float x = b[t];
    const bool r = s0[t] != 0;
    uint8_t out = r ? 1 : 0;
    if (m > 0) {
      if (!r && x < tau) {  // orphan
        bool admit = true;
        if (sel_o) {
          const uint32_t key = ord_key(x);
          admit = key < key_cut || (key == key_cut && eq_rank++ < take_eq);
        }
        if (admit) out = 1;
      } else if (r && !(t < a.n_sink || t >= rec0) && x >= tau) {  // donor
        bool evict = true;
        if (sel_d) {
          const uint32_t key = ~ord_key(x);
          evict = key < key_cut || (key == key_cut && eq_rank++ < take_eq);
        }
        if (evict) out = 0;
      }
    }
    s1[t] = out;
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
  hipLaunchKernelGGL(repair_kernel, dim3((unsigned)P), dim3(kRepThreads), 0, (hipStream_t)stream, a);
  return hipGetLastError();
}

}  // namespace twinkv
