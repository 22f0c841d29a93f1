// K3: the composable repair pass of Sec. 3.4 for one problem per workgroup.
//
//   orphan  i not in S0, b_i < tau
//   donor   j in S0, outside [0, n_sink) and [len - n_recent, len), b_j >= tau
//   m = min(|O|, |D|); admit the m orphans of lowest (b, position), evict the m donors of
//   highest b (ties: lowest position first); S1 has exactly |S0| members.
//
// Since m = min(|O|, |D|), at least one side is taken whole; the other side needs the
// m-th smallest key, found by an MSB-first radix select (11/11/10-bit digits, LDS
// histograms) on order-preserving float keys, then a block-wide scan in position order to
// take exactly the remaining members equal to that key.  1024 threads per problem (256 when
// every sequence is short); every
// pass streams b and S0 (5 bytes per token).
#include <hip/hip_runtime.h>

#include "../twinkv_internal.h"
#include "block_select.h"

namespace twinkv {
namespace {

// Order-preserving map of fp32 onto uint32 (+0 and -0 map to the same key).
__device__ inline uint32_t ord_key(float x) {
  const uint32_t u = __float_as_uint(x == 0.0f ? 0.0f : x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

template <int NT>
__global__ __launch_bounds__(NT) void repair_kernel(RepairArgs a) {
  __shared__ int s_wave[NT / 64];
  __shared__ int s_hist[kSelBins];
  __shared__ int s_pick[2];

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
  auto is_orphan = [&](int t, float x, bool r) { return !r && x < tau; };
  auto is_donor = [&](int t, float x, bool r) {
    return r && !(t < a.n_sink || t >= rec0) && x >= tau;
  };

  // ---- pass 1: counts ----
  int c_ret = 0, c_o = 0, c_d = 0, bad = 0;
  for (int t = tid; t < len; t += NT) {
    const float x = b[t];
    const bool r = s0[t] != 0;
    bad |= !(fabsf(x) <= 3.4e38f);
    c_ret += r;
    c_o += is_orphan(t, x, r);
    c_d += is_donor(t, x, r);
  }
  int tot_ret, tot_o, tot_d, tot_bad;
  (void)sel_exclusive_scan<NT>(c_ret, s_wave, tot_ret);
  (void)sel_exclusive_scan<NT>(c_o, s_wave, tot_o);
  (void)sel_exclusive_scan<NT>(c_d, s_wave, tot_d);
  (void)sel_exclusive_scan<NT>(bad, s_wave, tot_bad);

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
    key_cut = block_select<NT>(
        len, m,
        [&](int t, uint32_t& key) {
          const float x = b[t];
          const bool r = s0[t] != 0;
          if (sel_o) {
            key = ord_key(x);
            return is_orphan(t, x, r);
          }
          key = ~ord_key(x);
          return is_donor(t, x, r);
        },
        s_hist, s_wave, s_pick, take_eq);
  }

  // ---- final pass: contiguous ranges per thread so equal keys are ranked by position ----
  const int chunk = (len + NT - 1) / NT;
  const int t0 = min(len, tid * chunk);
  const int t1 = min(len, t0 + chunk);
  int eq_here = 0;
  if (sel_o || sel_d) {
    for (int t = t0; t < t1; ++t) {
      const float x = b[t];
      const bool r = s0[t] != 0;
      if (sel_o) eq_here += (is_orphan(t, x, r) && ord_key(x) == key_cut);
      else eq_here += (is_donor(t, x, r) && ~ord_key(x) == key_cut);
    }
  }
  int dummy;
  int eq_rank = sel_exclusive_scan<NT>(eq_here, s_wave, dummy);
  for (int t = t0; t < t1; ++t) {
    const float x = b[t];
    const bool r = s0[t] != 0;
    uint8_t out = r ? 1 : 0;
    if (m > 0) {
      if (is_orphan(t, x, r)) {
        bool admit = true;
        if (sel_o) {
          const uint32_t key = ord_key(x);
          admit = key < key_cut || (key == key_cut && eq_rank++ < take_eq);
        }
        if (admit) out = 1;
      } else if (is_donor(t, x, r)) {
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
  // short sequences: 256 threads per problem keep more problems in flight
  if (a.max_len > 4096)
    hipLaunchKernelGGL(repair_kernel<1024>, dim3((unsigned)P), dim3(1024), 0, (hipStream_t)stream, a);
  else
    hipLaunchKernelGGL(repair_kernel<256>, dim3((unsigned)P), dim3(256), 0, (hipStream_t)stream, a);
  return hipGetLastError();
}

}  // namespace twinkv
