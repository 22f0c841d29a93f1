// Nested retained sets S_1 within S_2 within ... within S_L (a budget sweep of one policy,
// Sec. 3.4 Eq. 4 for each set): b_i(S_k) is the best of the per-group maxima over the level
// groups G_1 .. G_k (G_g = S_g minus S_{g-1}), each group computed once by the retained-only
// similarity sweep.  These two small kernels select a group's mask and merge the maxima.
#include <hip/hip_runtime.h>

#include "../twinkv_internal.h"

namespace twinkv {
namespace {

constexpr int kThreads = 256;

// mask = the tokens of group sel: level == sel for sel >= 1; for sel == 0 the tokens in no
// set (level 0 or above n_levels).
__global__ __launch_bounds__(kThreads) void select_level_kernel(const uint8_t* __restrict__ level,
                                                                uint8_t* __restrict__ mask,
                                                                int64_t n, int sel, int n_levels) {
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i >= n) return;
  const int lv = level[i];
  mask[i] = (sel > 0 ? lv == sel : (lv == 0 || lv > n_levels)) ? 1 : 0;
}

// (v2, j2) beats (v1, j1): a candidate beats none; then the larger value; then the smaller
// position (the tie rule of the single-set sweep).
__device__ inline bool beats(float v2, int j2, float v1, int j1) {
  if (j2 < 0) return false;
  if (j1 < 0) return true;
  return v2 > v1 || (v2 == v1 && j2 < j1);
}

__global__ __launch_bounds__(kThreads) void combine_levels_kernel(CombineArgs a) {
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i >= a.n) return;
  float v = -1.0f;
  int j = -1;
  for (int g = 0; g < a.n_groups; ++g) {
    const float v2 = a.gbest[g * a.n + i];
    const int j2 = a.garg[g * a.n + i];
    if (beats(v2, j2, v, j)) {
      v = v2;
      j = j2;
    }
    if (g < a.n_levels) {
      if (a.best_lvl) a.best_lvl[g * a.n + i] = v;
      if (a.arg_lvl) a.arg_lvl[g * a.n + i] = j;
    }
  }
  if (a.best_all) a.best_all[i] = v;
  if (a.arg_all) a.arg_all[i] = j;
}

}  // namespace

int launch_select_level(const uint8_t* level, uint8_t* mask, int64_t n, int sel, int n_levels,
                        void* stream) {
  if (n == 0) return hipSuccess;
  const int64_t blocks = (n + kThreads - 1) / kThreads;
  hipLaunchKernelGGL(select_level_kernel, dim3((unsigned)blocks), dim3(kThreads), 0,
                     (hipStream_t)stream, level, mask, n, sel, n_levels);
  return hipGetLastError();
}

int launch_combine_levels(const CombineArgs& a, void* stream) {
  if (a.n == 0) return hipSuccess;
  const int64_t blocks = (a.n + kThreads - 1) / kThreads;
  hipLaunchKernelGGL(combine_levels_kernel, dim3((unsigned)blocks), dim3(kThreads), 0,
                     (hipStream_t)stream, a);
  return hipGetLastError();
}

}  // namespace twinkv
