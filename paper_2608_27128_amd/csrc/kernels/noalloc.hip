// twinkv_repair_from_scores_noalloc: twinkv_repair_from_scores without a workspace, for
// callers that cannot allocate device memory.  Its only scratch, the per-sequence table K3
// reads, lives in the file-scope device array `scratch` below.  Each GPU holds its own copy
// (allocated with the code object, kept until the process ends); its address on the current
// device is looked up once with hipGetSymbolAddress and that pointer, never the array's name,
// is what host code hands to the kernels.
#include <hip/hip_runtime.h>

#include <mutex>

#include "twinkv.h"
#include "../twinkv_internal.h"

namespace twinkv {
namespace {

constexpr size_t kScratchBytes = (size_t)TWINKV_NOALLOC_MAX_SEQS * sizeof(SeqInfo);
static_assert(kScratchBytes == 64 * 1024, "2048 sequences of 32-byte table entries");

__device__ __align__(256) char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on the current device, looked up on the first call there.
void* scratch_address() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return nullptr;
    g_scratch_ptr[dev] = p;
  }
  return g_scratch_ptr[dev];
}

}  // namespace
}  // namespace twinkv

extern "C" int twinkv_repair_from_scores_noalloc(const float* b, const uint8_t* retained_in,
                                                 uint8_t* retained_out, int n_heads, int n_seqs,
                                                 const int64_t* cu_seqlens, const int64_t* budget,
                                                 float tau, int n_sink, int n_recent,
                                                 int32_t* stats, void* stream) {
  return twinkv::repair_from_scores_into(b, retained_in, retained_out, n_heads, n_seqs,
                                         cu_seqlens, budget, tau, n_sink, n_recent, stats,
                                         nullptr, twinkv::kScratchBytes,
                                         &twinkv::scratch_address, stream);
}
