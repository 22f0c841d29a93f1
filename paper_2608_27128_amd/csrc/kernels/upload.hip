// Host tables (the per-sequence schedule, the compaction's chunk list) reach the device as
// kernel arguments: each launch carries up to kUploadBytes of the table by value and its
// threads store it to the workspace with vector stores.  The arguments are copied when the
// launch is enqueued (or captured into a graph), so nothing reads the caller's host memory
// later, and no pageable host-to-device copy stalls the host.
#include <hip/hip_runtime.h>

#include <cstring>

#include "twinkv_internal.h"

namespace twinkv {
namespace {

constexpr int kUploadWords = 896;  // 3584 bytes of the 4 KB kernel-argument limit
constexpr int kUploadThreads = 256;

struct UploadPiece {
  uint32_t w[kUploadWords];
};

__global__ void __launch_bounds__(kUploadThreads) upload_kernel(const UploadPiece piece,
                                                                uint32_t* __restrict__ dst,
                                                                int n_words) {
  for (int i = threadIdx.x; i < n_words; i += kUploadThreads) dst[i] = piece.w[i];
}

}  // namespace

int launch_upload(const void* src, size_t bytes, void* dst, void* stream) {
  if (bytes % 4 != 0) return (int)hipErrorInvalidValue;
  const uint32_t* s = static_cast<const uint32_t*>(src);
  uint32_t* d = static_cast<uint32_t*>(dst);
  size_t words = bytes / 4;
  UploadPiece piece;
  while (words > 0) {
    const int n = (int)(words < (size_t)kUploadWords ? words : (size_t)kUploadWords);
    std::memcpy(piece.w, s, 4 * (size_t)n);
    hipLaunchKernelGGL(upload_kernel, dim3(1), dim3(kUploadThreads), 0, (hipStream_t)stream,
                       piece, d, n);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return (int)e;
    s += n;
    d += n;
    words -= (size_t)n;
  }
  return 0;
}

}  // namespace twinkv
