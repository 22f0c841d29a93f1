// K5: KV compaction (Sec. 3.1): eviction keeps only the keys and values at the retained
// positions, so each problem's kept rows are gathered, in ascending position order, into
// its reserved rows of a dense cache.
//
// HBM-bound gather in two launches over (head, 2048-token chunk) workgroups:
//  * K5a reads the retained mask once and writes the number of kept positions per chunk.
//  * K5b sums the counts of the earlier chunks of its sequence (the first output row of the
//    chunk) and of all its chunks (the problem total, for the capacity check), ranks the
//    kept positions of the chunk with wave ballots, lists them in LDS, and copies their rows
//    16 bytes a lane: consecutive lanes take consecutive 16-byte pieces of consecutive kept
//    rows, so a wave moves 1 KB of contiguous output per instruction.  Reserved rows past the
//    kept count (or all of them, when the problem keeps more than it has rows) are zeroed
//    by the chunk that covers them.
#include <hip/hip_runtime.h>

#include "../twinkv_internal.h"

namespace twinkv {
namespace {

#ifndef TWINKV_COMPACT_THREADS
#define TWINKV_COMPACT_THREADS 256
#endif
#ifndef TWINKV_COMPACT_UNROLL
#define TWINKV_COMPACT_UNROLL 4
#endif
#ifndef TWINKV_COMPACT_NT
#define TWINKV_COMPACT_NT 1
#endif
constexpr int kThreads = TWINKV_COMPACT_THREADS;
constexpr int kSlabs = kCompactChunk / kThreads;  // mask bytes per thread per chunk
constexpr int kUnroll = TWINKV_COMPACT_UNROLL;    // 16-byte pieces in flight per lane
static_assert(kCompactChunk % kThreads == 0, "a chunk is a whole number of slabs");

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ inline u32x4 load16(const char* p) {
  if constexpr (TWINKV_COMPACT_NT) return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  else return *reinterpret_cast<const u32x4*>(p);
}
__device__ inline void store16(char* p, u32x4 v) {
  if constexpr (TWINKV_COMPACT_NT) __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(p));
  else *reinterpret_cast<u32x4*>(p) = v;
}

// Block-wide sum of two ints (every thread gets both totals).
__device__ inline void block_sum2(int& x, int& y, int (*s_red)[kThreads / 64]) {
  for (int off = 32; off > 0; off >>= 1) {
    x += __shfl_xor(x, off);
    y += __shfl_xor(y, off);
  }
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    s_red[0][w] = x;
    s_red[1][w] = y;
  }
  __syncthreads();
  x = 0;
  y = 0;
#pragma unroll
  for (int k = 0; k < kThreads / 64; ++k) {
    x += s_red[0][k];
    y += s_red[1][k];
  }
  __syncthreads();
}

struct ChunkPos {
  int h, g, c;      // head, global chunk, chunk inside its sequence
  CompactSeq cs;
};

__device__ inline ChunkPos chunk_pos(const CompactArgs& a) {
  ChunkPos p;
  p.h = (int)(blockIdx.x / (unsigned)a.n_chunks);
  p.g = (int)(blockIdx.x - (unsigned)p.h * (unsigned)a.n_chunks);
  p.cs = a.seqs[a.chunk_seq[p.g]];
  p.c = p.g - p.cs.chunk0;
  return p;
}

__global__ __launch_bounds__(kThreads) void compact_count_kernel(CompactArgs a) {
  __shared__ int s_red[2][kThreads / 64];
  const ChunkPos p = chunk_pos(a);
  const uint8_t* m = a.retained + (int64_t)p.h * a.T + p.cs.start;
  const int t0 = p.c * kCompactChunk;
  int cnt = 0, dummy = 0;
#pragma unroll
  for (int k = 0; k < kSlabs; ++k) {
    const int t = t0 + k * kThreads + (int)threadIdx.x;
    if (t < p.cs.len) cnt += m[t] != 0;
  }
  block_sum2(cnt, dummy, s_red);
  if (threadIdx.x == 0) a.chunk_cnt[(int64_t)p.h * a.n_chunks + p.g] = cnt;
}

// Copies (or, with s_src == nullptr, zeroes) `rows` rows of row_bytes starting at output
// row `orow`; row r's source is token s_src[r] of the sequence.
__device__ inline void move_rows(const CompactArgs& a, int h, int64_t tok0, int64_t orow,
                                 int rows, const int* s_src) {
  const int lpr = a.log2_pieces;  // 16-byte pieces per row, as a power of two
  const int pr = 1 << lpr;
  const int n = rows * pr;
  const char* kbase = a.keys + (int64_t)h * a.head_stride;
  const char* vbase = a.values ? a.values + (int64_t)h * a.v_head_stride : nullptr;
  char* kout = a.keys_out + orow * a.row_bytes;
  char* vout = a.values_out ? a.values_out + orow * a.row_bytes : nullptr;
  for (int p0 = (int)threadIdx.x; p0 < n; p0 += kUnroll * kThreads) {
    u32x4 kx[kUnroll], vx[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int p = p0 + u * kThreads;
      kx[u] = u32x4{0u, 0u, 0u, 0u};
      vx[u] = u32x4{0u, 0u, 0u, 0u};
      if (s_src != nullptr && p < n) {
        const int64_t t = tok0 + s_src[p >> lpr];
        const int off = (p & (pr - 1)) * 16;
        kx[u] = load16(kbase + t * a.token_stride + off);
        if (vbase) vx[u] = load16(vbase + t * a.v_token_stride + off);
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int p = p0 + u * kThreads;
      if (p < n) {
        store16(kout + (int64_t)p * 16, kx[u]);
        if (vout) store16(vout + (int64_t)p * 16, vx[u]);
      }
    }
  }
}

__global__ __launch_bounds__(kThreads) void compact_gather_kernel(CompactArgs a) {
  __shared__ int s_src[kCompactChunk];
  __shared__ int s_wc[kSlabs][kThreads / 64];
  __shared__ int s_red[2][kThreads / 64];
  const ChunkPos p = chunk_pos(a);
  const CompactSeq& cs = p.cs;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;

  // rows written by earlier chunks of this problem, and the problem's total
  int before = 0, total = 0;
  const int32_t* cnt = a.chunk_cnt + (int64_t)p.h * a.n_chunks + cs.chunk0;
  for (int k = tid; k < cs.nchunks; k += kThreads) {
    const int v = cnt[k];
    total += v;
    before += k < p.c ? v : 0;
  }
  block_sum2(before, total, s_red);
  const bool over = total > cs.cap;
  const int64_t orow0 = (int64_t)p.h * a.C + cs.out_start;  // first reserved row
  const int64_t tok0 = cs.start;
  const int t0 = p.c * kCompactChunk;

  if (!over) {
    // rank of each kept position inside the chunk: slab k (256 positions) after slab k-1,
    // wave w after wave w-1, lanes by ballot
    const uint8_t* m = a.retained + (int64_t)p.h * a.T + cs.start;
    uint64_t bal[kSlabs];
#pragma unroll
    for (int k = 0; k < kSlabs; ++k) {
      const int t = t0 + k * kThreads + tid;
      const bool keep = t < cs.len && m[t] != 0;
      bal[k] = __ballot(keep);
      if (lane == 0) s_wc[k][wave] = __popcll(bal[k]);
    }
    __syncthreads();
    const uint64_t below = lane ? (~0ull >> (64 - lane)) : 0ull;
    int run = 0;
#pragma unroll
    for (int k = 0; k < kSlabs; ++k) {
      int here = run;
#pragma unroll
      for (int w = 0; w < kThreads / 64; ++w) {
        here += w < wave ? s_wc[k][w] : 0;
        run += s_wc[k][w];
      }
      if ((bal[k] >> lane) & 1ull) s_src[here + __popcll(bal[k] & below)] = t0 + k * kThreads + tid;
    }
    const int nk = run;
    __syncthreads();
    move_rows(a, p.h, tok0, orow0 + before, nk, s_src);
    if (a.pos_out)
      for (int r = tid; r < nk; r += kThreads) a.pos_out[orow0 + before + r] = s_src[r];
  }

  // unused reserved rows: [used, cap) split by chunk ranges of rows (cap <= len, so the
  // chunks of the sequence cover every reserved row)
  const int used = over ? 0 : total;
  const int z0 = max(used, t0);
  const int z1 = min(cs.cap, t0 + kCompactChunk);
  if (z1 > z0) {
    move_rows(a, p.h, tok0, orow0 + z0, z1 - z0, nullptr);
    if (a.pos_out)
      for (int r = z0 + tid; r < z1; r += kThreads) a.pos_out[orow0 + r] = -1;
  }
  if (p.c == 0 && tid == 0) {
    int32_t* st = a.stats + 4 * ((int64_t)p.h * a.n_seqs + a.chunk_seq[p.g]);
    st[0] = total;
    st[1] = cs.cap;
    st[2] = over ? 1 : 0;
    st[3] = 0;
  }
}

}  // namespace

int launch_compact_count(const CompactArgs& a, void* stream) {
  const int64_t blocks = (int64_t)a.n_heads * a.n_chunks;
  if (blocks == 0) return hipSuccess;
  hipLaunchKernelGGL(compact_count_kernel, dim3((unsigned)blocks), dim3(kThreads), 0,
                     (hipStream_t)stream, a);
  return hipGetLastError();
}

int launch_compact_gather(const CompactArgs& a, void* stream) {
  const int64_t blocks = (int64_t)a.n_heads * a.n_chunks;
  if (blocks == 0) return hipSuccess;
  hipLaunchKernelGGL(compact_gather_kernel, dim3((unsigned)blocks), dim3(kThreads), 0,
                     (hipStream_t)stream, a);
  return hipGetLastError();
}

}  // namespace twinkv
