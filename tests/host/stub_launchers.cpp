// Host-only stand-ins for the kernel launchers of the library, for running the C ABI's host
// layer (csrc/api.cpp: validation, workspace layout, sequence tables, launch arguments) under
// AddressSanitizer / UndefinedBehaviorSanitizer on a machine without a GPU.
//
// Every "device" buffer in these tests is host memory of exactly the size the caller or the
// workspace query gives, so each stub touches the first and the last byte of every range a
// real kernel would address: a range that leaves its allocation is reported by the sanitizer.
// Tables uploaded with launch_upload are copied into their workspace slot the same way.
#include <hip/hip_runtime_api.h>

#include <cstdint>
#include <cstdio>
#include <cstring>

#include "twinkv_internal.h"

namespace stub {
int64_t g_launches = 0;
volatile unsigned char g_sink = 0;

// Reads the first and the last byte of [p, p + bytes) (no-op for an empty range).
void touch(const void* p, int64_t bytes) {
  if (bytes <= 0) return;
  if (p == nullptr) {
    std::fprintf(stderr, "stub: null pointer for a range of %lld bytes\n", (long long)bytes);
    std::abort();
  }
  const unsigned char* c = static_cast<const unsigned char*>(p);
  g_sink = g_sink ^ c[0] ^ c[bytes - 1];
}
// Writes the first and the last byte (output ranges).
void touch_out(void* p, int64_t bytes) {
  if (bytes <= 0 || p == nullptr) return;
  unsigned char* c = static_cast<unsigned char*>(p);
  c[0] = 0;
  c[bytes - 1] = 0;
}
}  // namespace stub

using stub::touch;
using stub::touch_out;

extern "C" hipError_t hipEventRecord(hipEvent_t, hipStream_t) { return hipSuccess; }

namespace twinkv {

int launch_upload(const void* src, size_t bytes, void* dst, void*) {
  ++stub::g_launches;
  std::memcpy(dst, src, bytes);
  return 0;
}

int launch_partition(const uint8_t* retained, const SeqInfo* seqtab, int n_heads, int n_seqs,
                     int64_t T, int64_t PT, int, int32_t* pcol, float* rcol, int32_t* prank,
                     ProblemMeta* pmeta, int32_t* status, void*) {
  ++stub::g_launches;
  touch(retained, retained ? (int64_t)n_heads * T : 0);  // null: no retained set
  touch(seqtab, (int64_t)sizeof(SeqInfo) * n_seqs);
  touch_out(pcol, 4 * (int64_t)n_heads * PT);
  touch_out(rcol, 4 * (int64_t)n_heads * PT);
  touch_out(prank, 4 * (int64_t)n_heads * PT);
  touch_out(pmeta, (int64_t)sizeof(ProblemMeta) * n_heads * n_seqs);
  touch_out(status, status ? 4 * (int64_t)n_heads * n_seqs : 0);
  return 0;
}

int prepare_tokens_per_block(int dtype, int d) { return dtype == 0 && d == 128 ? 64 : 32; }

int launch_prepare_keys(const void* keys, int dtype, int d, int n_heads, int64_t T,
                        int64_t head_stride, int64_t token_stride, int64_t PT, int, const uint8_t*,
                        const int32_t* prank, ProblemMeta* pmeta, const SeqInfo* seqtab,
                        int n_seqs, float* rinv, float* rcol, uint16_t* hilo, uint16_t* pkeys,
                        int32_t*, int, void*) {
  ++stub::g_launches;
  const int64_t esz = dtype == 1 ? 4 : 2;
  if (T > 0)
    touch(keys, esz * ((int64_t)(n_heads - 1) * head_stride + (T - 1) * token_stride + d));
  const int64_t dcol = dtype == 1 ? 2 * d : d;
  touch(prank, 4 * (int64_t)n_heads * PT);
  touch_out(pmeta, (int64_t)sizeof(ProblemMeta) * n_heads * n_seqs);
  touch(seqtab, (int64_t)sizeof(SeqInfo) * n_seqs);
  touch_out(rinv, 4 * (int64_t)n_heads * T);
  touch_out(rcol, 4 * (int64_t)n_heads * PT);
  if (dtype == 1) touch_out(hilo, 2 * (int64_t)n_heads * T * dcol);
  touch_out(pkeys, 2 * (int64_t)n_heads * PT * dcol);
  return 0;
}

int launch_prepare_keys_levels(const void* keys, int dtype, int d, int n_heads, int64_t T,
                               int64_t head_stride, int64_t token_stride, int64_t PT, int,
                               const PrepLevels& lv, const int32_t* prank, ProblemMeta* pmeta,
                               const SeqInfo* seqtab, int n_seqs, float* rinv, float* rcol,
                               uint16_t* hilo, uint16_t* pkeys, int32_t*, void*) {
  ++stub::g_launches;
  const int64_t esz = dtype == 1 ? 4 : 2;
  if (T > 0)
    touch(keys, esz * ((int64_t)(n_heads - 1) * head_stride + (T - 1) * token_stride + d));
  touch(lv.level, (int64_t)n_heads * T);
  const int64_t dcol = dtype == 1 ? 2 * d : d;
  touch(seqtab, (int64_t)sizeof(SeqInfo) * n_seqs);
  touch_out(rinv, 4 * (int64_t)n_heads * T);
  if (dtype == 1) touch_out(hilo, 2 * (int64_t)n_heads * T * dcol);
  for (int g = 0; g < lv.n_groups; ++g) {  // each group's arrays, group_stride bytes apart
    const int64_t off = (int64_t)g * lv.group_stride;
    touch(reinterpret_cast<const char*>(prank) + off, 4 * (int64_t)n_heads * PT);
    touch_out(reinterpret_cast<char*>(pmeta) + off, (int64_t)sizeof(ProblemMeta) * n_heads * n_seqs);
    touch_out(reinterpret_cast<char*>(rcol) + off, 4 * (int64_t)n_heads * PT);
    touch_out(reinterpret_cast<char*>(pkeys) + off, 2 * (int64_t)n_heads * PT * dcol);
  }
  return 0;
}

int sim_rows_per_block(int dtype, int d) {
  if (dtype == 0) return d == 128 ? 384 : 512;
  return 128;
}

int launch_sim_reduce(const SimArgs& a, int dtype, int d, void*) {
  ++stub::g_launches;
  const int64_t dcol = dtype == 1 ? 2 * d : d;
  if (a.T > 0)
    touch(a.keys, 2 * ((int64_t)(a.n_heads - 1) * a.head_stride + (a.T - 1) * a.token_stride + dcol));
  touch(a.rinv, 4 * (int64_t)a.n_heads * a.T);
  touch(a.pkeys, 2 * (int64_t)a.n_heads * a.PT * dcol);
  touch(a.pcol, 4 * (int64_t)a.n_heads * a.PT);
  touch(a.rcol, 4 * (int64_t)a.n_heads * a.PT);
  touch(a.prank, 4 * (int64_t)a.n_heads * a.PT);
  touch(a.pmeta, (int64_t)sizeof(ProblemMeta) * a.n_heads * a.n_seqs);
  touch(a.seqtab, (int64_t)sizeof(SeqInfo) * a.n_seqs);
  const int64_t nt = 4 * (int64_t)a.n_heads * a.T;
  touch_out(a.counts, a.counts ? nt : 0);
  touch_out(a.best_all, a.best_all ? nt : 0);
  touch_out(a.arg_all, a.arg_all ? nt : 0);
  touch_out(a.best_ret, a.best_ret ? nt : 0);
  touch_out(a.arg_ret, a.arg_ret ? nt : 0);
  return 0;
}

int launch_repair(const RepairArgs& a, void*) {
  ++stub::g_launches;
  const int64_t n = (int64_t)a.n_heads * a.T;
  touch(a.b, 4 * n);
  touch(a.s0, n);
  touch_out(a.s1, n);
  touch(a.seqtab, (int64_t)sizeof(SeqInfo) * a.n_seqs);
  touch(a.pmeta, a.pmeta ? (int64_t)sizeof(ProblemMeta) * a.n_heads * a.n_seqs : 0);
  touch_out(a.stats, 16 * (int64_t)a.n_heads * a.n_seqs);
  return 0;
}

int launch_evict(const EvictArgs& a, void*) {
  ++stub::g_launches;
  const int64_t n = (int64_t)a.n_heads * a.T;
  touch(a.counts, a.counts ? 4 * n : 0);
  touch(a.in_scores, a.in_scores ? 4 * n : 0);
  touch_out(a.retained, n);
  touch_out(a.scores, a.scores ? 4 * n : 0);
  touch_out(a.stats, a.stats ? 16 * (int64_t)a.n_heads * a.n_seqs : 0);
  touch(a.seqtab, (int64_t)sizeof(SeqInfo) * a.n_seqs);
  return 0;
}

int launch_prevalence(const PrevalenceArgs& a, void*) {
  ++stub::g_launches;
  touch(a.best, 4 * (int64_t)a.n_heads * a.T);
  touch_out(a.out, 4 * (int64_t)a.n_heads * a.n_seqs * a.n_taus);
  touch(a.seqtab, (int64_t)sizeof(SeqInfo) * a.n_seqs);
  return 0;
}

int launch_select_level(const uint8_t* level, uint8_t* mask, int64_t n, int, int, void*) {
  ++stub::g_launches;
  touch(level, n);
  touch_out(mask, n);
  return 0;
}

int launch_combine_levels(const CombineArgs& a, void*) {
  ++stub::g_launches;
  touch(a.gbest, 4 * a.n * a.n_groups);
  touch(a.garg, 4 * a.n * a.n_groups);
  touch_out(a.best_lvl, a.best_lvl ? 4 * a.n * a.n_levels : 0);
  touch_out(a.arg_lvl, a.arg_lvl ? 4 * a.n * a.n_levels : 0);
  touch_out(a.best_all, a.best_all ? 4 * a.n : 0);
  touch_out(a.arg_all, a.arg_all ? 4 * a.n : 0);
  return 0;
}

int launch_compact_count(const CompactArgs& a, void*) {
  ++stub::g_launches;
  touch(a.retained, (int64_t)a.n_heads * a.T);
  touch(a.seqs, (int64_t)sizeof(CompactSeq) * a.n_seqs);
  touch(a.chunk_seq, 4 * (int64_t)a.n_chunks);
  touch_out(a.chunk_cnt, 4 * (int64_t)a.n_heads * a.n_chunks);
  return 0;
}

int launch_compact_gather(const CompactArgs& a, void*) {
  ++stub::g_launches;
  if (a.T > 0) {
    touch(a.keys, (int64_t)(a.n_heads - 1) * a.head_stride + (a.T - 1) * a.token_stride + a.row_bytes);
    if (a.values)
      touch(a.values, (int64_t)(a.n_heads - 1) * a.v_head_stride + (a.T - 1) * a.v_token_stride + a.row_bytes);
  }
  const int64_t rows = (int64_t)a.n_heads * a.C;
  touch_out(a.keys_out, rows * a.row_bytes);
  touch_out(a.values_out, a.values_out ? rows * a.row_bytes : 0);
  touch_out(a.pos_out, a.pos_out ? 4 * rows : 0);
  touch_out(a.stats, 16 * (int64_t)a.n_heads * a.n_seqs);
  touch(a.chunk_cnt, 4 * (int64_t)a.n_heads * a.n_chunks);
  return 0;
}

}  // namespace twinkv
