// Host layer of the C ABI declared in include/twinkv.h: argument validation (pure host code,
// done before anything is enqueued), workspace layout, the per-sequence schedule table and
// the kernel launches (K1a partition, K1b key preparation, K2 similarity, K3 repair, K4 scorer
// eviction, policy selection and prevalence, K5 KV compaction).
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <numeric>
#include <vector>

#include "twinkv.h"
#include "twinkv_internal.h"

namespace twinkv {
namespace {

constexpr int kVersion = 100;  // 0.1.0
constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct Batch {
  int n_heads = 0, n_seqs = 0;
  int64_t T = 0, PT = 0;
};

// Shared checks of the batch description; fills `bt`.
int check_batch(int n_heads, int n_seqs, const int64_t* cu, Batch& bt) {
  if (cu == nullptr) return TWINKV_E_NULL;
  if (n_heads < 1 || n_seqs < 1) return TWINKV_E_ARG;
  if (cu[0] != 0) return TWINKV_E_ARG;
  for (int s = 0; s < n_seqs; ++s) {
    if (cu[s + 1] < cu[s]) return TWINKV_E_ARG;
  }
  const int64_t T = cu[n_seqs];
  const int64_t PT = T + (int64_t)kPermPad * n_seqs;
  // positions and per-head offsets are 32-bit inside the kernels
  if (PT > (int64_t)INT32_MAX / 2) return TWINKV_E_ARG;
  if ((int64_t)n_heads * n_seqs > (int64_t)INT32_MAX / 4) return TWINKV_E_ARG;
  bt.n_heads = n_heads;
  bt.n_seqs = n_seqs;
  bt.T = T;
  bt.PT = PT;
  return TWINKV_OK;
}

// Chunks of the compaction's chunk list: ceil(len / kCompactChunk), at least 1 per sequence.
int64_t compact_chunks(const int64_t* cu, int n_seqs) {
  int64_t n = 0;
  for (int s = 0; s < n_seqs; ++s)
    n += std::max<int64_t>(1, (cu[s + 1] - cu[s] + kCompactChunk - 1) / kCompactChunk);
  return n;
}

Layout layout_for(int op, int dtype, int d, const Batch& bt, const int64_t* cu = nullptr) {
  Layout L;
  size_t off = 0;
  if (op == TWINKV_OP_COMPACT) {
    const int64_t nch = compact_chunks(cu, bt.n_seqs);
    L.seqtab = off;
    off = align_up(off + sizeof(CompactSeq) * (size_t)bt.n_seqs);
    L.chunk_seq = off;
    off = align_up(off + 4 * (size_t)nch);
    L.chunk_cnt = off;
    off = align_up(off + 4 * (size_t)nch * (size_t)bt.n_heads);
    L.total = off + kAlign;
    return L;
  }
  L.seqtab = off;
  off = align_up(off + sizeof(SeqInfo) * (size_t)bt.n_seqs);
  if (op != TWINKV_OP_REPAIR_FROM_SCORES) {
    const size_t nt = (size_t)bt.n_heads * (size_t)bt.T;
    const size_t np = (size_t)bt.n_heads * (size_t)bt.PT;
    L.rinv = off;
    off = align_up(off + 4 * nt);
    L.pcol = off;
    off = align_up(off + 4 * np);
    L.rcol = off;
    off = align_up(off + 4 * np);
    L.prank = off;
    off = align_up(off + 4 * np);
    L.pmeta = off;
    off = align_up(off + sizeof(ProblemMeta) * (size_t)bt.n_heads * bt.n_seqs);
    const size_t dcol = dtype == TWINKV_F32 ? (size_t)(2 * d) : (size_t)d;
    if (dtype == TWINKV_F32) {
      L.hilo = off;
      off = align_up(off + 2 * nt * dcol);
    }
    L.pkeys = off;
    off = align_up(off + 2 * np * dcol);
    if (op == TWINKV_OP_REPAIR || op == TWINKV_OP_SCORE_EVICT) {
      L.bbuf = off;  // b for the repair pass, the twin counts for the scorer
      off = align_up(off + 4 * nt);
    }
  }
  L.total = off + kAlign;  // slack for aligning the caller's base pointer
  return L;
}

char* aligned_base(void* ws) {
  const uintptr_t p = reinterpret_cast<uintptr_t>(ws);
  return reinterpret_cast<char*>((p + kAlign - 1) / kAlign * kAlign);
}

int check_keys(const void* keys, int dtype, int d, int64_t head_stride, int64_t token_stride,
               int w) {
  if (dtype != TWINKV_BF16 && dtype != TWINKV_F32) return TWINKV_E_UNSUPPORTED;
  if (d != 64 && d != 128) return TWINKV_E_UNSUPPORTED;
  if (keys == nullptr) return TWINKV_E_NULL;
  const int64_t esz = dtype == TWINKV_F32 ? 4 : 2;
  if (token_stride < d || head_stride < 0) return TWINKV_E_ARG;
  if ((reinterpret_cast<uintptr_t>(keys) % 16) != 0) return TWINKV_E_ARG;
  if ((token_stride * esz) % 16 != 0 || (head_stride * esz) % 16 != 0) return TWINKV_E_ARG;
  if (w < 0) return TWINKV_E_ARG;
  return TWINKV_OK;
}

// Builds the per-sequence table (schedule of similarity row blocks, longest first).
std::vector<SeqInfo> seq_table(const int64_t* cu, int n_seqs, const int64_t* budget, int rows_per_block,
                               int& total_tiles, int prep_tokens = 0, int64_t* prep_blocks = nullptr) {
  std::vector<SeqInfo> tab(n_seqs);
  int64_t pb = 0;
  for (int s = 0; s < n_seqs; ++s) {
    tab[s].start = (int32_t)cu[s];
    tab[s].len = (int32_t)(cu[s + 1] - cu[s]);
    tab[s].budget = budget ? (int32_t)budget[s] : -1;
    tab[s].perm_off = (int32_t)(cu[s] + (int64_t)kPermPad * s);
    tab[s].prep_blk0 = (int32_t)pb;
    if (prep_tokens > 0) pb += (tab[s].len + prep_tokens - 1) / prep_tokens;
  }
  if (prep_blocks) *prep_blocks = pb;
  std::vector<int> order(n_seqs);
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(),
                   [&](int x, int y) { return tab[x].len > tab[y].len; });
  int cum = 0;
  for (int r = 0; r < n_seqs; ++r) {
    const int s = order[r];
    const int nb = rows_per_block > 0 ? (tab[s].len + rows_per_block - 1) / rows_per_block : 0;
    tab[r].sorted_seq = s;
    tab[r].tile_cum = cum;
    tab[r].nb = nb;
    cum += nb;
  }
  total_tiles = cum;
  return tab;
}

int hip_status(int e) { return e == 0 ? TWINKV_OK : TWINKV_E_HIP; }

int max_seq_len(const int64_t* cu, int n_seqs) {
  int64_t m = 0;
  for (int s = 0; s < n_seqs; ++s) m = std::max<int64_t>(m, cu[s + 1] - cu[s]);
  return (int)m;
}

int check_repair_common(const uint8_t* retained_in, uint8_t* retained_out,
                               const int64_t* budget, const int64_t* cu, int n_seqs, float tau,
                               int n_sink, int n_recent, int32_t* stats) {
  if (retained_in == nullptr || retained_out == nullptr || budget == nullptr || stats == nullptr)
    return TWINKV_E_NULL;
  if (!std::isfinite(tau)) return TWINKV_E_ARG;
  if (n_sink < 0 || n_recent < 0) return TWINKV_E_ARG;
  for (int s = 0; s < n_seqs; ++s) {
    if (budget[s] < 0 || budget[s] > cu[s + 1] - cu[s]) return TWINKV_E_ARG;
  }
  return TWINKV_OK;
}

// Events recorded around the similarity kernel, or the compaction's gather kernel
// (twinkv_profile_sim_events), per thread.
thread_local hipEvent_t g_sim_start = nullptr;
thread_local hipEvent_t g_sim_stop = nullptr;

// K1a + K1b: the sequence table, the column partition and the prepared keys, ready for K2.
struct Prepared {
  SimArgs args;         // everything but the outputs, w, want_all and the count mode
  SeqInfo* seqtab = nullptr;
  int prep_blocks = 0;  // K1b workgroups per head
};

// K1a, K1b (unless key_prep is false: the level groups run one K1b for all their column
// lists) and the similarity kernel's arguments for one column split.
int prepare_scores(const void* keys, int dtype, int d, const Batch& bt, const int64_t* cu,
                   const int64_t* budget, int64_t head_stride, int64_t token_stride,
                   const uint8_t* retained, int32_t* status, char* ws, const Layout& L,
                   bool copy_evicted, void* stream, Prepared& P, bool key_prep = true) {
  int total_tiles = 0;
  const int rpb = sim_rows_per_block(dtype, d);
  int64_t prep_blocks = 0;
  std::vector<SeqInfo> tab = seq_table(cu, bt.n_seqs, budget, rpb, total_tiles,
                                       prepare_tokens_per_block(dtype, d), &prep_blocks);
  if (prep_blocks > (int64_t)INT32_MAX) return TWINKV_E_ARG;
  P.prep_blocks = (int)prep_blocks;
  const int64_t groups = bt.n_heads >= 8 ? 8LL * ((bt.n_heads + 7) / 8) : bt.n_heads;
  if (groups * total_tiles > (int64_t)INT32_MAX) return TWINKV_E_ARG;

  SeqInfo* dtab = reinterpret_cast<SeqInfo*>(ws + L.seqtab);
  P.seqtab = dtab;
  if (launch_upload(tab.data(), sizeof(SeqInfo) * tab.size(), dtab, stream) != 0)
    return TWINKV_E_HIP;

  float* rinv = reinterpret_cast<float*>(ws + L.rinv);
  int32_t* pcol = reinterpret_cast<int32_t*>(ws + L.pcol);
  float* rcol = reinterpret_cast<float*>(ws + L.rcol);
  int32_t* prank = reinterpret_cast<int32_t*>(ws + L.prank);
  ProblemMeta* pmeta = reinterpret_cast<ProblemMeta*>(ws + L.pmeta);
  uint16_t* hilo = dtype == TWINKV_F32 ? reinterpret_cast<uint16_t*>(ws + L.hilo) : nullptr;
  uint16_t* pkeys = reinterpret_cast<uint16_t*>(ws + L.pkeys);

  int e = launch_partition(retained, dtab, bt.n_heads, bt.n_seqs, bt.T, bt.PT,
                           max_seq_len(cu, bt.n_seqs), pcol, rcol, prank, pmeta, status, stream);
  if (e) return hip_status(e);
  if (key_prep) {
    e = launch_prepare_keys(keys, dtype, d, bt.n_heads, bt.T, head_stride, token_stride, bt.PT,
                            (int)prep_blocks, retained, prank, pmeta, dtab, bt.n_seqs, rinv, rcol,
                            hilo, pkeys, status, copy_evicted ? 1 : 0, stream);
    if (e) return hip_status(e);
  }

  SimArgs& a = P.args;
  if (dtype == TWINKV_F32) {
    a.keys = hilo;
    a.head_stride = bt.T * 2 * d;
    a.token_stride = 2 * d;
  } else {
    a.keys = keys;
    a.head_stride = head_stride;
    a.token_stride = token_stride;
  }
  a.rinv = rinv;
  a.pkeys = pkeys;
  a.pcol = pcol;
  a.rcol = rcol;
  a.prank = prank;
  a.pmeta = pmeta;
  a.seqtab = dtab;
  a.n_heads = bt.n_heads;
  a.n_seqs = bt.n_seqs;
  a.T = bt.T;
  a.PT = bt.PT;
  a.total_tiles = total_tiles;
  a.w = 0;
  a.want_all = 0;
  a.tau = 0.0f;
  a.counts = nullptr;
  a.best_all = nullptr;
  a.arg_all = nullptr;
  a.best_ret = nullptr;
  a.arg_ret = nullptr;
  return TWINKV_OK;
}

// K2 on prepared keys.
int sim_scores(const Batch& bt, int dtype, int d, int w, bool want_all, float* best_all,
               int32_t* arg_all, float* best_ret, int32_t* arg_ret, float tau, int32_t* counts,
               Prepared& P, void* stream) {
  SimArgs a = P.args;
  // |i - j| <= T - 1 inside any sequence, so any w >= T behaves like w = T.
  a.w = (int)std::min<int64_t>(w, std::max<int64_t>(bt.T, 1));
  a.want_all = want_all ? 1 : 0;
  a.tau = tau;
  a.counts = counts;
  a.best_all = best_all;
  a.arg_all = arg_all;
  a.best_ret = best_ret;
  a.arg_ret = arg_ret;
  return hip_status(launch_sim_reduce(a, dtype, d, stream));
}

int record(hipEvent_t ev, void* stream) {
  return (ev && hipEventRecord(ev, (hipStream_t)stream) != hipSuccess) ? TWINKV_E_HIP : TWINKV_OK;
}

// K1a + K1b + K2 (shared by nn_scores, repair and the scorer).
int run_scores(const void* keys, int dtype, int d, const Batch& bt, const int64_t* cu,
               const int64_t* budget, int64_t head_stride, int64_t token_stride,
               const uint8_t* retained, int w, float* best_all, int32_t* arg_all,
               float* best_ret, int32_t* arg_ret, int32_t* status, char* ws, const Layout& L,
               bool want_all, void* stream, SeqInfo** seqtab_dev, float tau = 0.0f,
               int32_t* counts = nullptr) {
  Prepared P;
  int rc = prepare_scores(keys, dtype, d, bt, cu, budget, head_stride, token_stride, retained,
                          status, ws, L, want_all, stream, P);
  if (rc != TWINKV_OK) return rc;
  *seqtab_dev = P.seqtab;
  if ((rc = record(g_sim_start, stream)) != TWINKV_OK) return rc;
  rc = sim_scores(bt, dtype, d, w, want_all, best_all, arg_all, best_ret, arg_ret, tau, counts, P,
                  stream);
  if (rc != TWINKV_OK) return rc;
  return record(g_sim_stop, stream);
}

}  // namespace

int repair_from_scores_into(const float* b, const uint8_t* retained_in, uint8_t* retained_out,
                            int n_heads, int n_seqs, const int64_t* cu_seqlens,
                            const int64_t* budget, float tau, int n_sink, int n_recent,
                            int32_t* stats, void* table, size_t table_bytes,
                            void* (*resolve_table)(), void* stream) {
  if (b == nullptr) return TWINKV_E_NULL;
  Batch bt;
  int rc = check_batch(n_heads, n_seqs, cu_seqlens, bt);
  if (rc != TWINKV_OK) return rc;
  rc = check_repair_common(retained_in, retained_out, budget, cu_seqlens, n_seqs, tau, n_sink,
                           n_recent, stats);
  if (rc != TWINKV_OK) return rc;
  if (sizeof(SeqInfo) * (size_t)n_seqs > table_bytes) return TWINKV_E_CAPACITY;
  if (resolve_table != nullptr && (table = resolve_table()) == nullptr) return TWINKV_E_HIP;
  int tiles = 0;
  std::vector<SeqInfo> tab = seq_table(cu_seqlens, n_seqs, budget, 0, tiles);
  SeqInfo* dtab = reinterpret_cast<SeqInfo*>(table);
  if (launch_upload(tab.data(), sizeof(SeqInfo) * tab.size(), dtab, stream) != 0)
    return TWINKV_E_HIP;
  RepairArgs ra;
  ra.b = b;
  ra.s0 = retained_in;
  ra.s1 = retained_out;
  ra.seqtab = dtab;
  ra.pmeta = nullptr;
  ra.n_heads = n_heads;
  ra.n_seqs = n_seqs;
  ra.T = bt.T;
  ra.tau = tau;
  ra.n_sink = n_sink;
  ra.n_recent = n_recent;
  ra.stats = stats;
  ra.max_len = max_seq_len(cu_seqlens, n_seqs);
  return hip_status(launch_repair(ra, stream));
}

}  // namespace twinkv

using namespace twinkv;

extern "C" {

int64_t twinkv_workspace_bytes(int op, int dtype, int d, int n_heads, int n_seqs,
                               const int64_t* cu_seqlens) {
  if (op != TWINKV_OP_NN_SCORES && op != TWINKV_OP_REPAIR && op != TWINKV_OP_REPAIR_FROM_SCORES &&
      op != TWINKV_OP_TWIN_COUNTS && op != TWINKV_OP_SCORE_EVICT && op != TWINKV_OP_COMPACT)
    return -TWINKV_E_ARG;
  if (op != TWINKV_OP_REPAIR_FROM_SCORES && op != TWINKV_OP_COMPACT) {
    if (dtype != TWINKV_BF16 && dtype != TWINKV_F32) return -TWINKV_E_UNSUPPORTED;
    if (d != 64 && d != 128) return -TWINKV_E_UNSUPPORTED;
  }
  Batch bt;
  const int rc = check_batch(n_heads, n_seqs, cu_seqlens, bt);
  if (rc != TWINKV_OK) return -rc;
  return (int64_t)layout_for(op, dtype, d, bt, cu_seqlens).total;
}

int twinkv_nn_scores(const void* keys, int dtype, int d, int n_heads, int n_seqs,
                     const int64_t* cu_seqlens, int64_t head_stride, int64_t token_stride,
                     const uint8_t* retained, int w, float* best_all, int32_t* arg_all,
                     float* best_ret, int32_t* arg_ret, int32_t* status, void* workspace,
                     int64_t workspace_bytes, void* stream) {
  int rc = check_keys(keys, dtype, d, head_stride, token_stride, w);
  if (rc != TWINKV_OK) return rc;
  Batch bt;
  rc = check_batch(n_heads, n_seqs, cu_seqlens, bt);
  if (rc != TWINKV_OK) return rc;
  if (retained == nullptr && (best_ret != nullptr || arg_ret != nullptr)) return TWINKV_E_ARG;
  const Layout L = layout_for(TWINKV_OP_NN_SCORES, dtype, d, bt);
  if (workspace == nullptr || workspace_bytes < (int64_t)L.total) return TWINKV_E_WORKSPACE;
  char* ws = aligned_base(workspace);
  SeqInfo* dtab = nullptr;
  return run_scores(keys, dtype, d, bt, cu_seqlens, nullptr, head_stride, token_stride, retained,
                    w, best_all, arg_all, best_ret, arg_ret, status, ws, L,
                    /*want_all=*/true, stream, &dtab);
}


int twinkv_repair(const void* keys, int dtype, int d, int n_heads, int n_seqs,
                  const int64_t* cu_seqlens, int64_t head_stride, int64_t token_stride,
                  const uint8_t* retained_in, uint8_t* retained_out, const int64_t* budget,
                  float tau, int w, int n_sink, int n_recent, int32_t* stats, float* best_all,
                  int32_t* arg_all, float* best_ret, int32_t* arg_ret, void* workspace,
                  int64_t workspace_bytes, void* stream) {
  int rc = check_keys(keys, dtype, d, head_stride, token_stride, w);
  if (rc != TWINKV_OK) return rc;
  Batch bt;
  rc = check_batch(n_heads, n_seqs, cu_seqlens, bt);
  if (rc != TWINKV_OK) return rc;
  rc = check_repair_common(retained_in, retained_out, budget, cu_seqlens, n_seqs, tau, n_sink,
                           n_recent, stats);
  if (rc != TWINKV_OK) return rc;
  const Layout L = layout_for(TWINKV_OP_REPAIR, dtype, d, bt);
  if (workspace == nullptr || workspace_bytes < (int64_t)L.total) return TWINKV_E_WORKSPACE;
  char* ws = aligned_base(workspace);
  float* b = best_ret ? best_ret : reinterpret_cast<float*>(ws + L.bbuf);
  const bool want_all = best_all != nullptr || arg_all != nullptr;
  SeqInfo* dtab = nullptr;
  rc = run_scores(keys, dtype, d, bt, cu_seqlens, budget, head_stride, token_stride, retained_in,
                  w, best_all, arg_all, b, arg_ret, nullptr, ws, L, want_all, stream, &dtab);
  if (rc != TWINKV_OK) return rc;
  RepairArgs ra;
  ra.b = b;
  ra.s0 = retained_in;
  ra.s1 = retained_out;
  ra.seqtab = dtab;
  ra.pmeta = reinterpret_cast<const ProblemMeta*>(ws + L.pmeta);
  ra.n_heads = n_heads;
  ra.n_seqs = n_seqs;
  ra.T = bt.T;
  ra.tau = tau;
  ra.n_sink = n_sink;
  ra.n_recent = n_recent;
  ra.stats = stats;
  ra.max_len = max_seq_len(cu_seqlens, n_seqs);
  return hip_status(launch_repair(ra, stream));
}

int twinkv_repair_from_scores(const float* b, const uint8_t* retained_in, uint8_t* retained_out,
                              int n_heads, int n_seqs, const int64_t* cu_seqlens,
                              const int64_t* budget, float tau, int n_sink, int n_recent,
                              int32_t* stats, void* workspace, int64_t workspace_bytes,
                              void* stream) {
  Batch bt;
  int rc = check_batch(n_heads, n_seqs, cu_seqlens, bt);
  if (rc != TWINKV_OK) return rc;
  const Layout L = layout_for(TWINKV_OP_REPAIR_FROM_SCORES, 0, 64, bt);
  if (workspace == nullptr || workspace_bytes < (int64_t)L.total) return TWINKV_E_WORKSPACE;
  return twinkv::repair_from_scores_into(b, retained_in, retained_out, n_heads, n_seqs,
                                         cu_seqlens, budget, tau, n_sink, n_recent, stats,
                                         aligned_base(workspace) + L.seqtab,
                                         L.total - kAlign, nullptr, stream);
}

int twinkv_twin_counts(const void* keys, int dtype, int d, int n_heads, int n_seqs,
                       const int64_t* cu_seqlens, int64_t head_stride, int64_t token_stride,
                       float tau, int w, int32_t* counts, int32_t* status, void* workspace,
                       int64_t workspace_bytes, void* stream) {
  int rc = check_keys(keys, dtype, d, head_stride, token_stride, w);
  if (rc != TWINKV_OK) return rc;
  Batch bt;
  rc = check_batch(n_heads, n_seqs, cu_seqlens, bt);
  if (rc != TWINKV_OK) return rc;
  if (counts == nullptr) return TWINKV_E_NULL;
  if (!std::isfinite(tau)) return TWINKV_E_ARG;
  const Layout L = layout_for(TWINKV_OP_TWIN_COUNTS, dtype, d, bt);
  if (workspace == nullptr || workspace_bytes < (int64_t)L.total) return TWINKV_E_WORKSPACE;
  char* ws = aligned_base(workspace);
  SeqInfo* dtab = nullptr;
  // every column is an "evicted" column (no retained set): one all-keys sweep that counts
  return run_scores(keys, dtype, d, bt, cu_seqlens, nullptr, head_stride, token_stride, nullptr,
                    w, nullptr, nullptr, nullptr, nullptr, status, ws, L, /*want_all=*/true,
                    stream, &dtab, tau, counts);
}

int twinkv_score_evict(const void* keys, int dtype, int d, int n_heads, int n_seqs,
                       const int64_t* cu_seqlens, int64_t head_stride, int64_t token_stride,
                       const int64_t* budget, float tau, int w, int n_sink, int n_recent,
                       uint8_t* retained_out, int32_t* counts, float* scores, int32_t* stats,
                       void* workspace, int64_t workspace_bytes, void* stream) {
  int rc = check_keys(keys, dtype, d, head_stride, token_stride, w);
  if (rc != TWINKV_OK) return rc;
  Batch bt;
  rc = check_batch(n_heads, n_seqs, cu_seqlens, bt);
  if (rc != TWINKV_OK) return rc;
  if (retained_out == nullptr || budget == nullptr || stats == nullptr) return TWINKV_E_NULL;
  if (!std::isfinite(tau) || n_sink < 0 || n_recent < 0) return TWINKV_E_ARG;
  for (int s = 0; s < n_seqs; ++s) {
    if (budget[s] < 0 || budget[s] > INT32_MAX) return TWINKV_E_ARG;
  }
  const Layout L = layout_for(TWINKV_OP_SCORE_EVICT, dtype, d, bt);
  if (workspace == nullptr || workspace_bytes < (int64_t)L.total) return TWINKV_E_WORKSPACE;
  char* ws = aligned_base(workspace);
  int32_t* c = counts ? counts : reinterpret_cast<int32_t*>(ws + L.bbuf);
  SeqInfo* dtab = nullptr;
  rc = run_scores(keys, dtype, d, bt, cu_seqlens, budget, head_stride, token_stride, nullptr, w,
                  nullptr, nullptr, nullptr, nullptr, nullptr, ws, L, /*want_all=*/true, stream,
                  &dtab, tau, c);
  if (rc != TWINKV_OK) return rc;
  EvictArgs ea;
  ea.counts = c;
  ea.in_scores = nullptr;
  ea.retained = retained_out;
  ea.scores = scores;
  ea.stats = stats;
  ea.seqtab = dtab;
  ea.pmeta = reinterpret_cast<const ProblemMeta*>(ws + L.pmeta);
  ea.n_heads = n_heads;
  ea.n_seqs = n_seqs;
  ea.T = bt.T;
  ea.n_sink = n_sink;
  ea.n_recent = n_recent;
  ea.max_len = max_seq_len(cu_seqlens, n_seqs);
  return hip_status(launch_evict(ea, stream));
}

int twinkv_select_topk(const float* scores, int n_heads, int n_seqs, const int64_t* cu_seqlens,
                       const int64_t* budget, int n_sink, int n_recent, uint8_t* retained_out,
                       int32_t* stats, void* workspace, int64_t workspace_bytes, void* stream) {
  if (scores == nullptr || budget == nullptr || retained_out == nullptr) return TWINKV_E_NULL;
  if (n_sink < 0 || n_recent < 0) return TWINKV_E_ARG;
  Batch bt;
  int rc = check_batch(n_heads, n_seqs, cu_seqlens, bt);
  if (rc != TWINKV_OK) return rc;
  for (int s = 0; s < n_seqs; ++s) {
    if (budget[s] < 0 || budget[s] > INT32_MAX) return TWINKV_E_ARG;
  }
  const Layout L = layout_for(TWINKV_OP_REPAIR_FROM_SCORES, 0, 64, bt);
  if (workspace == nullptr || workspace_bytes < (int64_t)L.total) return TWINKV_E_WORKSPACE;
  char* ws = aligned_base(workspace);
  int tiles = 0;
  std::vector<SeqInfo> tab = seq_table(cu_seqlens, n_seqs, budget, 0, tiles);
  SeqInfo* dtab = reinterpret_cast<SeqInfo*>(ws + L.seqtab);
  if (launch_upload(tab.data(), sizeof(SeqInfo) * tab.size(), dtab, stream) != 0)
    return TWINKV_E_HIP;
  EvictArgs ea;
  ea.counts = nullptr;
  ea.in_scores = scores;
  ea.retained = retained_out;
  ea.scores = nullptr;
  ea.stats = stats;
  ea.seqtab = dtab;
  ea.pmeta = nullptr;
  ea.n_heads = n_heads;
  ea.n_seqs = n_seqs;
  ea.T = bt.T;
  ea.n_sink = n_sink;
  ea.n_recent = n_recent;
  ea.max_len = max_seq_len(cu_seqlens, n_seqs);
  return hip_status(launch_evict(ea, stream));
}

int twinkv_prevalence(const float* best_all, int n_heads, int n_seqs, const int64_t* cu_seqlens,
                      const float* taus, int n_taus, int32_t* out, void* workspace,
                      int64_t workspace_bytes, void* stream) {
  if (best_all == nullptr || taus == nullptr || out == nullptr) return TWINKV_E_NULL;
  if (n_taus < 1 || n_taus > kMaxTaus) return TWINKV_E_ARG;
  Batch bt;
  int rc = check_batch(n_heads, n_seqs, cu_seqlens, bt);
  if (rc != TWINKV_OK) return rc;
  const Layout L = layout_for(TWINKV_OP_REPAIR_FROM_SCORES, 0, 64, bt);
  if (workspace == nullptr || workspace_bytes < (int64_t)L.total) return TWINKV_E_WORKSPACE;
  char* ws = aligned_base(workspace);
  int tiles = 0;
  std::vector<SeqInfo> tab = seq_table(cu_seqlens, n_seqs, nullptr, 0, tiles);
  SeqInfo* dtab = reinterpret_cast<SeqInfo*>(ws + L.seqtab);
  if (launch_upload(tab.data(), sizeof(SeqInfo) * tab.size(), dtab, stream) != 0)
    return TWINKV_E_HIP;
  PrevalenceArgs pa;
  pa.best = best_all;
  pa.out = out;
  pa.seqtab = dtab;
  pa.n_heads = n_heads;
  pa.n_seqs = n_seqs;
  pa.T = bt.T;
  pa.n_taus = n_taus;
  for (int k = 0; k < kMaxTaus; ++k) pa.taus[k] = k < n_taus ? taus[k] : 0.0f;
  return hip_status(launch_prevalence(pa, stream));
}

// Nested sets: one sub-workspace per level group (partition and prepared keys), the group
// mask, and the per-group maxima.
struct LevelsLayout {
  size_t per = 0, mask = 0, gbest = 0, garg = 0, total = 0;
  int groups = 0;
};

LevelsLayout levels_layout(int dtype, int d, const Batch& bt, int n_levels, bool want_all) {
  LevelsLayout LL;
  LL.groups = n_levels + (want_all ? 1 : 0);
  LL.per = align_up(layout_for(TWINKV_OP_NN_SCORES, dtype, d, bt).total);
  const size_t n = (size_t)bt.n_heads * (size_t)bt.T;
  size_t off = LL.per * (size_t)LL.groups;
  LL.mask = off;
  off = align_up(off + n);
  LL.gbest = off;
  off = align_up(off + 4 * n * (size_t)LL.groups);
  LL.garg = off;
  off = align_up(off + 4 * n * (size_t)LL.groups);
  LL.total = off + kAlign;
  return LL;
}

int64_t twinkv_levels_workspace_bytes(int dtype, int d, int n_heads, int n_seqs,
                                      const int64_t* cu_seqlens, int n_levels, int want_all) {
  if (dtype != TWINKV_BF16 && dtype != TWINKV_F32) return -TWINKV_E_UNSUPPORTED;
  if (d != 64 && d != 128) return -TWINKV_E_UNSUPPORTED;
  if (n_levels < 1 || n_levels > kMaxLevels) return -TWINKV_E_ARG;
  Batch bt;
  const int rc = check_batch(n_heads, n_seqs, cu_seqlens, bt);
  if (rc != TWINKV_OK) return -rc;
  return (int64_t)levels_layout(dtype, d, bt, n_levels, want_all != 0).total;
}

int twinkv_nn_scores_levels(const void* keys, int dtype, int d, int n_heads, int n_seqs,
                            const int64_t* cu_seqlens, int64_t head_stride, int64_t token_stride,
                            const uint8_t* level, int n_levels, int w, float* best_all,
                            int32_t* arg_all, float* best_lvl, int32_t* arg_lvl, int32_t* status,
                            void* workspace, int64_t workspace_bytes, void* stream) {
  int rc = check_keys(keys, dtype, d, head_stride, token_stride, w);
  if (rc != TWINKV_OK) return rc;
  if (level == nullptr || best_lvl == nullptr) return TWINKV_E_NULL;
  if (n_levels < 1 || n_levels > kMaxLevels) return TWINKV_E_ARG;
  Batch bt;
  rc = check_batch(n_heads, n_seqs, cu_seqlens, bt);
  if (rc != TWINKV_OK) return rc;
  const bool want_all = best_all != nullptr || arg_all != nullptr;
  const LevelsLayout LL = levels_layout(dtype, d, bt, n_levels, want_all);
  if (workspace == nullptr || workspace_bytes < (int64_t)LL.total) return TWINKV_E_WORKSPACE;
  char* base = aligned_base(workspace);
  const Layout L = layout_for(TWINKV_OP_NN_SCORES, dtype, d, bt);
  const int64_t n = (int64_t)n_heads * bt.T;
  uint8_t* mask = reinterpret_cast<uint8_t*>(base + LL.mask);
  float* gbest = reinterpret_cast<float*>(base + LL.gbest);
  int32_t* garg = reinterpret_cast<int32_t*>(base + LL.garg);

  // every group's partition, then one key preparation for all groups (the keys are read
  // once; each goes to its own group's column list), then the similarity sweeps back to back
  Prepared P[kMaxLevels + 1];
  for (int g = 0; g < LL.groups; ++g) {
    const int sel = g < n_levels ? g + 1 : 0;  // the last group: the tokens in no set
    if (launch_select_level(level, mask, n, sel, n_levels, stream) != 0) return TWINKV_E_HIP;
    rc = prepare_scores(keys, dtype, d, bt, cu_seqlens, nullptr, head_stride, token_stride, mask,
                        g == 0 ? status : nullptr, base + LL.per * (size_t)g, L,
                        /*copy_evicted=*/false, stream, P[g], /*key_prep=*/false);
    if (rc != TWINKV_OK) return rc;
  }
  {
    // group 0's arrays; group g's lie g * LL.per bytes further, at the same layout offsets
    const PrepLevels lv{level, n_levels, LL.groups, (int64_t)LL.per};
    const int e = launch_prepare_keys_levels(
        keys, dtype, d, n_heads, bt.T, head_stride, token_stride, bt.PT, P[0].prep_blocks, lv,
        reinterpret_cast<const int32_t*>(base + L.prank),
        reinterpret_cast<ProblemMeta*>(base + L.pmeta), P[0].seqtab, n_seqs,
        reinterpret_cast<float*>(base + L.rinv), reinterpret_cast<float*>(base + L.rcol),
        dtype == TWINKV_F32 ? reinterpret_cast<uint16_t*>(base + L.hilo) : nullptr,
        reinterpret_cast<uint16_t*>(base + L.pkeys), status, stream);
    if (e) return hip_status(e);
    // the rows' inverse norms (and the fp32 row plane) exist once, in group 0's slice
    for (int g = 1; g < LL.groups; ++g) {
      P[g].args.rinv = P[0].args.rinv;
      if (dtype == TWINKV_F32) P[g].args.keys = P[0].args.keys;
    }
  }
  if ((rc = record(g_sim_start, stream)) != TWINKV_OK) return rc;
  for (int g = 0; g < LL.groups; ++g) {
    rc = sim_scores(bt, dtype, d, w, /*want_all=*/false, nullptr, nullptr, gbest + g * n,
                    garg + g * n, 0.0f, nullptr, P[g], stream);
    if (rc != TWINKV_OK) return rc;
  }
  if ((rc = record(g_sim_stop, stream)) != TWINKV_OK) return rc;
  CombineArgs ca;
  ca.gbest = gbest;
  ca.garg = garg;
  ca.n_groups = LL.groups;
  ca.n_levels = n_levels;
  ca.n = n;
  ca.best_lvl = best_lvl;
  ca.arg_lvl = arg_lvl;
  ca.best_all = best_all;
  ca.arg_all = arg_all;
  return hip_status(launch_combine_levels(ca, stream));
}

int twinkv_compact(const void* keys, const void* values, int dtype, int d, int n_heads,
                   int n_seqs, const int64_t* cu_seqlens, int64_t head_stride,
                   int64_t token_stride, int64_t v_head_stride, int64_t v_token_stride,
                   const uint8_t* retained, const int64_t* capacity, void* keys_out,
                   void* values_out, int32_t* pos_out, int32_t* stats, void* workspace,
                   int64_t workspace_bytes, void* stream) {
  int rc = check_keys(keys, dtype, d, head_stride, token_stride, 0);
  if (rc != TWINKV_OK) return rc;
  if (retained == nullptr || capacity == nullptr || keys_out == nullptr || stats == nullptr)
    return TWINKV_E_NULL;
  if ((values == nullptr) != (values_out == nullptr)) return TWINKV_E_NULL;
  if (values != nullptr) {
    rc = check_keys(values, dtype, d, v_head_stride, v_token_stride, 0);
    if (rc != TWINKV_OK) return rc;
  }
  if (reinterpret_cast<uintptr_t>(keys_out) % 16 != 0 ||
      reinterpret_cast<uintptr_t>(values_out) % 16 != 0)
    return TWINKV_E_ARG;
  Batch bt;
  rc = check_batch(n_heads, n_seqs, cu_seqlens, bt);
  if (rc != TWINKV_OK) return rc;
  int64_t C = 0;
  for (int s = 0; s < n_seqs; ++s) {
    if (capacity[s] < 0 || capacity[s] > cu_seqlens[s + 1] - cu_seqlens[s]) return TWINKV_E_ARG;
    C += capacity[s];
  }
  const int64_t nch = compact_chunks(cu_seqlens, n_seqs);
  if ((int64_t)n_heads * nch > (int64_t)INT32_MAX) return TWINKV_E_ARG;
  const Layout L = layout_for(TWINKV_OP_COMPACT, dtype, d, bt, cu_seqlens);
  if (workspace == nullptr || workspace_bytes < (int64_t)L.total) return TWINKV_E_WORKSPACE;
  char* ws = aligned_base(workspace);

  // sequence table and chunk list, one host-to-device copy
  const size_t tab_bytes = L.chunk_cnt - L.seqtab;
  std::vector<char> host(tab_bytes, 0);
  CompactSeq* tab = reinterpret_cast<CompactSeq*>(host.data());
  int32_t* cseq = reinterpret_cast<int32_t*>(host.data() + (L.chunk_seq - L.seqtab));
  int64_t out = 0, ck = 0;
  for (int s = 0; s < n_seqs; ++s) {
    const int64_t len = cu_seqlens[s + 1] - cu_seqlens[s];
    const int64_t nc = std::max<int64_t>(1, (len + kCompactChunk - 1) / kCompactChunk);
    tab[s].start = (int32_t)cu_seqlens[s];
    tab[s].len = (int32_t)len;
    tab[s].cap = (int32_t)capacity[s];
    tab[s].out_start = (int32_t)out;
    tab[s].chunk0 = (int32_t)ck;
    tab[s].nchunks = (int32_t)nc;
    for (int64_t c = 0; c < nc; ++c) cseq[ck + c] = s;
    out += capacity[s];
    ck += nc;
  }
  if (launch_upload(host.data(), tab_bytes, ws + L.seqtab, stream) != 0) return TWINKV_E_HIP;

  const int64_t esz = dtype == TWINKV_F32 ? 4 : 2;
  CompactArgs a;
  a.keys = static_cast<const char*>(keys);
  a.values = static_cast<const char*>(values);
  a.head_stride = head_stride * esz;
  a.token_stride = token_stride * esz;
  a.v_head_stride = v_head_stride * esz;
  a.v_token_stride = v_token_stride * esz;
  a.row_bytes = (int)(d * esz);
  int lp = 0;
  while ((16 << lp) < a.row_bytes) ++lp;
  a.log2_pieces = lp;
  a.retained = retained;
  a.seqs = reinterpret_cast<const CompactSeq*>(ws + L.seqtab);
  a.chunk_seq = reinterpret_cast<const int32_t*>(ws + L.chunk_seq);
  a.chunk_cnt = reinterpret_cast<int32_t*>(ws + L.chunk_cnt);
  a.keys_out = static_cast<char*>(keys_out);
  a.values_out = static_cast<char*>(values_out);
  a.pos_out = pos_out;
  a.stats = stats;
  a.n_heads = n_heads;
  a.n_seqs = n_seqs;
  a.n_chunks = (int)nch;
  a.T = bt.T;
  a.C = C;
  int e = launch_compact_count(a, stream);
  if (e) return hip_status(e);
  if (g_sim_start && hipEventRecord(g_sim_start, (hipStream_t)stream) != hipSuccess) return TWINKV_E_HIP;
  e = launch_compact_gather(a, stream);
  if (e) return hip_status(e);
  if (g_sim_stop && hipEventRecord(g_sim_stop, (hipStream_t)stream) != hipSuccess) return TWINKV_E_HIP;
  return TWINKV_OK;
}

const char* twinkv_status_string(int status) {
  switch (status) {
    case TWINKV_OK: return "ok";
    case TWINKV_E_NULL: return "a required pointer is NULL";
    case TWINKV_E_ARG: return "invalid argument";
    case TWINKV_E_UNSUPPORTED: return "unsupported head dimension or key dtype";
    case TWINKV_E_WORKSPACE: return "workspace missing or too small";
    case TWINKV_E_HIP: return "HIP runtime error";
    case TWINKV_E_CAPACITY: return "the batch needs more than the static scratch buffer holds";
    default: return "unknown status";
  }
}

int twinkv_version(void) { return kVersion; }

void twinkv_profile_sim_events(void* start_event, void* stop_event) {
  g_sim_start = reinterpret_cast<hipEvent_t>(start_event);
  g_sim_stop = reinterpret_cast<hipEvent_t>(stop_event);
}

}  // extern "C"
