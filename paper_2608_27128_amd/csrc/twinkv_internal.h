// Internal declarations shared by the host layer (api.cpp) and the HIP kernels.
// Nothing here is part of the public ABI (include/twinkv.h).
#pragma once

#include <cstddef>
#include <cstdint>

namespace twinkv {

// Per-sequence table copied into the workspace.  Entries [s].start/len/budget/perm_off
// describe sequence s; entries [r].sorted_seq/tile_cum/nb describe the sequence of rank r
// in the longest-first order used to schedule similarity tiles.
struct SeqInfo {
  int32_t start;       // first global token of the sequence
  int32_t len;         // tokens in the sequence
  int32_t budget;      // |S0| every problem of this sequence must have (-1: not checked)
  int32_t perm_off;    // offset of this sequence's partitioned column list inside a head
  int32_t sorted_seq;  // sequence at rank r (longest first)
  int32_t tile_cum;    // row-block tiles of ranks < r
  int32_t nb;          // row-block tiles of the sequence at rank r
  int32_t prep_blk0;   // first key-preparation workgroup of sequence s (K1b grid)
};

// Per-problem result of the partition step.
struct ProblemMeta {
  int32_t n_ret;         // |S0|
  int32_t ret_chunks;    // 32-column chunks of the S0 group (padded to kGroupAlign columns)
  int32_t total_chunks;  // chunks of S0 followed by chunks of the evicted columns
  int32_t flags;         // bit 0: a key of the problem is non-finite
};

constexpr int kChunk = 32;           // columns per MFMA chunk (the 32x32x16 tile)
// The S0 group of a column list is padded to a multiple of kGroupAlign columns, so the
// evicted group starts on a column-tile boundary of the similarity kernel.
#ifndef TWINKV_GROUP_ALIGN
#define TWINKV_GROUP_ALIGN 128
#endif
constexpr int kGroupAlign = TWINKV_GROUP_ALIGN;
constexpr int kPermPad = kGroupAlign + kChunk;  // padding per (head, sequence) in the column lists
constexpr int kFlagNonfinite = 1;

// Workspace layout shared by the size query and the launchers.
struct Layout {
  size_t seqtab = 0, rinv = 0, pcol = 0, rcol = 0, prank = 0, pmeta = 0, hilo = 0, pkeys = 0,
         bbuf = 0, chunk_seq = 0, chunk_cnt = 0;
  size_t total = 0;
};

// ---- launchers (defined in the kernel translation units) ----
// Each returns 0 on success or a hipError_t value.

// Copies `bytes` (a multiple of 4) of host memory to device memory `dst` on `stream` through
// kernel arguments: the host buffer may be freed as soon as the call returns, also when the
// launches are captured into a graph.
int launch_upload(const void* src, size_t bytes, void* dst, void* stream);

// K1a: stable partition of each problem's positions into [S0 | evicted] column lists from the
// retained mask: pcol (positions, -1 for padding), prank[t] = number of S0 positions before t
// (t = 0..len), the per-problem meta, rcol = 0 at padding, status = 0.
int launch_partition(const uint8_t* retained, const SeqInfo* seqtab, int n_heads, int n_seqs,
                     int64_t T, int64_t PT, int max_len, int32_t* pcol, float* rcol,
                     int32_t* prank, ProblemMeta* pmeta, int32_t* status, void* stream);

// K1b: one pass over the keys after K1a: inverse l2 norm of every key (fp64 accumulation) to
// rinv and to rcol at the key's column slot, the key copied to pkeys[h][PT][dcol] at that slot
// (bf16; dcol = 2d bf16 hi/lo for fp32 keys, which also go to the row plane hilo
// [n_heads][T][2d]); a non-finite key sets the problem's flag and status.  With copy_evicted
// = 0 only the S0 columns are copied (sweeps over the retained columns alone).
// Tokens one K1b workgroup prepares for this (dtype, d); sequence s owns workgroups
// [seqtab[s].prep_blk0, seqtab[s].prep_blk0 + ceil(len / that)) of each head.
int prepare_tokens_per_block(int dtype, int d);
int launch_prepare_keys(const void* keys, int dtype, int d, int n_heads, int64_t T,
                        int64_t head_stride, int64_t token_stride, int64_t PT, int total_blocks,
                        const uint8_t* retained, const int32_t* prank, ProblemMeta* pmeta,
                        const SeqInfo* seqtab, int n_seqs, float* rinv, float* rcol,
                        uint16_t* hilo, uint16_t* pkeys, int32_t* status, int copy_evicted,
                        void* stream);
// K1b for the level groups of nested retained sets in one pass over the keys: a token of
// level l in [1, n_levels] goes to the S0 list of group l - 1, a token of level 0 or above
// n_levels to group n_levels when n_groups > n_levels (the tokens in no set) and nowhere
// otherwise.  prank, pmeta, rcol and pkeys are group 0's; group g's lie g * group_stride
// bytes further (each group partitioned by K1a beforehand).  rinv (and the fp32 row plane)
// is written once.
struct PrepLevels {
  const uint8_t* level;   // [n_heads][T]
  int n_levels;
  int n_groups;
  int64_t group_stride;   // bytes between consecutive groups' arrays
};
int launch_prepare_keys_levels(const void* keys, int dtype, int d, int n_heads, int64_t T,
                               int64_t head_stride, int64_t token_stride, int64_t PT,
                               int total_blocks, const PrepLevels& lv, const int32_t* prank,
                               ProblemMeta* pmeta, const SeqInfo* seqtab, int n_seqs, float* rinv,
                               float* rcol, uint16_t* hilo, uint16_t* pkeys, int32_t* status,
                               void* stream);

struct SimArgs {
  const void* keys;          // bf16 keys, or the hi/lo planes for fp32 keys
  int64_t head_stride;       // elements (of uint16) between heads of `keys`
  int64_t token_stride;      // elements between tokens of `keys`
  const float* rinv;         // [n_heads][T]
  const uint16_t* pkeys;     // [n_heads][PT][dcol] column keys in partitioned order
  const int32_t* pcol;       // [n_heads][PT]
  const float* rcol;         // [n_heads][PT]
  const int32_t* prank;      // [n_heads][PT]: S0 positions before t
  const ProblemMeta* pmeta;  // [n_heads * n_seqs]
  const SeqInfo* seqtab;     // [n_seqs]
  int n_heads, n_seqs;
  int64_t T, PT;
  int w;
  int want_all;              // also reduce over evicted columns (best_all / arg_all)
  float tau;                 // count mode: the twin threshold of Eq. 2
  int32_t* counts;           // non-null: count mode, [n_heads][T] twin counts (Eq. 2)
  int total_tiles;           // row-block tiles of all sequences (sum of nb)
  float* best_all;
  int32_t* arg_all;
  float* best_ret;
  int32_t* arg_ret;
};

// Rows covered by one workgroup of the similarity kernel for this (dtype, d).
int sim_rows_per_block(int dtype, int d);
// K2: fused MFMA similarity with the two masked row max / argmax reductions, or (counts set)
// the per-token twin counts of Eq. 2 over all columns.
int launch_sim_reduce(const SimArgs& a, int dtype, int d, void* stream);

struct RepairArgs {
  const float* b;            // [n_heads][T]
  const uint8_t* s0;         // [n_heads][T]
  uint8_t* s1;               // [n_heads][T]
  const SeqInfo* seqtab;
  const ProblemMeta* pmeta;  // nullable: key status from the partition step
  int n_heads, n_seqs;
  int64_t T;
  float tau;
  int n_sink, n_recent;
  int max_len;               // longest sequence (picks the workgroup size)
  int32_t* stats;            // [n_heads * n_seqs][4]
};
// K3: orphan / donor classification, radix selection of the m most severe, swap.
int launch_repair(const RepairArgs& a, void* stream);

// The body of twinkv_repair_from_scores and of its variant without allocation: validates the
// arguments (returning TWINKV_E_* before any HIP call), returns TWINKV_E_CAPACITY when the
// sequence table needs more than table_bytes, then takes the table's device address from
// resolve_table() when that is non-null (else `table`), uploads the table and launches K3.
int repair_from_scores_into(const float* b, const uint8_t* retained_in, uint8_t* retained_out,
                            int n_heads, int n_seqs, const int64_t* cu_seqlens,
                            const int64_t* budget, float tau, int n_sink, int n_recent,
                            int32_t* stats, void* table, size_t table_bytes,
                            void* (*resolve_table)(), void* stream);

struct EvictArgs {
  const int32_t* counts;     // [n_heads][T] Eq. 2 twin counts (scorer)
  const float* in_scores;    // [n_heads][T] a policy's scores (policy selection), else null
  uint8_t* retained;         // [n_heads][T] out: kept set
  float* scores;             // nullable [n_heads][T] out: Eq. 3 scores
  int32_t* stats;            // [n_heads * n_seqs][4]
  const SeqInfo* seqtab;     // budget per sequence in .budget
  const ProblemMeta* pmeta;  // key status from the key preparation
  int n_heads, n_seqs;
  int64_t T;
  int n_sink, n_recent;
  int max_len;               // longest sequence (picks the workgroup size)
};
// K4a: the standalone scorer's retained set (the budget highest Eq. 3 scores), or with
// in_scores a score-based policy's retained set.
int launch_evict(const EvictArgs& a, void* stream);

constexpr int kMaxTaus = 32;
struct PrevalenceArgs {
  const float* best;         // [n_heads][T] best_all
  int32_t* out;              // [n_heads * n_seqs][n_taus]
  const SeqInfo* seqtab;
  int n_heads, n_seqs;
  int64_t T;
  int n_taus;
  float taus[kMaxTaus];
};
// K4b: tokens with at least one twin per threshold (best_all > tau).
int launch_prevalence(const PrevalenceArgs& a, void* stream);

// Nested retained sets: the 0/1 mask of one level group, and the merge of per-group maxima.
constexpr int kMaxLevels = 4;
int launch_select_level(const uint8_t* level, uint8_t* mask, int64_t n, int sel, int n_levels,
                        void* stream);
struct CombineArgs {
  const float* gbest;        // [n_groups][n]: best over each level group (-1 if none)
  const int32_t* garg;       // [n_groups][n]: its position (-1 if none)
  int n_groups;              // n_levels, plus one for the tokens in no set (best_all)
  int n_levels;
  int64_t n;                 // n_heads * T
  float* best_lvl;           // [n_levels][n] nullable
  int32_t* arg_lvl;          // [n_levels][n] nullable
  float* best_all;           // [n] nullable
  int32_t* arg_all;          // [n] nullable
};
int launch_combine_levels(const CombineArgs& a, void* stream);

// KV compaction: positions per chunk of the retained mask, one workgroup per (head, chunk).
#ifndef TWINKV_COMPACT_CHUNK
#define TWINKV_COMPACT_CHUNK 2048
#endif
constexpr int kCompactChunk = TWINKV_COMPACT_CHUNK;
struct CompactSeq {
  int32_t start;      // first global token of the sequence
  int32_t len;        // tokens
  int32_t cap;        // reserved output rows per problem of this sequence (<= len)
  int32_t out_start;  // first reserved row inside a head's block of C rows
  int32_t chunk0;     // first chunk of the sequence in the chunk list
  int32_t nchunks;    // chunks of the sequence (at least 1, so every problem reports stats)
  int32_t pad[2];
};
struct CompactArgs {
  const char* keys;          // byte addresses; rows of row_bytes at the given byte strides
  const char* values;        // nullable
  int64_t head_stride, token_stride;      // bytes
  int64_t v_head_stride, v_token_stride;  // bytes
  int row_bytes;             // d * element size, a multiple of 16
  int log2_pieces;           // log2(row_bytes / 16)
  const uint8_t* retained;   // [n_heads][T]
  const CompactSeq* seqs;    // [n_seqs]
  const int32_t* chunk_seq;  // [n_chunks]: sequence of each chunk
  int32_t* chunk_cnt;        // [n_heads][n_chunks]: kept positions per chunk (workspace)
  char* keys_out;            // [n_heads][C] rows
  char* values_out;          // nullable, like keys_out
  int32_t* pos_out;          // nullable [n_heads][C]
  int32_t* stats;            // [n_heads * n_seqs][4]
  int n_heads, n_seqs, n_chunks;
  int64_t T, C;
};
// K5a: kept positions per (head, chunk) into chunk_cnt.
int launch_compact_count(const CompactArgs& a, void* stream);
// K5b (after K5a): the kept rows of every problem gathered in position order into its
// reserved rows, unused rows zeroed, stats written.
int launch_compact_gather(const CompactArgs& a, void* stream);

}  // namespace twinkv
