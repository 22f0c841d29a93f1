/*
 * twinkv.h -- C ABI of the TwinKV redundancy / repair library for AMD MI355X (gfx950).
 *
 * TwinKV (paper: "TwinKV: A Composable Repair Pass for KV Cache Eviction via Pairwise
 * Key Redundancy") works per (layer, KV head) on the keys of one sequence (Sec. 3.1):
 *   - Eq. 1: sim(i, j) = k_hat_i . k_hat_j with k_hat = k / ||k||_2 (Sec. 3.2);
 *   - twin rule: j is a twin of i iff sim(i, j) > tau and |i - j| > w (Sec. 3.2, Eq. 2);
 *   - Eq. 4: b_i(S0) = max over j in S0, |i - j| > w of sim(i, j), or -1 if no such j;
 *   - repair (Sec. 3.4): orphans (i not in S0, b_i < tau) and redundant donors (j in S0,
 *     outside the protected sink / recent regions, b_j >= tau) are ranked by severity
 *     (orphans by ascending b, donors by descending b) and the m = min(|O|, |D|) most severe
 *     pairs are swapped, so |S1| = |S0| = K exactly;
 *   - the standalone scorer (Sec. 3.2, Eq. 2-3): twin counts r_i, scores s_i = -r_i / n, and
 *     the retained set of the K highest scores with the sink / recent regions kept first;
 *   - the prevalence statistic of Sec. 2 (Fig. 1b): tokens with at least one twin;
 *   - a wrapped policy's retained set from its per-token scores (Sec. 3.1: K positions per
 *     head and layer; Sec. 3.2: the sink / recent regions at the maximum score), the S0 the
 *     repair takes;
 *   - KV compaction (Sec. 3.1): only the keys and values at the retained positions are kept
 *     for generation, gathered here into a dense cache.
 *
 * Problems.  A batch holds n_heads (layer, KV head) pairs times n_seqs sequences.  Sequence s
 * owns global token positions [cu_seqlens[s], cu_seqlens[s+1]) and T = cu_seqlens[n_seqs].
 * Problem q = h * n_seqs + s is (head h, sequence s); problems are independent (Sec. 3.1).
 * Indices reported by the library are 0-based positions inside the sequence.
 *
 * Memory.  Unless marked "(host)", pointers are DEVICE pointers owned by the caller.  The
 * library allocates nothing: scratch space is the caller's `workspace` (size from
 * twinkv_workspace_bytes).  Keys: element (h, t, c) is at keys[h*head_stride + t*token_stride
 * + c] (strides in elements, channels contiguous); the pointer and both strides (in bytes)
 * must be multiples of 16.  Per-token arrays (retained masks, scores, indices) are contiguous
 * [n_heads][T].  Every entry point enqueues work on `stream` (a hipStream_t passed as void*;
 * NULL = the default stream) and returns without waiting; results are valid once the stream
 * has reached that point.  The small per-sequence table built from the host arrays reaches
 * the workspace as the kernel arguments of upload launches, so the host arrays are consumed
 * before the call returns and no host memory is read later.  A call enqueues kernel launches
 * only (no memset, no host copy, no allocation), so it may be captured into a HIP graph; a
 * replay repeats the captured batch description (sequence lengths, budgets, tau, w) and
 * re-reads the device buffers it was given.  twinkv_profile_sim_events adds event records.
 *
 * Errors.  Argument errors are detected on the host before anything is enqueued and are
 * returned synchronously (TWINKV_E_*).  A HIP failure while enqueueing returns TWINKV_E_HIP.
 * Data-dependent conditions are reported per problem (TWINKV_PROBLEM_*), never by failing.
 * Concurrent calls are safe as long as they use different workspaces.
 */
#ifndef TWINKV_H
#define TWINKV_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Return codes. */
#define TWINKV_OK             0
#define TWINKV_E_NULL         1  /* a required pointer is NULL */
#define TWINKV_E_ARG          2  /* an argument value is out of range or inconsistent */
#define TWINKV_E_UNSUPPORTED  3  /* head dimension or dtype not supported */
#define TWINKV_E_WORKSPACE    4  /* workspace missing or smaller than required */
#define TWINKV_E_HIP          5  /* the HIP runtime reported an error */
#define TWINKV_E_CAPACITY     6  /* the batch needs more than the static scratch buffer holds */

/* Key element types. */
#define TWINKV_BF16 0
#define TWINKV_F32  1

/* Operations, for twinkv_workspace_bytes. */
#define TWINKV_OP_NN_SCORES          0
#define TWINKV_OP_REPAIR             1
#define TWINKV_OP_REPAIR_FROM_SCORES 2
#define TWINKV_OP_TWIN_COUNTS        3
#define TWINKV_OP_SCORE_EVICT        4
#define TWINKV_OP_COMPACT            5

/* Most thresholds twinkv_prevalence takes in one call. */
#define TWINKV_MAX_TAUS 32

/* Most nested retained sets twinkv_nn_scores_levels takes in one call. */
#define TWINKV_MAX_LEVELS 4

/* Per-problem status codes (stats[q][3] / status[q]). */
#define TWINKV_PROBLEM_OK              0
#define TWINKV_PROBLEM_BUDGET_MISMATCH 1  /* |S0| differs from the budget; S1 = S0 */
#define TWINKV_PROBLEM_NONFINITE       2  /* a key (or a given score) is NaN/Inf; S1 = S0 */

/*
 * Bytes of workspace `op` needs for this batch; negative (-TWINKV_E_*) on invalid arguments.
 * cu_seqlens (host, n_seqs + 1 entries, non-decreasing, cu_seqlens[0] = 0).
 * dtype and d are ignored for TWINKV_OP_REPAIR_FROM_SCORES and TWINKV_OP_COMPACT.
 */
int64_t twinkv_workspace_bytes(int op, int dtype, int d, int n_heads, int n_seqs,
                               const int64_t* cu_seqlens);

/*
 * Best twin of every token (Sec. 3.2 Eq. 1 + the twin rule's window; Sec. 3.4 Eq. 4).
 *
 *   keys       [n_heads][T][d] bf16 or fp32 (see Memory).  d must be 64 or 128.
 *   retained   [n_heads][T] uint8, nonzero = in S0; NULL skips the retained reduction.
 *   w          window half-width, >= 0: pairs with |i - j| <= w are never compared.
 *   best_all   [n_heads][T] fp32: max over j with |i-j| > w of sim(i, j); -1 if none.  Nullable.
 *   arg_all    [n_heads][T] int32: the maximising j (position in the sequence); -1 if none.
 *              On near-equal candidates the reported j is one whose similarity is within
 *              2^-15 (3.1e-5) of the maximum for bf16 keys with d = 128 and 2^-17 (7.6e-6)
 *              otherwise; on exact equality it is the smallest such j.  Nullable.
 *   best_ret   [n_heads][T] fp32: b_i(S0) of Eq. 4 (-1 if no retained j beyond the window).
 *              Nullable; must be NULL when retained is NULL.
 *   arg_ret    [n_heads][T] int32: the maximising retained j, -1 if none.  Nullable.
 *   status     [n_heads * n_seqs] int32 TWINKV_PROBLEM_* (only OK / NONFINITE).  Nullable.
 *              The scores of a problem with a non-finite key are unspecified (the similarity
 *              is undefined there); every other problem's are unaffected.
 *
 * Similarities are computed from the stored key values with fp32 accumulation; their error
 * against exact arithmetic is below 1e-4 for bf16 and fp32 keys (this includes the rounding
 * down of reported values by less than the tie bound above).  Every result is independent of
 * a key's length as Eq. 1 is: scaling a key by a power of two changes no output bit, as long
 * as its elements, their products with the other keys' elements and its norm stay in fp32's
 * normal range (below 2^120 and above 2^-126 in magnitude).
 */
int twinkv_nn_scores(const void* keys, int dtype, int d, int n_heads, int n_seqs,
                     const int64_t* cu_seqlens, int64_t head_stride, int64_t token_stride,
                     const uint8_t* retained, int w,
                     float* best_all, int32_t* arg_all, float* best_ret, int32_t* arg_ret,
                     int32_t* status,
                     void* workspace, int64_t workspace_bytes, void* stream);

/*
 * The full repair pass of Sec. 3.4 for every problem: Eq. 4 scores, orphan / donor
 * classification, severity ranking and the budget-preserving swap.
 *
 *   retained_in   [n_heads][T] uint8, the wrapped policy's S0 (nonzero = retained).
 *   retained_out  [n_heads][T] uint8, receives S1 as 0/1.  May alias retained_in.
 *   budget        (host) [n_seqs] int64: K = |S0| of every problem of sequence s.  A problem
 *                 whose |S0| differs gets TWINKV_PROBLEM_BUDGET_MISMATCH and S1 = S0.
 *   tau           duplicate threshold (finite).  Orphan: b < tau.  Donor: b >= tau.
 *   w             window half-width, >= 0.
 *   n_sink, n_recent  >= 0: positions [0, n_sink) and [len - n_recent, len) are protected
 *                 (never donors).
 *   stats         [n_heads * n_seqs][4] int32 = {|O|, |D|, m, status}.
 *   best_all, arg_all, best_ret, arg_ret   optional outputs as in twinkv_nn_scores (nullable).
 *                 When best_all and arg_all are both NULL, similarities against evicted keys
 *                 are skipped (only S0 columns are needed for b).
 *
 * Ranking ties resolve by ascending position (among equal b, the earlier orphan is admitted
 * and the earlier donor evicted first).
 */
int twinkv_repair(const void* keys, int dtype, int d, int n_heads, int n_seqs,
                  const int64_t* cu_seqlens, int64_t head_stride, int64_t token_stride,
                  const uint8_t* retained_in, uint8_t* retained_out,
                  const int64_t* budget, float tau, int w, int n_sink, int n_recent,
                  int32_t* stats,
                  float* best_all, int32_t* arg_all, float* best_ret, int32_t* arg_ret,
                  void* workspace, int64_t workspace_bytes, void* stream);

/*
 * Classification, severity ranking and swap of Sec. 3.4 from given scores b = b_i(S0)
 * ([n_heads][T] fp32), e.g. produced by twinkv_nn_scores or by another scorer.  Arguments as
 * in twinkv_repair.  A NaN/Inf score gives TWINKV_PROBLEM_NONFINITE and S1 = S0.
 */
int twinkv_repair_from_scores(const float* b, const uint8_t* retained_in, uint8_t* retained_out,
                              int n_heads, int n_seqs, const int64_t* cu_seqlens,
                              const int64_t* budget, float tau, int n_sink, int n_recent,
                              int32_t* stats,
                              void* workspace, int64_t workspace_bytes, void* stream);

/*
 * twinkv_repair_from_scores for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): no workspace
 * argument.  The only scratch the call needs, the per-sequence table, lives in a static
 * device buffer of the library (64 KiB per GPU, held until the process ends), so at most
 * TWINKV_NOALLOC_MAX_SEQS sequences per call; a larger batch returns TWINKV_E_CAPACITY before
 * anything is enqueued.  The buffer of the current device is used (the stream must belong to
 * it).  Every call on one GPU shares that buffer: calls that overlap on one GPU (different
 * streams, or host threads enqueueing concurrently) race and must be serialised by the
 * caller.  Nothing in the buffer needs to start at zero (each call writes the whole table it
 * reads).  The call allocates nothing; results equal twinkv_repair_from_scores.
 */
#define TWINKV_NOALLOC_MAX_SEQS 2048
int twinkv_repair_from_scores_noalloc(const float* b, const uint8_t* retained_in,
                                      uint8_t* retained_out, int n_heads, int n_seqs,
                                      const int64_t* cu_seqlens, const int64_t* budget,
                                      float tau, int n_sink, int n_recent, int32_t* stats,
                                      void* stream);

/*
 * Twin counts of Sec. 3.2 Eq. 2 for every token:
 *   counts[h][t] = #{ j in t's sequence : |i - j| > w, sim(i, j) > tau },  i = t's position.
 *
 *   keys, dtype, d, n_heads, n_seqs, cu_seqlens, strides, w   as in twinkv_nn_scores.
 *   tau      twin threshold (finite).
 *   counts   [n_heads][T] int32 (required).
 *   status   [n_heads * n_seqs] int32 TWINKV_PROBLEM_* (only OK / NONFINITE).  Nullable.
 *            The counts of a problem with a non-finite key are unspecified.
 *   workspace  twinkv_workspace_bytes(TWINKV_OP_TWIN_COUNTS, ...) bytes.
 *
 * The decision sim > tau is taken on fp32 similarities (error below 1e-4, typically 1e-6):
 * pairs whose exact similarity is that close to tau may fall on either side.
 */
int twinkv_twin_counts(const void* keys, int dtype, int d, int n_heads, int n_seqs,
                       const int64_t* cu_seqlens, int64_t head_stride, int64_t token_stride,
                       float tau, int w, int32_t* counts, int32_t* status,
                       void* workspace, int64_t workspace_bytes, void* stream);

/*
 * b_i(S_k) of Sec. 3.4 Eq. 4 for nested retained sets S_1 within S_2 within ... within S_L
 * (for example the retained sets of one policy at increasing budgets), in one call.
 * The tokens of each level group G_k = S_k minus S_{k-1} are swept once as the retained
 * columns, so the similarity work is N * |S_L| per problem (plus N * (N - |S_L|) when the
 * all-keys result is asked for), instead of N * (|S_1| + ... + |S_L|) for L separate calls.
 *
 *   level     [n_heads][T] uint8: k in 1..n_levels = the smallest set that holds the token;
 *             0 = in none.  Values above n_levels count as 0.
 *   n_levels  1 <= L <= TWINKV_MAX_LEVELS.
 *   best_lvl  [n_levels][n_heads][T] fp32: b_i(S_k) (-1 if no j of S_k lies outside the
 *             window).  Required.
 *   arg_lvl   [n_levels][n_heads][T] int32: the maximising position, -1 if none.  Nullable.
 *   best_all, arg_all  as in twinkv_nn_scores.  Nullable; when both are NULL the tokens in
 *             no set are never swept as columns.
 *   workspace twinkv_levels_workspace_bytes(dtype, d, n_heads, n_seqs, cu_seqlens,
 *             n_levels, want_all) bytes, want_all = (best_all or arg_all given).
 * Other arguments as in twinkv_nn_scores.  Results equal those of separate
 * twinkv_nn_scores calls with retained = S_k, bit for bit: every value is the same
 * computation, and equal values go to the smaller position in both.
 */
int twinkv_nn_scores_levels(const void* keys, int dtype, int d, int n_heads, int n_seqs,
                            const int64_t* cu_seqlens, int64_t head_stride, int64_t token_stride,
                            const uint8_t* level, int n_levels, int w, float* best_all,
                            int32_t* arg_all, float* best_lvl, int32_t* arg_lvl, int32_t* status,
                            void* workspace, int64_t workspace_bytes, void* stream);

/* Workspace bytes of twinkv_nn_scores_levels; negative (-TWINKV_E_*) on invalid arguments. */
int64_t twinkv_levels_workspace_bytes(int dtype, int d, int n_heads, int n_seqs,
                                      const int64_t* cu_seqlens, int n_levels, int want_all);

/*
 * The standalone TwinKV scorer of Sec. 3.2: Eq. 2 twin counts, Eq. 3 scores
 * s_i = -r_i / n (n = the sequence length), and the retained set of the `budget` highest
 * scores.  The sink region [0, n_sink) and recent region [len - n_recent, len) take the
 * maximum score, so they are kept first; among equal scores the later position is kept
 * first (recency).  With budget >= len every token is kept; with budget 0 none.
 *
 *   budget        (host) [n_seqs] int64 in [0, 2^31 - 1]: tokens to keep per problem of
 *                 sequence s (the paper's ceil((1 - rho) n) for compression ratio rho is the
 *                 caller's).
 *   retained_out  [n_heads][T] uint8, receives the kept set as 0/1 (required).
 *   counts        [n_heads][T] int32, the Eq. 2 counts.  Nullable (then kept in workspace).
 *   scores        [n_heads][T] fp32, the Eq. 3 scores.  Nullable.
 *   stats         [n_heads * n_seqs][4] int32 = {tokens kept, count at the cut (-1 when the
 *                 cut falls inside the protected regions or nothing is cut), status, 0}.
 *                 A problem with a non-finite key (status NONFINITE) still keeps exactly its
 *                 budget, protected regions first; which other tokens is unspecified.
 *   workspace     twinkv_workspace_bytes(TWINKV_OP_SCORE_EVICT, ...) bytes.
 * Other arguments as in twinkv_twin_counts.
 */
int twinkv_score_evict(const void* keys, int dtype, int d, int n_heads, int n_seqs,
                       const int64_t* cu_seqlens, int64_t head_stride, int64_t token_stride,
                       const int64_t* budget, float tau, int w, int n_sink, int n_recent,
                       uint8_t* retained_out, int32_t* counts, float* scores, int32_t* stats,
                       void* workspace, int64_t workspace_bytes, void* stream);

/*
 * A score-based policy's retained set (Sec. 3.1: a policy keeps |S| = K positions per head
 * and layer; Sec. 3.2: the sink and recent regions take the maximum score): per problem,
 * the budget positions first in this order: protected positions (by position), then higher
 * scores, equal scores by lower position, NaN scores after every number (-0 equals +0).
 * With budget >= len every token is kept; with budget 0 none.  The result is the S0 that
 * twinkv_repair takes, so a wrapped policy that computes per-token scores on the GPU
 * (attention mass, an expected-attention estimate, a recency score) stays on the GPU.
 *
 *   scores        [n_heads][T] fp32 (any values, NaN and infinities included).
 *   budget        (host) [n_seqs] int64 in [0, 2^31 - 1]: tokens to keep per problem of
 *                 sequence s (values above the length keep everything).
 *   retained_out  [n_heads][T] uint8, receives the kept set as 0/1 (required).
 *   stats         [n_heads * n_seqs][4] int32 = {tokens kept, NaN scores, 0, 0}.  Nullable.
 *   workspace     twinkv_workspace_bytes(TWINKV_OP_REPAIR_FROM_SCORES, ...) bytes (the
 *                 sequence table).
 * Errors: NULL scores / budget / retained_out, a negative n_sink / n_recent or budget, or a
 * malformed cu_seqlens are rejected before anything is enqueued.
 */
int twinkv_select_topk(const float* scores, int n_heads, int n_seqs, const int64_t* cu_seqlens,
                       const int64_t* budget, int n_sink, int n_recent, uint8_t* retained_out,
                       int32_t* stats, void* workspace, int64_t workspace_bytes, void* stream);

/*
 * Twin prevalence (Sec. 2, Fig. 1b): for every problem q and threshold taus[k],
 *   out[q][k] = #{ tokens i of q : best_all[i] > taus[k] },
 * the number of tokens with at least one twin at that threshold (Eq. 2), from best_all as
 * produced by twinkv_nn_scores or twinkv_repair.
 *
 *   best_all  [n_heads][T] fp32.
 *   taus      (host) [n_taus] fp32, 1 <= n_taus <= TWINKV_MAX_TAUS.
 *   out       [n_heads * n_seqs][n_taus] int32.
 *   workspace  twinkv_workspace_bytes(TWINKV_OP_REPAIR_FROM_SCORES, ...) bytes (the sequence
 *              table).
 */
int twinkv_prevalence(const float* best_all, int n_heads, int n_seqs, const int64_t* cu_seqlens,
                      const float* taus, int n_taus, int32_t* out,
                      void* workspace, int64_t workspace_bytes, void* stream);

/*
 * KV compaction (Sec. 3.1): eviction keeps only the keys and values at the retained
 * positions.  For every problem (h, s) the rows of its retained tokens are copied, bit for
 * bit and in ascending position order, into the problem's `capacity[s]` reserved rows of a
 * dense cache; the usual caller passes S1 from twinkv_repair (or the scorer's retained set)
 * with capacity = the budget.
 *
 *   keys, values  [n_heads][T][d] bf16 or fp32 at (head_stride, token_stride) and
 *                 (v_head_stride, v_token_stride) elements (see Memory); d must be 64 or
 *                 128.  values may be NULL (keys only), and then values_out must be NULL.
 *   retained      [n_heads][T] uint8, nonzero = keep.
 *   capacity      (host) [n_seqs] int64, 0 <= capacity[s] <= length of sequence s: rows
 *                 reserved for each problem of sequence s.
 *   keys_out, values_out  [n_heads][C][d] dense, same dtype, 16-byte aligned,
 *                 C = sum of capacity.  Problem (h, s) owns rows [c_s, c_s + capacity[s]) of
 *                 head h, c_s = sum of capacity[s'] for s' < s.  Must not overlap the inputs.
 *   pos_out       [n_heads][C] int32: the position in the sequence of each row's token; -1
 *                 for unused rows.  Nullable.
 *   stats         [n_heads * n_seqs][4] int32 = {retained positions, capacity, status, 0};
 *                 status TWINKV_PROBLEM_BUDGET_MISMATCH when a problem retains more
 *                 positions than its capacity (then all its rows are zero, positions -1).
 *                 Reserved rows past the retained count are zero with position -1.
 *   workspace     twinkv_workspace_bytes(TWINKV_OP_COMPACT, ...) bytes.
 */
int twinkv_compact(const void* keys, const void* values, int dtype, int d, int n_heads,
                   int n_seqs, const int64_t* cu_seqlens, int64_t head_stride,
                   int64_t token_stride, int64_t v_head_stride, int64_t v_token_stride,
                   const uint8_t* retained, const int64_t* capacity, void* keys_out,
                   void* values_out, int32_t* pos_out, int32_t* stats, void* workspace,
                   int64_t workspace_bytes, void* stream);

/*
 * Profiling hook.  For calls made afterwards from the calling thread, record the given
 * hipEvent_t handles on the call's stream immediately before and immediately after the
 * launch of the call's main kernel -- the similarity kernel (the fused contraction +
 * reductions), or in twinkv_compact the row gather -- so its duration can be read with
 * hipEventElapsedTime.  The events stay owned by the caller; pass NULL, NULL to
 * stop recording.
 */
void twinkv_profile_sim_events(void* start_event, void* stop_event);

/* Static description of a return code (TWINKV_OK, TWINKV_E_*); never freed. */
const char* twinkv_status_string(int status);

/* Library version as major * 10000 + minor * 100 + patch. */
int twinkv_version(void);

#ifdef __cplusplus
}
#endif

#endif /* TWINKV_H */
