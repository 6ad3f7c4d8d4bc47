/*
 * sparse_engine.h — C-ABI of the sparse-first decode hot path on MI355X (gfx950).
 *
 * The library implements the per-step work of sparse-attention methods over a
 * paged, per-KV-head KV cache (H2O and Quest decode; SnapKV prompt compaction;
 * OmniKV cross-layer selection; H2O chunk-wise prefill eviction; interval
 * prefix-cache pruning), following the SparseEngine paper's statement of the
 * problem:
 *   - the cache manager owns layout, position mapping and write/update/release
 *     (Section 3.1, "Method-Customized CacheManager");
 *   - attention reads a view of the cache: o = Attention(q, BuildView(C, I))
 *     (Section 3.1, eq. attention-view), whose payload pairs the physical KV with
 *     context lengths and page-table coordinates (Appendix B, "Attention View
 *     Payloads");
 *   - H2O grows accumulated scores and evicts to a budget with a protected recent
 *     window (Appendix A.3, eqs. background-h2o-score, background-h2o-retention);
 *   - Quest ranks pages by a min/max upper bound of the logits and reads the best
 *     pages (Appendix A.3, eqs. background-quest-summary, background-quest-score);
 *   - SnapKV, OmniKV and the prefill and pruning operations are declared below,
 *     each with the passages that define it.
 *
 * Conventions shared by every call
 * --------------------------------
 *  Units.   A unit is one (request, KV head) of one layer: unit = req * Hkv + h.
 *           Units are independent.  A multi-layer cache is one view per layer
 *           (each with its own block_table and lengths rows; pools may be shared).
 *  GQA.     Query head a reads KV head floor(a / G), G = q_per_kv (Appendix A.1,
 *           "MHA, MQA, and GQA"), so a unit's G query rows are contiguous.
 *  Layout.  Slot s of a unit lives in physical page block_table[unit][s / 16] at
 *           row s % 16 (Appendix A.2, "Logical Positions and Physical Blocks", in
 *           0-based form).  A page holds its 16 keys, then its 16 values.
 *  Memory.  Every pointer argument is a DEVICE pointer owned by the caller, except
 *           `kv` (the view struct itself, host memory, read during the call) and
 *           the `host_out` of se_read_device_errors.  The library allocates no
 *           memory and keeps no state between calls; calls on different streams
 *           may run concurrently when their buffers do not overlap.
 *  Streams. Every compute call only enqueues work on `stream` and returns without
 *           waiting (so a sequence of calls can be captured in a hipGraph).  Only
 *           se_read_device_errors synchronises.
 *  Errors.  The host checks only scalars and pointer presence and returns a status
 *           before enqueuing anything.  Problems that can only be seen on the device
 *           (a bad page id, a full unit, a length above max_len) set bits in the
 *           int32 word *dev_err (atomic OR) and the affected unit is left unchanged;
 *           read and clear the word with se_read_device_errors.
 *  Numbers. K/V/q are bf16; logits, softmax and accumulation are fp32; outputs fp32.
 *  Limits.  page_size must be 16; head_dim 64 or 128; q_per_kv 1, 2, 4 or 8
 *           (se_accumulate_scores and se_omnikv_select: 1 .. 8).
 */
#ifndef SPARSE_ENGINE_H
#define SPARSE_ENGINE_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum se_status {
  SE_OK = 0,
  SE_ERR_INVALID_ARGUMENT = 1, /* a NULL required pointer, a negative size, ...     */
  SE_ERR_UNSUPPORTED = 2,      /* a size the kernels are not built for               */
  SE_ERR_WORKSPACE = 3,        /* ws is NULL or smaller than se_workspace_bytes()    */
  SE_ERR_HIP = 4               /* a HIP launch error                                  */
} se_status;

/* Bits of the device error word. */
#define SE_DEVERR_BAD_PAGE      1u  /* a block-table entry outside [0, num_pages)          */
#define SE_DEVERR_CAPACITY      2u  /* an append past max_pages * page_size                */
#define SE_DEVERR_BAD_LENGTH    4u  /* lengths[unit] < 0, or above max_len / capacity     */
#define SE_DEVERR_BAD_SELECTION 8u  /* a sel_pages entry outside the unit's pages          */
#define SE_DEVERR_BAD_POSITIONS 16u /* eviction found repeated positions (retained != B),
                                       or a SnapKV prompt not in increasing position order */
#define SE_DEVERR_BAD_INTERVAL  32u /* se_prune_interval: an interval wider than the mask
                                       row, or a negative budget                           */

/* Flags of se_decode_attend. */
#define SE_ATTEND_ACCUMULATE 1u /* fused H2O score update (eq. background-h2o-score)   */

/* Flags of se_quest_select. */
#define SE_QUEST_SCORES_GIVEN 1u /* skip the bound; select from page_scores (input)   */

/* Flags of se_snapkv_compact. */
#define SE_SNAPKV_SCORE_ONLY 1u /* write the pooled scores; retain and compact nothing */

/* Operation ids for se_workspace_bytes. */
#define SE_OP_DECODE_ATTEND 1
#define SE_OP_QUEST_SELECT  2
#define SE_OP_QUEST_STEP    3
#define SE_OP_SNAPKV        4
#define SE_OP_OMNIKV_SELECT 5
#define SE_OP_H2O_PREFILL   6

/* The cache view (Section 3.1, eq. attention-view; Appendix B, "Attention View
 * Payloads").  Only the pointers an operation needs must be non-NULL. */
typedef struct se_kv_view {
  void*          kv_pool;     /* bf16 [num_pages][2][page_size][head_dim]: K block, V block */
  int32_t*       pos_pool;    /* int32 [num_pages][page_size]: logical position per slot    */
  float*         score_pool;  /* fp32 [num_pages][page_size]: H2O accumulated score, or NULL */
  void*          meta_pool;   /* bf16 [num_pages][2][head_dim]: Quest per-page min, max, or NULL */
  const int32_t* block_table; /* int32 [num_units][max_pages]: physical page of each logical page */
  int32_t*       lengths;     /* int32 [num_units]: resident slots, updated on the device   */
  int64_t        num_pages;   /* pages in the pools (bounds for block-table entries)        */
  int32_t        num_units;   /* requests * num_kv_heads                                    */
  int32_t        num_kv_heads;
  int32_t        max_pages;   /* block-table row length; a unit holds <= max_pages*16 slots */
  int32_t        page_size;   /* must be 16                                                 */
  int32_t        head_dim;    /* 64 or 128                                                  */
} se_kv_view;

/*
 * se_decode_attend — append the decode token, then attention over the view.
 *
 * Per unit, with L the value of lengths[unit] on entry:
 *  1. Append (when k_new and v_new are both non-NULL): the new token's key and value
 *     go to slot L, pos_pool gets new_pos[req], score_pool (if non-NULL) gets 0,
 *     meta_pool (if non-NULL) folds the key into its page's min/max (a fresh page
 *     starts from the key), and lengths[unit] becomes L + 1 (Appendix A.3: the
 *     available set is the retained set plus the new token, which starts with
 *     score zero; Quest: a new key updates its page's extrema).
 *  2. Attention (Appendix A.1, eq. background-selected-attention) for each of the
 *     G query rows of the unit over its read set S:
 *       sel_pages == NULL: S = every resident slot (H2O: the whole available set);
 *       otherwise S = the slots of the logical pages sel_pages[unit][0..top_k)
 *       (entries < 0 are skipped; each must be a page below the current one) plus
 *       the current page, the page of the newest resident slot (Quest).
 *     z_j = scale * <q, k_j>, out = sum_j softmax_S(z)_j v_j, lse = log sum_j e^{z_j}.
 *  3. With SE_ATTEND_ACCUMULATE (needs score_pool): every slot of S gets its weight
 *     summed over the unit's G query heads added to its score (eq.
 *     background-h2o-score; GQA reading: sum over the group).
 *
 *  q        bf16 [num_req][num_kv_heads * q_per_kv][head_dim]
 *  k_new,
 *  v_new    bf16 [num_req][num_kv_heads][head_dim], or both NULL (no append)
 *  new_pos  int32 [num_req], needed with an append
 *  sel_pages int32 [num_units][top_k] logical page ids, or NULL
 *  scale    logit scale, normally 1/sqrt(head_dim) rounded to float32
 *  max_len  upper bound on the resident slots of any unit after the append; sizes
 *           the launch.  A unit above it sets SE_DEVERR_BAD_LENGTH and is skipped.
 *           So does an empty unit without an append (nothing to attend): its rows
 *           of out and lse are left as they were.  With an append an empty unit
 *           holds one slot and attends it (out = its value row).
 *  out      fp32 [num_req][num_kv_heads * q_per_kv][head_dim]
 *  lse      fp32 [num_req][num_kv_heads * q_per_kv], or NULL
 *  logits   fp32 [num_units][q_per_kv][logits_stride] (z per slot), or NULL; only
 *           with sel_pages == NULL; logits_stride >= max_len
 *  ws       device workspace of se_workspace_bytes(SE_OP_DECODE_ATTEND, ...) bytes (no
 *           initial contents needed).  Not shared between calls that may overlap.
 *  dev_err  int32 device word (see SE_DEVERR_*), never NULL
 */
se_status se_decode_attend(const se_kv_view* kv, int32_t q_per_kv, const void* q,
                           const void* k_new, const void* v_new, const int32_t* new_pos,
                           const int32_t* sel_pages, int32_t top_k, float scale,
                           int32_t max_len, uint32_t flags, float* out, float* lse,
                           float* logits, int32_t logits_stride, void* ws, size_t ws_bytes,
                           int32_t* dev_err, hipStream_t stream);

/*
 * se_accumulate_scores — the H2O score update as its own pass (eq.
 * background-h2o-score): for every unit and every resident slot j < lengths[unit],
 *   score(j) += sum over the unit's G query heads a of exp(logits[unit][a][j] - lse[a]).
 * logits and lse are those se_decode_attend wrote in the same step (all-slots mode).
 *  logits fp32 [num_units][q_per_kv][logits_stride]; lse fp32 [num_req][Hq]
 *  max_len upper bound on lengths[unit]; a unit above it sets SE_DEVERR_BAD_LENGTH.
 */
se_status se_accumulate_scores(const se_kv_view* kv, int32_t q_per_kv, const float* logits,
                               int32_t logits_stride, const float* lse, int32_t max_len,
                               int32_t* dev_err, hipStream_t stream);

/*
 * se_evict_compact — H2O retention and in-place compaction (Appendix A.3, eq.
 * background-h2o-retention; Section 3.1: eviction updates the retained-slot mapping
 * and the context length, then releases the discarded slots).
 * Per unit with L = lengths[unit] > budget (otherwise nothing changes):
 *   W = the min(recent, budget) slots with the largest positions;
 *   keep W plus the best budget - |W| other slots by (score desc, position asc);
 *   holes = evicted slots below budget (ascending), movers = kept slots at or above
 *   budget (ascending); the k-th mover's key, value, position and score move into
 *   the k-th hole; lengths[unit] = budget.
 *  freed_pages int32 [num_units][freed_stride] or NULL: receives the physical ids of
 *              the unit's pages that hold no slot afterwards, i.e. logical pages
 *              ceil(budget/16) .. ceil(L/16)-1 in order; freed_count[unit] (int32,
 *              may be NULL) their number (0 when nothing was evicted).  The block
 *              table is not modified: a caller that hands these pages to another
 *              owner must install a fresh page before a later append reaches them.
 *  budget  1 .. 8192; recent >= 0; max_len an upper bound on lengths[unit].
 */
se_status se_evict_compact(const se_kv_view* kv, int32_t budget, int32_t recent,
                           int32_t max_len, int32_t* freed_pages, int32_t freed_stride,
                           int32_t* freed_count, int32_t* dev_err, hipStream_t stream);

/*
 * se_decode_step_h2o — one H2O decode step of one layer in one call: exactly the
 * effect of se_decode_attend (with k_new/v_new, all resident slots read,
 * SE_ATTEND_ACCUMULATE) followed by se_evict_compact(budget, recent) — the
 * attention of the step and its finish_step work (Section 3.1, "Fine-Grained
 * Lifecycle Hooks": H2O's cumulative-score update and online eviction at the end
 * of a decode step; Appendix A.3, eqs. background-h2o-score and
 * background-h2o-retention).  The eviction runs in the epilogue of the attention
 * pass (one launch): a unit one slot over the budget whose recent window is the run
 * of its newest positions (every step after the first eviction) evicts from
 * registers; any other unit over the budget runs the general selection there.
 *  Arguments as for se_decode_attend and se_evict_compact; ws is the
 *  SE_OP_DECODE_ATTEND workspace.  budget 1 .. 8192.
 */
se_status se_decode_step_h2o(const se_kv_view* kv, int32_t q_per_kv, const void* q,
                             const void* k_new, const void* v_new, const int32_t* new_pos,
                             float scale, int32_t budget, int32_t recent, int32_t max_len,
                             float* out, float* lse, int32_t* freed_pages, int32_t freed_stride,
                             int32_t* freed_count, void* ws, size_t ws_bytes, int32_t* dev_err,
                             hipStream_t stream);

/*
 * se_decode_step_h2o_noalloc — se_decode_step_h2o for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): the same step, bit for bit, with the
 * workspace taken from a static device array of se_static_scratch_bytes()
 * bytes (256 MiB) that the library holds on each GPU it runs on until the
 * process ends.  The call allocates nothing; the first call on a device looks
 * up that device's copy of the array.
 *  Arguments as for se_decode_step_h2o without ws / ws_bytes.
 *  Returns SE_ERR_WORKSPACE when se_workspace_bytes(SE_OP_DECODE_ATTEND,
 *  num_units, max_len, max_pages, q_per_kv, head_dim, 0) exceeds the array
 *  (for example 512 units of 32769 slots need 289 MB; a steady 4096-slot step
 *  of 2048 units needs 147 MB).  Every call on one GPU shares the array, so
 *  calls that may overlap on one GPU (different streams, or concurrent host
 *  threads) race: serialize them.  The array needs no initial contents.
 */
se_status se_decode_step_h2o_noalloc(const se_kv_view* kv, int32_t q_per_kv, const void* q,
                                     const void* k_new, const void* v_new, const int32_t* new_pos,
                                     float scale, int32_t budget, int32_t recent, int32_t max_len,
                                     float* out, float* lse, int32_t* freed_pages, int32_t freed_stride,
                                     int32_t* freed_count, int32_t* dev_err, hipStream_t stream);

/* Bytes of the static device array se_decode_step_h2o_noalloc uses. */
size_t se_static_scratch_bytes(void);

/*
 * se_quest_summarize — per-page key min/max for every resident page (Appendix A.3,
 * eq. background-quest-summary): for each unit and logical page b < ceil(L/16),
 * meta_pool[page][0][c] = min and [1][c] = max of k[c] over the page's slots < L.
 * Used once after prefill; se_decode_attend maintains the summaries afterwards.
 */
se_status se_quest_summarize(const se_kv_view* kv, int32_t max_len, int32_t* dev_err,
                             hipStream_t stream);

/*
 * se_quest_select — Quest page selection (Appendix A.3, eq. background-quest-score).
 * Called before the step's se_decode_attend, with the current decode query.  With
 * L = lengths[unit], the token about to be appended opens or continues page
 * floor(L/16), the current page, which is always read; the candidates are the pages
 * [0, floor(L/16)).  For candidate b and query row a of the group:
 *   zhat_a(b) = scale * sum_c max(q_a[c] * min_b[c], q_a[c] * max_b[c]),
 * the page score is max over the group's rows (GQA reading), and sel_pages[unit]
 * receives the top_k candidates by (score desc, page index asc), in ascending page
 * order, padded with -1 when there are fewer candidates than top_k.
 *  q           bf16 [num_req][num_kv_heads * q_per_kv][head_dim]
 *  sel_pages   int32 [num_units][top_k] (output)
 *  page_scores fp32 [num_units][scores_stride], or NULL: receives the page scores of
 *              the candidates; with SE_QUEST_SCORES_GIVEN it is the input instead and
 *              the bound is not computed (q may then be NULL).
 *  top_k       1 .. 4096; max_len an upper bound on lengths[unit];
 *              scores_stride >= max_pages.
 *  ws          se_workspace_bytes(SE_OP_QUEST_SELECT, ...) bytes (no zero-fill needed)
 */
se_status se_quest_select(const se_kv_view* kv, int32_t q_per_kv, const void* q, float scale,
                          int32_t top_k, int32_t max_len, uint32_t flags, int32_t* sel_pages,
                          float* page_scores, int32_t scores_stride, void* ws, size_t ws_bytes,
                          int32_t* dev_err, hipStream_t stream);

/*
 * se_decode_step_quest — one Quest decode step of one layer in one call: exactly the
 * effect of se_quest_select (page bounds from the min/max summaries, top_k pages per
 * unit, written to sel_pages) followed by se_decode_attend with that selection
 * (append, attention over the selected pages and the current page) — Section 3.1:
 * selection before attention, changing only what attention reads; Appendix A.3,
 * eq. background-quest-score.  When every unit is read by one work-group and a
 * unit has at most 4608 candidate pages, the selection runs inside the attention
 * kernel (one launch; the candidates' scores stay in LDS); otherwise the two calls
 * run in order.
 *  Arguments as for se_quest_select and se_decode_attend (k_new/v_new/new_pos may be
 *  NULL together: no append).  sel_pages int32 [num_units][top_k] (output).
 *  ws  se_workspace_bytes(SE_OP_QUEST_STEP, ..., top_k) bytes (no zero-fill needed).
 */
se_status se_decode_step_quest(const se_kv_view* kv, int32_t q_per_kv, const void* q,
                               const void* k_new, const void* v_new, const int32_t* new_pos,
                               float scale, int32_t top_k, int32_t max_len, int32_t* sel_pages,
                               float* out, float* lse, void* ws, size_t ws_bytes, int32_t* dev_err,
                               hipStream_t stream);

/*
 * se_snapkv_compact — SnapKV prompt compaction after the last prefill chunk
 * (Appendix A.3, "SnapKV: Prompt Selection from an Observation Window", eqs.
 * background-snapkv-score and background-snapkv-retention; Section 3.1: SnapKV's
 * selection and eviction in finish_step after the final prompt chunk).  For every
 * unit with L = lengths[unit] > budget (other units are not touched):
 *   O = the last `window` slots, which hold the largest positions: the unit's slots
 *       must hold strictly increasing positions (a prefilled prompt), else
 *       SE_DEVERR_BAD_POSITIONS is raised and the unit is compacted on unspecified
 *       scores;
 *   u(j) = sum over the window positions t and the group's query heads a of
 *       softmax_j(scale * q_{t,a} . k_j) over the slots j with pos_j <= pos of O[t]
 *       (causal attention of the observation queries; the group's heads summed);
 *   s(j) = max of u over the candidates (slots outside O) whose positions are
 *       within kernel/2 of pos_j, for every candidate j (max pooling of width
 *       `kernel`);
 *   score_pool receives s on the candidates and 0 on O; then, unless
 *   SE_SNAPKV_SCORE_ONLY, exactly se_evict_compact(budget, recent = window): O plus
 *   the budget - window candidates with the largest s (ties: lower position) are
 *   kept and compacted into slots [0, budget), and lengths[unit] = budget.
 *  q_obs   bf16 [num_req][window][num_kv_heads * q_per_kv][head_dim]: the query of
 *          every head at the window's positions, in increasing position order (the
 *          prefill computed them); query head a belongs to KV head a / q_per_kv.
 *  window  1 .. budget, window * q_per_kv <= 1024 (above 128 rows the scores are summed over
 *          row blocks of 128 rows, and the workspace query needs top_k = window);
 *          kernel odd, 1 .. 31;
 *  scale   > 0 (softmax scale, usually 1/sqrt(head_dim)); budget window .. 8192;
 *  flags   0 or SE_SNAPKV_SCORE_ONLY (freed_* are then unused);
 *  freed_pages, freed_stride, freed_count, max_len as for se_evict_compact;
 *  ws      se_workspace_bytes(SE_OP_SNAPKV, num_units, max_len, max_pages, q_per_kv,
 *          head_dim, window) bytes (no zero-fill needed).
 */
se_status se_snapkv_compact(const se_kv_view* kv, int32_t q_per_kv, const void* q_obs,
                            int32_t window, int32_t kernel, float scale, int32_t budget,
                            int32_t max_len, uint32_t flags, int32_t* freed_pages,
                            int32_t freed_stride, int32_t* freed_count, void* ws, size_t ws_bytes,
                            int32_t* dev_err, hipStream_t stream);

/*
 * se_h2o_prefill_chunk — H2O's chunk-wise eviction during chunked prefill (Section 3.1:
 * finish_step after a prefill chunk; Appendix A.3, eqs. background-h2o-score and
 * background-h2o-retention; Appendix D: prefill scores from a scoring window).  Called
 * after the chunk's keys, values and positions were written to the last chunk_len slots
 * of each unit (lengths[unit] = L includes them; their positions increase and exceed
 * every older resident position).  For every unit:
 *   the chunk's slots start from score 0; the scoring queries are the chunk's last
 *   score_window positions: query t (t = 0 .. s-1) reads every slot up to its own
 *   position -- all older slots and the chunk's slots up to it -- and every slot it
 *   reads gains its weight summed over the group's G query heads (as a decode
 *   step's update, eq. background-h2o-score, for each of the s queries);
 *   then exactly se_evict_compact(budget, recent) (units with L <= budget keep all).
 *  q_score      bf16 [num_req][score_window][num_kv_heads * q_per_kv][head_dim], query t
 *               of the chunk's (chunk_len - score_window + t)-th position
 *  score_window 1 .. chunk_len, score_window * q_per_kv <= 1024; a unit with L <
 *               chunk_len sets SE_DEVERR_BAD_LENGTH and its scores are not updated
 *               (the eviction still applies to it)
 *  scale, budget, recent, max_len, freed_* as for se_evict_compact; max_len <= 131072;
 *               a budget of at least max_len may exceed se_evict_compact's 8192: no unit
 *               evicts, so the call only scores the chunk
 *  ws           se_workspace_bytes(SE_OP_H2O_PREFILL, num_units, max_len, max_pages,
 *               q_per_kv, head_dim, score_window) bytes (no zero-fill needed)
 */
se_status se_h2o_prefill_chunk(const se_kv_view* kv, int32_t q_per_kv, const void* q_score,
                               int32_t score_window, int32_t chunk_len, float scale, int32_t budget,
                               int32_t recent, int32_t max_len, int32_t* freed_pages,
                               int32_t freed_stride, int32_t* freed_count, void* ws, size_t ws_bytes,
                               int32_t* dev_err, hipStream_t stream);

/*
 * se_omnikv_select — OmniKV's observation-layer selection (Appendix A.3, "OmniKV:
 * Selection Reuse across Layers", eq. background-omnikv-selection), from the logits
 * se_decode_attend wrote for every resident slot of this layer in the same step
 * (all-slots mode, after the step's append).  Per request, with L = lengths of its
 * units (every KV head of a request holds the same slots; unequal lengths raise
 * SE_DEVERR_BAD_LENGTH and select nothing):
 *   s(j) = max over the request's Hq = num_kv_heads * q_per_kv query heads a of
 *          logits[unit(a)][a mod q_per_kv][j], for slots j < L;
 *   sel_slots[req] = the budget slots with the largest s (ties: lower slot), in
 *          increasing order; every slot followed by -1 when L <= budget.
 *  logits    fp32 [num_units][q_per_kv][logits_stride] as se_decode_attend writes it
 *  sel_slots int32 [num_req][budget] (output); budget 1 .. 8192; q_per_kv 1 .. 8
 *  ws        se_workspace_bytes(SE_OP_OMNIKV_SELECT, num_units / num_kv_heads, max_len,
 *            ...) bytes (no zero-fill needed)
 */
se_status se_omnikv_select(const se_kv_view* kv, int32_t q_per_kv, const float* logits,
                           int32_t logits_stride, int32_t budget, int32_t max_len,
                           int32_t* sel_slots, void* ws, size_t ws_bytes, int32_t* dev_err,
                           hipStream_t stream);

/*
 * se_attend_slots — a sparse layer's decode step under OmniKV's reuse (Appendix A.3,
 * eq. background-omnikv-reuse; Appendix A.1, eq. background-selected-attention with
 * S = the selection): the append of se_decode_attend (when k_new and v_new are given),
 * then for every unit the G query rows attend over S = the slots sel_slots[req][i]
 * (i < sel_count) of the unit's own cache — the slots an observation layer selected,
 * shared by the request's KV heads.  Entries < 0 are skipped; an entry at or past the
 * unit's length (after the append) sets SE_DEVERR_BAD_SELECTION and is skipped.  An
 * empty S gives out = 0 and lse = -inf.
 *  q, k_new, v_new, new_pos, scale, max_len, out, lse as for se_decode_attend;
 *  sel_slots int32 [num_req][sel_count], sel_count 1 .. 8192; q_per_kv 1, 2, 4 or 8.
 *  No workspace; the score field is not touched.
 */
se_status se_attend_slots(const se_kv_view* kv, int32_t q_per_kv, const void* q, const void* k_new,
                          const void* v_new, const int32_t* new_pos, const int32_t* sel_slots,
                          int32_t sel_count, float scale, int32_t max_len, float* out, float* lse,
                          int32_t* dev_err, hipStream_t stream);

/* Workspace bytes an operation needs for these sizes (0 if none).  op is one of
 * SE_OP_*; max_len as passed to the call; top_k for SE_OP_DECODE_ATTEND with a
 * selection and for SE_OP_QUEST_STEP (0 otherwise).  For SE_OP_OMNIKV_SELECT,
 * num_units is the number of requests; for SE_OP_H2O_PREFILL, top_k is the score
 * window. */
size_t se_workspace_bytes(int32_t op, int32_t num_units, int32_t max_len, int32_t max_pages,
                          int32_t q_per_kv, int32_t head_dim, int32_t top_k);

/* Waits for `stream`, copies the device error word to *host_out and clears it. */
se_status se_read_device_errors(int32_t* dev_err, int32_t* host_out, hipStream_t stream);

/* A static string naming a status. */
const char* se_status_string(se_status status);

/* Library version as MAJOR*10000 + MINOR*100 + PATCH. */
int32_t se_version(void);

/* se_probe_read_pages — a measurement aid, not a step of the method (no passage of
 * the paper defines it): the plain read rate of a page gather, which bounds what an
 * HBM-bound kernel reading the same pages can reach.  Reads all page_bytes bytes of
 * each page pages[0 .. n_pages) of `pool` (pool_pages pages of page_bytes bytes;
 * entries outside [0, pool_pages) read page 0) with the decode stream's 16-byte
 * nontemporal loads, on `grid` work-groups of 512 threads, and stores one XOR fold
 * per thread in sink (uint32 [grid * 512], written, never read).  The call's time
 * over n_pages * page_bytes is the read rate.
 *  page_bytes must be 8192 (a 16-slot page at d = 128); grid >= 1; n_pages >= 1.
 *  Errors: null pointers or other sizes -> SE_ERR_INVALID_ARGUMENT. */
se_status se_probe_read_pages(const void* pool, int64_t pool_pages, const int32_t* pages, int64_t n_pages,
                              int32_t page_bytes, int32_t grid, uint32_t* sink, hipStream_t stream);

/*
 * se_prune_interval — sparsity-based prefix-cache pruning of a history interval
 * (Section 3.2, "Sparsity-Based Prefix-Cache Pruning", eq. prefix-pruning; Appendix C.2,
 * "Pruning Metadata and Cache Operations").  For every unit, with L = lengths[unit],
 * T = the logical positions lo <= p < hi (interval[unit] = {lo, hi}, zero-based; lo >= hi
 * is an empty interval) and R the unit's resident positions:
 *   I = the positions of R within T that stay:
 *       mask mode (keep_mask != NULL): position p stays iff
 *         keep_mask[unit * mask_stride + (p - lo)] != 0 (entries of positions that are
 *         not resident are ignored); hi - lo must not exceed mask_stride;
 *       budget mode (keep_budget != NULL, needs score_pool): the keep_budget[unit] slots
 *         of T with the largest score_pool values stay (equal scores: lower position);
 *         all of them when T holds fewer, none for 0 (a retention ratio r over a fully
 *         resident interval is the budget r * (hi - lo), rounded by the caller);
 *   R' = (R \ T) u I.  The slots of R' keep their relative slot order and close up
 *   into slots [0, |R'|) with their key, value, position and score (positions are
 *   not renumbered: the logical prefix is unchanged); lengths[unit] = |R'|.
 *   Quest summaries (meta_pool != NULL) of the pages from the interval's first slot
 *   on are rebuilt.  Logical pages ceil(|R'|/16) .. ceil(L/16)-1 hold no resident slot
 *   afterwards: their physical ids go to freed_pages[unit][0..n) with n in
 *   freed_count[unit] (either may be NULL); a unit that loses nothing reports 0.
 * The caller applies it to idle units only: no other call on those units may be in
 * flight (Appendix C.2: pruning touches only blocks without active references).
 * Positions within a unit must be distinct.
 *  interval     int32 [num_units][2] (device)
 *  keep_mask    uint8 [num_units][mask_stride] (device) or NULL
 *  keep_budget  int32 [num_units] (device) or NULL; exactly one of the two
 *  max_len      bound on every unit's length, <= 131072; a unit above it, or an
 *               interval/budget the mode rejects, sets a device error bit and is
 *               left unchanged
 *  freed_stride >= max_pages when freed_pages is given
 */
se_status se_prune_interval(const se_kv_view* kv, const int32_t* interval, const uint8_t* keep_mask,
                            int32_t mask_stride, const int32_t* keep_budget, int32_t max_len,
                            int32_t* freed_pages, int32_t freed_stride, int32_t* freed_count,
                            int32_t* dev_err, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* SPARSE_ENGINE_H */
