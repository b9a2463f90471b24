/*
 * actkv.h -- C ABI of libactkv, the MI355X (gfx950) library for the compression step of
 * ActKV's action-oriented KV-cache eviction ("ActKV: Efficient LLM Agents through
 * Action-Guided KV Cache Management").
 *
 * The step standardises compression into three primitives (Sec. 3.3):
 *     AttnScore <- CalAttn(target queries, K cache)          actkv_score
 *     KeepMask  <- Eviction(AttnScore, Budget)               actkv_select
 *     KVCache   <- Compaction(KVCache, KeepMask)             actkv_compact (fresh pages)
 *                                                            actkv_compact_inplace (Alg. 4)
 * and actkv_step / actkv_step_inplace run all three back to back on one stream;
 * actkv_lrfu_select / actkv_step_lrfu evict by LRFU keep scores (Sec. 5.1).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Pointers are DEVICE pointers unless the name ends in _h (host memory).
 *  - bf16 tensors are passed as void* and hold IEEE bfloat16 values.
 *  - The paged cache (Sec. 2.5) is bf16 kv_cache[2][num_pages][page_size][num_kv_heads]
 *    [head_dim]: index 0 holds K, index 1 holds V.  Logical token t of request r lives in
 *    physical page block_table[r * bt_stride + t / page_size], slot t % page_size.
 *  - Query head g belongs to KV head g / G, G = num_q_heads / num_kv_heads (GQA groups,
 *    Alg. 3 input GQAGroup).
 *  - Action query j of request r (0 <= j < q_lens[r]) is row (sum_{r'<r} q_lens[r'] + j)
 *    of q; it sits at token position seq_lens[r] - q_lens[r] + j and, when causal, sees
 *    keys t <= that position.  Non-causal queries see all seq_lens[r] keys.
 *  - Scores are one fp32 per (request, KV head, token), ragged and concatenated in
 *    (r, h, t) order: request r's head h segment starts at Hkv * sum_{r'<r} L_r' + h * L_r.
 *  - Kept indices are int32 token indices, ascending within each (request, KV head),
 *    concatenated in (r, h) order; segment (r, h) holds k_rh = min(budget_rh, L_r)
 *    entries.
 *  - Ownership: the caller owns every buffer, including the workspace whose size
 *    actkv_query reports.  The library allocates no device memory and keeps no pointer to
 *    a caller's buffer after a call returns.  Its process-wide state: caches of the CU count
 *    per device and of per-kernel occupancy figures (written once, with atomics), the
 *    kernels' dynamic-LDS limits (set before a launch that needs more than 64 KiB), the
 *    overlap setting of actkv_set_overlap, a second stream and its events per device
 *    (created the first time a step is pipelined), and actkv_step_noalloc's static device
 *    array.  Concurrent calls are safe as long as their buffers do not overlap (calls of
 *    actkv_step_noalloc on one device share its array: see there).
 *  - Asynchrony: each call validates its arguments on the host, then enqueues kernels on
 *    `stream` (a hipStream_t; NULL is the default stream) and returns without
 *    synchronising.  Outputs are valid once the stream reaches that point.
 *  - Errors: every argument error is detected on the host before anything is enqueued,
 *    and then nothing is written.  ACTKV_ERR_HIP reports a failed kernel launch.  Faults
 *    inside kernels surface at the caller's next synchronisation.
 *  - Unspecified results (never a fault): block-table or free-list entries outside
 *    [0, num_pages) are not dereferenced -- the keys behind them read as zero and the
 *    compacted slots they would feed are left unwritten.
 *  - Undefined behaviour: non-finite q or K, device mirrors that disagree with the host
 *    mirrors, fresh pages that are still live, and buffers that overlap where the text
 *    says they must not.
 */
#ifndef ACTKV_H
#define ACTKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum actkv_status {
  ACTKV_OK = 0,
  ACTKV_ERR_INVALID_ARGUMENT = -1,    /* shapes, lengths, flags or pointers out of contract */
  ACTKV_ERR_UNSUPPORTED = -2,         /* valid request the library does not handle         */
  ACTKV_ERR_WORKSPACE_TOO_SMALL = -3, /* workspace_bytes below actkv_query's figure        */
  ACTKV_ERR_OUT_OF_PAGES = -4,        /* free list shorter than the fresh pages needed     */
  ACTKV_ERR_HIP = -5                  /* a HIP launch or runtime call failed               */
} actkv_status;

typedef enum actkv_agg {
  /* sum over the G query heads of a KV head and over the action queries */
  ACTKV_AGG_SUM = 0,
  /* max over the G query heads, mean over the action queries (Alg. 3 steps 4-5 and the
   * running mean of Sec. 7.1); needs G in {1, 2, 4, 8, 16} */
  ACTKV_AGG_MAX_MEAN = 1
} actkv_agg;

/*
 * One compression step over one layer for a batch of requests (Alg. 3 inputs Q,
 * PagedKV, BlockTable, LSE, GQAGroup, ActionReq; Alg. 4 inputs SeqUsedK, B, BlockSize;
 * Alg. 1 input B).  The batch passed in IS the set of requests being compressed.
 */
typedef struct actkv_problem {
  int32_t num_reqs;         /* R >= 0                                                    */
  int32_t num_q_heads;      /* Hq > 0, a multiple of num_kv_heads                        */
  int32_t num_kv_heads;     /* Hkv: 1..64                                                */
  int32_t head_dim;         /* D: 64 or 128                                              */
  int32_t page_size;        /* slots per page: 16                                        */
  int64_t num_pages;        /* physical pages in kv_cache                                */
  int32_t bt_stride;        /* block_table row stride (int32 elements), >= every
                               ceil(seq_lens[r] / page_size)                             */
  const int32_t* seq_lens_h;  /* host [R]: cached tokens L_r >= 0 (SeqUsedK)             */
  const int32_t* q_lens_h;    /* host [R]: action queries n_r >= 0 (<= L_r when causal)  */
  const int32_t* budgets_h;   /* host [R * Hkv]: entries to keep per (r, h), >= 0        */
  const int32_t* seq_lens_d;  /* device mirror of seq_lens_h                             */
  const int32_t* q_lens_d;    /* device mirror of q_lens_h                               */
  const int32_t* budgets_d;   /* device mirror of budgets_h                              */
  float sm_scale;           /* logits are sm_scale * q.k; 0 selects 1 / sqrt(head_dim)   */
  int32_t pool_window;      /* odd, 1..63: centred max-pool width over token positions;
                               1 = no pooling                                            */
  int32_t causal;           /* 1: causal visibility (see conventions), 0: all keys       */
  int32_t agg;              /* actkv_agg                                                 */
  uint32_t flags;           /* ACTKV_FLAG_*; 0 for the default behaviour                 */
} actkv_problem;

/*
 * ACTKV_FLAG_PLANNED: the workspace already holds this problem's per-request plan (the
 * offsets, page counts and scoring split every kernel reads), written by actkv_plan or by
 * any earlier call on the same problem and the same workspace; the call then does not plan
 * again.  Lets a caller that composes the stages (actkv_score, actkv_select, actkv_compact,
 * ...) plan once per step.  The plan carries a signature of the problem (its sizes and its
 * lengths, query counts and budgets); a kernel that finds a plan of another problem in the
 * workspace returns at once, so a wrong flag leaves the outputs unwritten, never a fault.
 */
#define ACTKV_FLAG_PLANNED 1u

/*
 * ACTKV_FLAG_SMALL_SELECT: TopK selection (actkv_select, actkv_step, actkv_step_inplace)
 * runs on the small-footprint kernel (256 threads and about 17 KB of LDS per segment, the
 * segment read from global memory in each pass) in place of the default one (1024 threads,
 * the segment held in LDS or registers).  Same results, bit for bit; slower alone (about
 * 95 us against 41 us for 128 segments of 35,000 entries on MI355X), but its small
 * register and LDS budget lets it run beside other kernels on another stream (the
 * pipelined actkv_step uses it for all groups but the last, whatever the flag).
 */
#define ACTKV_FLAG_SMALL_SELECT 2u

/*
 * Host-only planning (the per-request counts of Alg. 4, steps 1-5: Y = ceil(L_r /
 * page_size) blocks in use, X = ceil(k / page_size) blocks the survivors need; here k is
 * the largest per-head budget of the request, capped at L_r): no GPU work, callable
 * without a device.  Reports the workspace size the other calls need for `p` (the maximum
 * over them, so one workspace serves every entry point), the number of kept entries
 * sum_{r,h} min(budget, L_r), the fresh pages compaction pops from the free list (the sum
 * of X over compacted requests) and the pages it returns (the sum of Y over compacted
 * requests).  A request whose every head has budget >= L_r is left untouched by
 * compaction.  Errors: ACTKV_ERR_INVALID_ARGUMENT / ACTKV_ERR_UNSUPPORTED as for every
 * entry point, nothing written.  Any output pointer may be NULL.
 */
actkv_status actkv_query(const actkv_problem* p, size_t* workspace_bytes, int64_t* num_kept,
                         int64_t* fresh_pages_needed, int64_t* pages_freed);

/*
 * Writes the problem's plan into the workspace (the per-request counts and offsets of Alg. 4
 * steps 1-5 -- blocks in use, blocks kept, where each request's scores, kept entries, fresh
 * and freed pages start -- and the split of the scoring over the workgroups), for later
 * calls that pass ACTKV_FLAG_PLANNED.  Every other launching entry point plans by itself
 * unless that flag is set.  Errors as for every entry point.
 */
actkv_status actkv_plan(const actkv_problem* p, void* workspace, size_t workspace_bytes,
                        void* stream);

/*
 * Log-sum-exp of every action-query row (Sec. 7.1: LSE = log sum_j exp(s_ij) over the
 * keys the query sees), the normaliser a paged-attention backend produces as a
 * by-product.  q: bf16 [sum n][Hq][D]; lse_out: fp32 [sum n][Hq], natural log.
 */
actkv_status actkv_lse(const actkv_problem* p, const void* q, const void* kv_cache,
                       const int32_t* block_table, float* lse_out, void* workspace,
                       size_t workspace_bytes, void* stream);

/*
 * Recovery-based attention scoring (Sec. 7.1, Alg. 3): for every cached entry t of
 * request r and KV head h,
 *   SUM:      scores = sum_{g in group(h)} sum_{j sees t} exp(sm_scale q_jg . k_t - LSE_jg)
 *   MAX_MEAN: scores = (1/n_r) sum_{j sees t} max_{g in group(h)} exp(...)
 * lse: fp32 [sum n][Hq] natural-log LSE over the same keys and scale (the paper's input),
 * or NULL to have the library compute it first (actkv_lse into the workspace).
 * scores: fp32, ragged (see conventions).
 */
actkv_status actkv_score(const actkv_problem* p, const void* q, const void* kv_cache,
                         const int32_t* block_table, const float* lse, float* scores,
                         void* workspace, size_t workspace_bytes, void* stream);

/*
 * Streaming scoring (Alg. 3 as the paper runs it: one action query per request per decode
 * step, its LSE from that step's attention, the per-entry aggregate updated in place and
 * reset by the caller at the start of each action region): acc += the scores of this call,
 * as actkv_score would compute them (q_lens[r] = the new queries of request r, usually 1;
 * 0 adds nothing).  acc: fp32 in/out in the score layout of this call's seq_lens, 16-byte
 * aligned; when a sequence grows between steps the caller extends its segment with zeros
 * for the new entries.  n steps of one query each add up to one actkv_score call with all
 * n queries (SUM; with MAX_MEAN each step adds max over the group, so acc / n is the
 * running mean of Sec. 7.1).  A call with at most one query per request (a decode step)
 * and a group of at most 16 query heads is scored and added in one pass; otherwise the
 * step's scores pass through the workspace.  Either way each entry of acc is updated by
 * exactly one thread (no atomics): results do not depend on scheduling.
 */
actkv_status actkv_score_accumulate(const actkv_problem* p, const void* q, const void* kv_cache,
                                    const int32_t* block_table, const float* lse, float* acc,
                                    void* workspace, size_t workspace_bytes, void* stream);

/*
 * Eviction (Alg. 1 step 5, TopK(score, k = B)): per (request, KV head) the
 * k_rh = min(budget_rh, L_r) entries with the largest pooled score are kept, ties going
 * to the lower token index, and written ascending into `kept` ([num_kept] int32).
 * pooled (nullable): fp32, same layout as scores, receives the max-pooled scores
 * (pool_window 1 copies them; -0 is written as +0).  scores is not modified.  Scores may
 * be any fp32 values but NaN (NaN scores give unspecified selections, never a fault).
 */
actkv_status actkv_select(const actkv_problem* p, const float* scores, float* pooled,
                          int32_t* kept, void* workspace, size_t workspace_bytes,
                          void* stream);

/*
 * Fresh-page compaction (the compaction primitive of Sec. 3.3 with the freed-block
 * return of Sec. 7.2).  For each request in order that is not left untouched, with
 * X = ceil(max_h k_rh / page_size) and Y = ceil(L_r / page_size):
 *   fresh = free_pages[off .. off + X), off advancing over the compacted requests;
 *   for every head h and j < k_rh, the K and V rows of token kept[j] are copied bit for
 *   bit to page fresh[j / page_size], slot j % page_size (ascending token order);
 *   freed_pages receives the old block_table[r, 0..Y) (request order);
 *   block_table[r, 0..X) = fresh, block_table[r, X..Y) = -1 (rewritten in place);
 *   new_lens[r * Hkv + h] = k_rh.
 * Untouched requests keep their row, free nothing and get new_lens = L_r.  Slots of a
 * fresh page at or beyond k_rh (for head h) are left unwritten.  Only fresh pages are
 * written; old pages are returned intact.  free_pages must not contain live pages.
 * num_free < fresh_pages_needed gives ACTKV_ERR_OUT_OF_PAGES.  freed_pages holds
 * pages_freed entries (see actkv_query); new_lens is int32 [R * Hkv].
 */
actkv_status actkv_compact(const actkv_problem* p, void* kv_cache, int32_t* block_table,
                           const int32_t* kept, const int32_t* free_pages, int64_t num_free,
                           int32_t* freed_pages, int32_t* new_lens, void* workspace,
                           size_t workspace_bytes, void* stream);

/*
 * Eviction then fresh-page compaction (Alg. 1 steps 5 and 6): actkv_select followed by
 * actkv_compact on the kept entries, in one call.  Arguments as there; pooled and kept
 * may be NULL (kept in the workspace).  Results are those of the two calls, bit for bit.
 * For small problems (at most 32 (request, KV head) segments keeping at most 512 entries
 * each, and without ACTKV_FLAG_SMALL_SELECT) both run in a single kernel: one workgroup per
 * segment selects and then copies its own head's rows, and the last workgroup of a request
 * to finish rewrites its block-table row (a counter per request in the workspace; nothing
 * waits on another workgroup).
 */
actkv_status actkv_select_compact(const actkv_problem* p, const float* scores, float* pooled,
                                  int32_t* kept, void* kv_cache, int32_t* block_table,
                                  const int32_t* free_pages, int64_t num_free,
                                  int32_t* freed_pages, int32_t* new_lens, void* workspace,
                                  size_t workspace_bytes, void* stream);

/*
 * The whole step (Alg. 1 steps 1, 5 and 6): score -> select -> compact on `stream`.
 * scores, pooled and kept are optional outputs (NULL keeps them in the workspace);
 * lse may be NULL as in actkv_score.  The other arguments are as above.  Selection and
 * compaction run as in actkv_select_compact.
 * A large batch (several requests) is cut into request groups and pipelined: while group
 * g is scored on `stream`, group g - 1 is selected and compacted on a second stream that
 * the library creates on first use (one per device, default priority, never destroyed),
 * with events between the two; the call returns with `stream` waiting for all of it, so
 * work queued on `stream` afterwards sees the whole step.  Calls from several host threads
 * are serialised while they enqueue.  Results are identical, bit for bit, to the
 * unpipelined order.  See actkv_set_overlap.
 */
actkv_status actkv_step(const actkv_problem* p, const void* q, void* kv_cache,
                        int32_t* block_table, const float* lse, const int32_t* free_pages,
                        int64_t num_free, float* scores, float* pooled, int32_t* kept,
                        int32_t* freed_pages, int32_t* new_lens, void* workspace,
                        size_t workspace_bytes, void* stream);

/*
 * Tuning of actkv_step's pipelining, process-wide: groups = 0 (the default) chooses
 * automatically (at present: never, the sequential order measuring faster on MI355X);
 * 1 never pipelines; 2 .. ACTKV_MAX_OVERLAP_GROUPS pipelines every batch of at least two
 * requests in that many groups (fewer when there are fewer requests).  Other values: ACTKV_ERR_INVALID_ARGUMENT.  actkv_get_overlap
 * returns the current setting.  actkv_step_noalloc never pipelines.
 */
#define ACTKV_MAX_OVERLAP_GROUPS 8
actkv_status actkv_set_overlap(int32_t groups);
int32_t actkv_get_overlap(void);

/*
 * actkv_step for callers that cannot allocate: code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc.  Same arguments, results and errors as actkv_step,
 * but no workspace argument: the step's intermediates live in a static device array of
 * ACTKV_NOALLOC_SCRATCH_BYTES bytes inside the library, of which every GPU the library runs
 * on holds its own copy until the process ends.  Neither this call nor any kernel it
 * launches allocates or frees memory.  A problem whose workspace (actkv_query) exceeds the
 * array is refused with ACTKV_ERR_WORKSPACE_TOO_SMALL before anything else happens (the
 * array holds the 32 x 35,000-token, 32/4-head, d = 128, 64-query batch); ACTKV_ERR_HIP if
 * the array's device address cannot be looked up.  All calls on one GPU share that GPU's
 * array, so calls that overlap in time on one GPU (concurrent streams, or several host
 * threads) race: order them on one stream.  The array keeps the last call's contents; no
 * part of it needs to start at zero.
 */
#define ACTKV_NOALLOC_SCRATCH_BYTES (64u << 20)
actkv_status actkv_step_noalloc(const actkv_problem* p, const void* q, void* kv_cache,
                                int32_t* block_table, const float* lse,
                                const int32_t* free_pages, int64_t num_free, float* scores,
                                float* pooled, int32_t* kept, int32_t* freed_pages,
                                int32_t* new_lens, void* stream);

/*
 * Eviction with attention-aware LRFU keep scores (Sec. 5.1 keep-score update; Alg. 1
 * steps 2-5) in place of plain TopK on the scores.  Per (request, KV head):
 *   att     = the max-pooled scores (pool_window; 1 = the scores), also written to `pooled`
 *             when it is not NULL;
 *   hit     = the shortest prefix of the entries ordered by att descending (ties: lower
 *             token index first) whose mass reaches top_p times the segment's total
 *             (GetHitMask, step 3); none where that target is not positive; top_p = 1 hits
 *             every entry with att > 0.  att is a probability-like score: entries with
 *             att <= 0 carry no mass;
 *   ks      = decay * ks + (hit ? att : 0), in place, in fp32 with the product and the sum
 *             each rounded (step 4);
 *   kept    = the k_rh entries with the largest ks, ties to the lower token index, written
 *             ascending as in actkv_select (TopK on the keep scores, step 5);
 *   ks_kept = ks of the kept entries, in the order of `kept`: the keep scores that travel
 *             with the compacted K/V (KS' of Alg. 1).
 * ks: fp32 [num_scores] in/out, same layout as the scores; entries new since the last step
 * enter with 0 (step 2 is the caller's concatenation).  hit (nullable): uint8 [num_scores],
 * 1 = hit.  ks_kept: fp32 [num_kept].  top_p and decay in [0, 1] (else
 * ACTKV_ERR_INVALID_ARGUMENT).  ks must not overlap scores or pooled.  Segments longer than
 * 64,512 entries, or longer than 38,400 with a pool_window above 7: ACTKV_ERR_UNSUPPORTED.
 * The mass sums are exact 64-bit fixed-point sums of
 * the scores scaled by a power of two (deterministic); where the prefix boundary falls within
 * that resolution of the target, the boundary entry may differ from a floating-point
 * evaluation.
 */
actkv_status actkv_lrfu_select(const actkv_problem* p, const float* scores, float top_p,
                               float decay, float* ks, uint8_t* hit, float* pooled,
                               int32_t* kept, float* ks_kept, void* workspace,
                               size_t workspace_bytes, void* stream);

/*
 * The whole step with LRFU eviction (Alg. 1 steps 1-6): score -> actkv_lrfu_select ->
 * compact on `stream`.  Arguments as in actkv_step and actkv_lrfu_select; scores, pooled,
 * hit and kept are optional outputs (NULL keeps them in the workspace, hit NULL: not
 * written).
 */
actkv_status actkv_step_lrfu(const actkv_problem* p, const void* q, void* kv_cache,
                             int32_t* block_table, const float* lse, const int32_t* free_pages,
                             int64_t num_free, float top_p, float decay, float* ks,
                             float* ks_kept, float* scores, float* pooled, uint8_t* hit,
                             int32_t* kept, int32_t* freed_pages, int32_t* new_lens,
                             void* workspace, size_t workspace_bytes, void* stream);

/*
 * Host-only planning for the in-place compaction: the pages it returns, sum over compacted
 * requests of Y_r - X_r (Alg. 4: Y = ceil(L_r / page_size), X = ceil(max_h k_rh /
 * page_size)).  pages_freed may be NULL.
 */
actkv_status actkv_query_inplace(const actkv_problem* p, int64_t* pages_freed);

/*
 * In-place compaction (Alg. 4, conflict-free slot planning of Sec. 7.2): no free list and
 * no staging buffer.  For each request in order that is not left untouched, with
 * Y = ceil(L_r / page_size), X = ceil(max_h k_rh / page_size) (shared by the heads: a page
 * holds every head's row of a slot) and, per head h, Start = (Y - X) * page_size,
 * End = Start + k_rh:
 *   destinations = the logical slots of [Start, End) holding no kept entry, ascending
 *                  (slots at or past L_r in the last page count: they exist and are free);
 *   sources      = the kept entries outside [Start, End), ascending;
 *   the i-th source's K and V rows of head h are copied bit for bit to the i-th
 *   destination (through the block table as it was on entry).  Sources and destinations
 *   are disjoint, so every copy runs in one pass.
 * Afterwards head h's survivors occupy logical slots [Start, End), i.e. new slots
 * [0, k_rh) of the shortened row: block_table[r, 0..X) = old block_table[r, Y-X..Y),
 * block_table[r, X..Y) = -1; freed_pages receives the old block_table[r, 0..Y-X) (request
 * order; pages_freed entries from actkv_query_inplace); new_lens[r * Hkv + h] = k_rh.
 * Survivors do not stay in token order: new_order (nullable, int32 [num_kept], laid out like
 * kept) receives for every new slot j < k_rh the original token index now there, so
 * callers can carry per-entry state (e.g. the LRFU keep scores: next ks = ks_kept
 * permuted by it).  Untouched requests keep their row and get new_order = kept.
 * kept must be ascending within each (r, h) with entries in [0, L_r) (what actkv_select
 * and actkv_lrfu_select write); otherwise the result is unspecified (out-of-range entries
 * are never dereferenced).  Only destination rows are written.
 */
actkv_status actkv_compact_inplace(const actkv_problem* p, void* kv_cache, int32_t* block_table,
                                   const int32_t* kept, int32_t* freed_pages, int32_t* new_lens,
                                   int32_t* new_order, void* workspace, size_t workspace_bytes,
                                   void* stream);

/*
 * The whole step with the in-place compaction: score -> select -> actkv_compact_inplace on
 * `stream`.  Arguments as in actkv_step and actkv_compact_inplace (no free list).
 */
actkv_status actkv_step_inplace(const actkv_problem* p, const void* q, void* kv_cache,
                                int32_t* block_table, const float* lse, float* scores,
                                float* pooled, int32_t* kept, int32_t* freed_pages,
                                int32_t* new_lens, int32_t* new_order, void* workspace,
                                size_t workspace_bytes, void* stream);

/*
 * Token-level confidence (Sec. 6.1; Alg. 2 step 1, GetTokenConf): for every row r of
 * logits, the negative mean log-probability of the top_k most likely tokens,
 *   conf[r] = LSE(logits[r]) - (1/k) sum of the k largest logits[r][v],  k = min(top_k, vocab).
 * logits: fp32 [rows][row_stride] (the first `vocab` entries of each row are used; -inf
 * entries are masked tokens); conf: fp32 [rows].  top_k in 1..64 and vocab up to 262,144
 * (else ACTKV_ERR_UNSUPPORTED).  The log-sum-exp is accumulated in fp32 (fixed reduction
 * order: deterministic), the top-k sum in fp64.  workspace: at least the bytes
 * actkv_token_confidence_workspace reports.
 */
actkv_status actkv_token_confidence_workspace(int64_t rows, int64_t vocab, int32_t top_k,
                                              size_t* workspace_bytes);
actkv_status actkv_token_confidence(const float* logits, int64_t rows, int64_t vocab,
                                    int64_t row_stride, int32_t top_k, float* conf,
                                    void* workspace, size_t workspace_bytes, void* stream);

/*
 * Budget update before compression (Alg. 2 steps 2-4), per request r with token
 * confidences T = token_conf[offsets[r] .. offsets[r + 1]) (the trace so far):
 *   R'_m  = min T[m * stride .. m * stride + window), m = 0 .. (n - window) / stride;
 *   Q     = the bottom_pct-th percentile of R' by linear interpolation between order
 *           statistics (position bottom_pct / 100 * (M - 1));
 *   alpha = least-squares slope of R'_m against m over the windows with R'_m <= Q, sums in
 *           window order in fp64 (0 with fewer than two such windows or n < window);
 *   budgets_out[r] = min(floor(budgets_in[r] * scale_up), budget_upper) if alpha < 0, else
 *           budgets_in[r].
 * The call is made when compression triggers (the paper's TriggerCompress).  offsets:
 * int64 [num_reqs + 1] on the host (validation) and on the device; budgets int32 [num_reqs]
 * on the device (budgets_out may alias budgets_in); slopes, thresholds (fp64, NaN with no
 * window) and retained (int32 window counts) are optional device outputs.  At most 16,384
 * windows per request (ACTKV_ERR_UNSUPPORTED beyond).  The percentile, the sums and the
 * budget rule are evaluated in fp64 with every operation rounded on its own, so results
 * are reproducible bit for bit.
 */
actkv_status actkv_budget_update(const float* token_conf, const int64_t* offsets_h,
                                 const int64_t* offsets_d, int32_t num_reqs, int32_t window,
                                 int32_t stride, float bottom_pct, float scale_up,
                                 int32_t budget_upper, const int32_t* budgets_in,
                                 int32_t* budgets_out, double* slopes, double* thresholds,
                                 int32_t* retained, void* stream);

/* Static text for a status code. */
/*
 * Device-side check of what the fresh-page compaction takes on trust (the caller's
 * guarantee to actkv_compact and actkv_step: the copies of Sec. 7.2 are conflict-free only
 * when no page written is one that is read).  On `stream`, with the device mirrors of `p`:
 *   ACTKV_CHECK_MIRRORS     the device seq_lens, q_lens or budgets differ from the host ones
 *                           (compared through a 64-bit checksum of each array);
 *   ACTKV_CHECK_TABLE_RANGE an entry bt[r, 0 .. ceil(L_r / page_size)) lies outside
 *                           [0, num_pages);
 *   ACTKV_CHECK_FREE_RANGE  one of the pages the step would take, free_pages[0 ..
 *                           fresh_pages_needed), lies outside [0, num_pages);
 *   ACTKV_CHECK_FRESH_LIVE  one of them is live (appears in such a block-table entry);
 *   ACTKV_CHECK_FRESH_DUP   one of them appears twice.
 * The bits found are OR-ed into *status (device, uint32, set to 0 first); 0 means all of
 * it holds.  scratch: device memory of at least ACTKV_CHECK_SCRATCH_BYTES(num_pages) bytes
 * (two page bitmaps), overwritten.  Host errors as for actkv_compact (OUT_OF_PAGES when
 * num_free < fresh_pages_needed; WORKSPACE_TOO_SMALL for a short scratch), nothing enqueued
 * then.  The kernels only read the problem's arrays and never index with a page they have
 * not range-checked, so any content of them is safe to check.
 */
#define ACTKV_CHECK_MIRRORS 1u
#define ACTKV_CHECK_TABLE_RANGE 2u
#define ACTKV_CHECK_FREE_RANGE 4u
#define ACTKV_CHECK_FRESH_LIVE 8u
#define ACTKV_CHECK_FRESH_DUP 16u
#define ACTKV_CHECK_SCRATCH_BYTES(num_pages) (8u * (((size_t)(num_pages) + 31u) / 32u))
actkv_status actkv_check_pages(const actkv_problem* p, const int32_t* block_table,
                               const int32_t* free_pages, int64_t num_free, uint32_t* status,
                               void* scratch, size_t scratch_bytes, void* stream);

const char* actkv_status_str(actkv_status status);

#ifdef __cplusplus
}
#endif

#endif /* ACTKV_H */
