// Internal definitions shared by the libactkv host code and its HIP kernels.
// Nothing here is part of the public ABI (include/actkv.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "actkv.h"

namespace actkv {

constexpr int kPageSize = 16;        // slots per page (the only page size built)
constexpr int kRowsPerChunk = 512;   // query rows (G * n) one scoring pass holds on chip
constexpr int kKeyTile = 64;         // keys per scoring / LSE pipeline step (4 pages)
// Scoring cost of one 64-key tile of a row chunk, in units of 32 query rows: the scoring
// kernel adds rows in steps of kScoreRowStep (one 16-row tile in each of its 8 waves), so a
// chunk of `rows` rows costs its rows rounded up to that step, plus a fixed share per tile
// (the K gather, the barrier, the per-key finish) worth five units.  A chunk of at most half
// a step leaves every other wave idle, one busy wave per SIMD, and costs half a step.
// Workgroups split the scoring by this cost.  (Measured per workgroup on the ragged batches,
// a tile of <= 64, 128, 256, 384 and 512 rows takes 0.33, 0.44, 0.62, 0.79 and 1 times the
// time of a full one, which these costs, 7/21, 9/21, 13/21, 17/21 and 21/21, follow; rounding
// every chunk to 64-row steps instead was slower.)
constexpr int kScoreRowStep = 128;
constexpr int kTileCostFixed = 5;
__host__ __device__ constexpr int64_t score_tile_cost(int64_t units) { return units + kTileCostFixed; }
// 32-row units of one key tile of a row chunk holding `rows` query rows (a chunk with no
// row costs what one row costs)
__host__ __device__ constexpr int64_t chunk_units(int64_t rows) {
  return rows <= kScoreRowStep / 2
             ? kScoreRowStep / 64
             : ((rows < kRowsPerChunk ? rows : kRowsPerChunk) + kScoreRowStep - 1) /
                   kScoreRowStep * (kScoreRowStep / 32);
}
constexpr int kLseKeysPerBlock = 2048;  // keys one LSE workgroup reduces (32 key tiles)
constexpr int kMaxPoolWindow = 63;

// Per-request plan, written on the device by plan_kernel from the device mirrors.
struct ReqPlan {
  int32_t L, n;            // cached tokens, action queries
  int32_t X, Y;            // fresh pages popped / old pages returned (0 when untouched)
  int32_t skip;            // every head keeps everything: request left untouched
  int32_t nchunk;          // query-row chunks of kRowsPerChunk rows (>= 1)
  int32_t q_off;           // sum of n over earlier requests
  int32_t fresh_off;       // sum of X over earlier requests
  int32_t freed_off;       // sum of Y over earlier requests
  int32_t lse_blocks;      // ceil(L / kLseKeysPerBlock)
  int32_t ip_freed_off;    // sum of Y - X over earlier requests (in-place compaction)
  int64_t seg_off;         // Hkv * sum of L over earlier requests (score offset, head 0)
  int64_t lse_part_off;    // sum over earlier requests of n * Hq * lse_blocks
};

// Everything the host derives from the host mirrors before launching anything.
struct HostPlan {
  int32_t R = 0, Hq = 0, Hkv = 0, G = 0, D = 0;
  int32_t max_chunks = 1;
  int64_t sum_n = 0, sum_L = 0, num_scores = 0;
  int64_t num_kept = 0, fresh_needed = 0, pages_freed = 0;
  int64_t max_fresh = 0;          // most fresh pages (X) of one request
  int64_t max_k = 0;              // most kept entries of one (request, KV head)
  int64_t pages_freed_inplace = 0;  // sum of Y - X over compacted requests
  int64_t num_segments = 0;       // R * max_chunks * Hkv
  int64_t score_cost = 0;         // total scoring cost units (key tiles x row tiles)
  int64_t lse_parts = 0;          // sum_r n_r * Hq * lse_blocks_r
  int64_t max_lse_blocks = 0;     // max_r ceil(L_r / kLseKeysPerBlock)
  int64_t max_L = 0;              // longest request
  int64_t max_n = 0;              // most action queries of one request
};

// Byte offsets of the workspace regions (each 256-byte aligned).
struct WsLayout {
  size_t sig = 0;          // uint64: signature of the problem whose plan the workspace holds
  size_t plan = 0;         // ReqPlan[R]
  size_t kept_off = 0;     // int64[R * Hkv + 1]
  size_t seg_cost = 0;     // int64[num_segments + 1]
  size_t lse = 0;          // float[sum_n * Hq]
  size_t lse_part = 0;     // float2[lse_parts]
  size_t scores = 0;       // float[num_scores]
  size_t score_part = 0;   // float[(max_chunks - 1) * num_scores]
  size_t pooled = 0;       // float[num_scores]
  size_t kept = 0;         // int32[num_kept]
  size_t ip_src = 0;       // int32[num_kept]: in-place copy sources by rank, at kept_off
  size_t ip_order = 0;     // int32[num_kept]: in-place new slot order when the caller has none
  size_t req_done = 0;     // int32[R]: per-request counters of the fused selection+compaction
  size_t total = 0;
};

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Compute units of the current device (asked once per device; 256 if the query fails).
inline int device_cus() {
  static int cache[64] = {};   // 0: not asked yet
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int c = __atomic_load_n(&cache[dev], __ATOMIC_RELAXED);
  if (c > 0) return c;
  if (hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      c <= 0)
    c = 256;
  __atomic_store_n(&cache[dev], c, __ATOMIC_RELAXED);
  return c;
}

inline WsLayout ws_layout(const HostPlan& hp) {
  WsLayout w;
  size_t o = 0;
  auto take = [&](size_t bytes) { size_t at = o; o = align256(o + bytes); return at; };
  w.sig = take(sizeof(uint64_t));
  w.plan = take(sizeof(ReqPlan) * (size_t)(hp.R > 0 ? hp.R : 1));
  w.kept_off = take(sizeof(int64_t) * (size_t)(hp.R * hp.Hkv + 1));
  w.seg_cost = take(sizeof(int64_t) * (size_t)(hp.num_segments + 1));
  w.lse = take(sizeof(float) * (size_t)(hp.sum_n * hp.Hq));
  w.lse_part = take(2 * sizeof(float) * (size_t)hp.lse_parts);
  w.scores = take(sizeof(float) * (size_t)hp.num_scores);
  w.score_part = take(sizeof(float) * (size_t)(hp.max_chunks - 1) * (size_t)hp.num_scores);
  w.pooled = take(sizeof(float) * (size_t)hp.num_scores);
  w.kept = take(sizeof(int32_t) * (size_t)hp.num_kept);
  w.ip_src = take(sizeof(int32_t) * (size_t)hp.num_kept);
  w.ip_order = take(sizeof(int32_t) * (size_t)hp.num_kept);
  w.req_done = take(sizeof(int32_t) * (size_t)(hp.R > 0 ? hp.R : 1));
  w.total = o;
  return w;
}

// Common argument block for the device kernels.
struct DevProblem {
  int32_t R, Hq, Hkv, G, D;
  int64_t num_pages;
  int32_t bt_stride;
  int32_t max_chunks;
  int32_t pool_window;
  int32_t causal;
  int32_t agg;
  float sm_scale;
  const int32_t* seq_lens;
  const int32_t* q_lens;
  const int32_t* budgets;
  ReqPlan* plan;           // workspace
  int64_t* kept_off;       // workspace [R*Hkv + 1]
  int64_t* seg_cost;       // workspace [num_segments + 1]
  int64_t num_segments;
  uint64_t sig;            // signature of this problem (host-computed)
  uint64_t* plan_sig;      // workspace: signature of the problem the plan was written for
  int32_t* req_done;       // workspace [R]: zero between launches (see select_compact_kernel)
};


// Page and mirror check (actkv_check_pages): one term of the order-dependent checksum of a
// mirrored array (sum over i of term(i, v[i]), modulo 2^64), the same on host and device.
__host__ __device__ inline uint64_t mirror_term(int64_t i, int32_t v) {
  return (uint64_t)(uint32_t)v * (0x9E3779B97F4A7C15ull * (uint64_t)(i + 1));
}
// 32-bit words of one page bitmap.
__host__ __device__ inline int64_t check_bitmap_words(int64_t num_pages) {
  return (num_pages + 31) / 32;
}
// The check's kernels; scratch holds two bitmaps of check_bitmap_words(num_pages) words.
hipError_t launch_check_pages(const int32_t* seq_lens, const int32_t* q_lens,
                              const int32_t* budgets, int R, int Hkv, const int32_t* bt,
                              int bt_stride, int64_t num_pages, const int32_t* free_pages,
                              int64_t n_fresh, const uint64_t want[3], uint32_t* status,
                              uint32_t* scratch, hipStream_t s);

// The whole step (actkv_step) on a caller-chosen workspace: validation, planning and the
// launches of every stage.  actkv_step_noalloc passes its static scratch array and
// may_overlap = false (the overlapped form creates a stream and events on first use).
actkv_status step_impl(const actkv_problem* p, const void* q, void* kv_cache,
                       int32_t* block_table, const float* lse, const int32_t* free_pages,
                       int64_t num_free, float* scores, float* pooled, int32_t* kept,
                       int32_t* freed_pages, int32_t* new_lens, void* workspace,
                       size_t workspace_bytes, void* stream, bool may_overlap);

// Kernel launchers (each returns the hipGetLastError() of its launches).
hipError_t launch_plan(const DevProblem& dp, hipStream_t s);
hipError_t launch_lse(const DevProblem& dp, const HostPlan& hp, const void* q, const void* kv,
                      const int32_t* bt, float* lse_out, float2* lse_part, hipStream_t s);
hipError_t launch_score(const DevProblem& dp, const HostPlan& hp, const void* q,
                        const void* kv, const int32_t* bt, const float* lse, float* scores,
                        float* score_part, hipStream_t s);
// The scoring of requests [r0, r1), whose cost units sum to `cost` (the scoring kernel,
// then the row-chunk reduction of those requests when some request has several chunks).
hipError_t launch_score_range(const DevProblem& dp, const HostPlan& hp, int r0, int r1,
                              int64_t cost, const void* q, const void* kv, const int32_t* bt,
                              const float* lse, float* scores, float* score_part,
                              hipStream_t s);
// acc[i] += s[i], i < n (both 16-byte aligned or n handled element-wise at the tail).
hipError_t launch_accumulate(float* acc, const float* s, int64_t n, hipStream_t st);
// Decode-step scoring added straight into acc: every request has at most one action query
// and G <= kDecodeMaxGroup (the caller checks).
constexpr int kDecodeMaxGroup = 16;
hipError_t launch_score_decode(const DevProblem& dp, const HostPlan& hp, const void* q,
                               const void* kv, const int32_t* bt, const float* lse, float* acc,
                               hipStream_t s);
hipError_t launch_select(const DevProblem& dp, const HostPlan& hp, const float* scores,
                         float* pooled, int32_t* kept, hipStream_t s);
// The selection of requests [r0, r1) only: select_kernel (one 1024-thread workgroup per
// segment), or select_side_kernel (512 threads, few registers, small LDS: for running beside
// other kernels).  Both give the same pooled scores and kept indices.
hipError_t launch_select_range(const DevProblem& dp, const HostPlan& hp, int r0, int r1,
                               const float* scores, float* pooled, int32_t* kept,
                               hipStream_t s);
hipError_t launch_select_side(const DevProblem& dp, const HostPlan& hp, int r0, int r1,
                              const float* scores, float* pooled, int32_t* kept,
                              hipStream_t s);
// Selection and fresh-page compaction of every request in one kernel (select_compact_splits
// workgroups per segment, each selecting it and copying a share of its rows; the rewrite of
// a request by its last workgroup): the results of launch_select then launch_compact.
int select_compact_splits(const HostPlan& hp, int head_dim);
hipError_t launch_select_compact(const DevProblem& dp, const HostPlan& hp, const float* scores,
                                 float* pooled, int32_t* kept, void* kv, int32_t* bt,
                                 const int32_t* free_pages, int32_t* freed, int32_t* new_lens,
                                 hipStream_t s);
// LRFU selection (attention-aware keep scores): segments up to kLrfuMaxLen entries; those
// longer than kLrfuLdsLen only with pooling windows up to kLrfuRegMaxWindow.
constexpr int64_t kLrfuLdsLen = 38400;
constexpr int64_t kLrfuMaxLen = 64512;
constexpr int kLrfuRegMaxWindow = 7;
hipError_t launch_lrfu_select(const DevProblem& dp, const HostPlan& hp, const float* scores,
                              float top_p, float decay, float* ks, uint8_t* hit, float* pooled,
                              int32_t* kept, float* ks_kept, hipStream_t s);
// Confidence monitor (Sec. 6.1, Alg. 2).
constexpr int kConfMaxTopK = 64;          // largest k of the token confidence
constexpr int kConfChunkLogits = 16384;   // logits one partial workgroup handles
constexpr int kConfMaxSplits = 16;        // chunks per row: vocab <= 262,144
constexpr int kMaxBudgetWindows = 16384;  // min-pool windows one request may have
int conf_splits(int64_t vocab);
hipError_t launch_token_confidence(const float* logits, int64_t rows, int64_t vocab,
                                   int64_t row_stride, int k, float2* ms, float* top,
                                   float* conf, hipStream_t s);
hipError_t launch_budget_update(const float* tconf, const int64_t* offsets, int num_reqs,
                                int window, int stride, float bottom_pct, float scale_up,
                                int budget_upper, const int32_t* budgets_in,
                                int32_t* budgets_out, double* slopes, double* thresholds,
                                int32_t* retained, hipStream_t s);
hipError_t launch_compact(const DevProblem& dp, const HostPlan& hp, void* kv, int32_t* bt,
                          const int32_t* kept, const int32_t* free_pages, int32_t* freed,
                          int32_t* new_lens, hipStream_t s);
// The compaction of requests [r0, r1), of which none takes more than max_x fresh pages.
hipError_t launch_compact_range(const DevProblem& dp, const HostPlan& hp, int r0, int r1,
                                int64_t max_x, void* kv, int32_t* bt, const int32_t* kept,
                                const int32_t* free_pages, int32_t* freed, int32_t* new_lens,
                                hipStream_t s);
// In-place compaction (Alg. 4): slot planning into new_order (required), row copies,
// block-table rewrite.
hipError_t launch_compact_inplace(const DevProblem& dp, const HostPlan& hp, void* kv,
                                  int32_t* bt, const int32_t* kept, int32_t* src_rank,
                                  int32_t* freed, int32_t* new_lens, int32_t* new_order,
                                  hipStream_t s);

}  // namespace actkv
