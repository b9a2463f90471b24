// libactkv C ABI: host-side validation, planning and workspace carving, then kernel
// launches on the caller's stream.  See include/actkv.h for the contract.
#include <math.h>
#include <string.h>

#include <atomic>
#include <mutex>
#include <vector>

#include "actkv.h"
#include "actkv_internal.h"

using actkv::DevProblem;
using actkv::HostPlan;
using actkv::WsLayout;

namespace {

bool valid_pool_window(int32_t w) { return w >= 1 && w <= actkv::kMaxPoolWindow && (w % 2) == 1; }

// Scoring cost units of a request (every row chunk and KV head): its key tiles times
// score_tile_cost of each chunk's row tiles.
int64_t request_score_cost(int64_t L, int64_t n, int32_t G, int32_t Hkv) {
  const int64_t ntiles = (L + actkv::kKeyTile - 1) / actkv::kKeyTile;
  const int64_t M = n * G;
  const int64_t chunks = M > 0 ? (M + actkv::kRowsPerChunk - 1) / actkv::kRowsPerChunk : 1;
  int64_t cost = 0;
  for (int64_t c = 0; c < chunks; ++c) {
    const int64_t rows = M - c * actkv::kRowsPerChunk;
    const int64_t rt = actkv::chunk_units(rows);
    cost += ntiles * actkv::score_tile_cost(rt) * Hkv;
  }
  return cost;
}

// Fresh pages request r takes (X; 0 when every head keeps everything).  Budgets are
// checked non-negative by plan_host.
int64_t request_fresh_pages(const actkv_problem* p, int r) {
  const int64_t L = p->seq_lens_h[r];
  int64_t kmax = 0, bmin = INT64_MAX;
  for (int h = 0; h < p->num_kv_heads; ++h) {
    const int64_t b = p->budgets_h[(int64_t)r * p->num_kv_heads + h];
    const int64_t k = b < L ? b : L;
    kmax = k > kmax ? k : kmax;
    bmin = b < bmin ? b : bmin;
  }
  return bmin < L ? (kmax + actkv::kPageSize - 1) / actkv::kPageSize : 0;
}

// Validates `p` and derives the host plan from the host mirrors.  Touches no device memory.
actkv_status plan_host(const actkv_problem* p, HostPlan* hp) {
  if (!p) return ACTKV_ERR_INVALID_ARGUMENT;
  if (p->num_reqs < 0 || p->num_q_heads <= 0 || p->num_kv_heads <= 0 || p->head_dim <= 0 ||
      p->page_size <= 0 || p->num_pages <= 0 || p->bt_stride <= 0)
    return ACTKV_ERR_INVALID_ARGUMENT;
  if (p->num_q_heads % p->num_kv_heads) return ACTKV_ERR_INVALID_ARGUMENT;
  if (!valid_pool_window(p->pool_window)) return ACTKV_ERR_INVALID_ARGUMENT;
  if (p->causal != 0 && p->causal != 1) return ACTKV_ERR_INVALID_ARGUMENT;
  if (p->agg != ACTKV_AGG_SUM && p->agg != ACTKV_AGG_MAX_MEAN) return ACTKV_ERR_INVALID_ARGUMENT;
  if (!isfinite(p->sm_scale) || p->sm_scale < 0.f) return ACTKV_ERR_INVALID_ARGUMENT;
  if (p->flags & ~(ACTKV_FLAG_PLANNED | ACTKV_FLAG_SMALL_SELECT)) return ACTKV_ERR_INVALID_ARGUMENT;
  if (p->head_dim != 64 && p->head_dim != 128) return ACTKV_ERR_UNSUPPORTED;
  if (p->page_size != actkv::kPageSize) return ACTKV_ERR_UNSUPPORTED;
  if (p->num_kv_heads > 64) return ACTKV_ERR_UNSUPPORTED;
  const int32_t G = p->num_q_heads / p->num_kv_heads;
  if (p->agg == ACTKV_AGG_MAX_MEAN && !(G == 1 || G == 2 || G == 4 || G == 8 || G == 16))
    return ACTKV_ERR_UNSUPPORTED;
  if (p->num_reqs > 0) {
    if (!p->seq_lens_h || !p->q_lens_h || !p->budgets_h) return ACTKV_ERR_INVALID_ARGUMENT;
  }
  hp->R = p->num_reqs;
  hp->Hq = p->num_q_heads;
  hp->Hkv = p->num_kv_heads;
  hp->G = G;
  hp->D = p->head_dim;
  const int BS = actkv::kPageSize;
  int32_t max_chunks = 1;
  for (int r = 0; r < p->num_reqs; ++r) {
    const int64_t L = p->seq_lens_h[r], n = p->q_lens_h[r];
    if (L < 0 || n < 0) return ACTKV_ERR_INVALID_ARGUMENT;
    if (p->causal && n > L) return ACTKV_ERR_INVALID_ARGUMENT;
    if ((L + BS - 1) / BS > p->bt_stride) return ACTKV_ERR_INVALID_ARGUMENT;
    if (n * G > (int64_t)actkv::kRowsPerChunk * 64) return ACTKV_ERR_UNSUPPORTED;
    const int32_t chunks = n * G > 0 ? (int32_t)((n * G + actkv::kRowsPerChunk - 1) / actkv::kRowsPerChunk) : 1;
    max_chunks = chunks > max_chunks ? chunks : max_chunks;
  }
  hp->max_chunks = max_chunks;
  for (int r = 0; r < p->num_reqs; ++r) {
    const int64_t L = p->seq_lens_h[r], n = p->q_lens_h[r];
    int64_t kmax = 0, bmin = INT64_MAX;
    for (int h = 0; h < p->num_kv_heads; ++h) {
      const int64_t b = p->budgets_h[(int64_t)r * p->num_kv_heads + h];
      if (b < 0) return ACTKV_ERR_INVALID_ARGUMENT;
      const int64_t k = b < L ? b : L;
      hp->num_kept += k;
      hp->max_k = k > hp->max_k ? k : hp->max_k;
      kmax = k > kmax ? k : kmax;
      bmin = b < bmin ? b : bmin;
    }
    if (bmin < L) {
      const int64_t X = (kmax + BS - 1) / BS;
      hp->max_fresh = X > hp->max_fresh ? X : hp->max_fresh;
      hp->fresh_needed += X;
      hp->pages_freed += (L + BS - 1) / BS;
      hp->pages_freed_inplace += (L + BS - 1) / BS - (kmax + BS - 1) / BS;
    }
    hp->sum_n += n;
    hp->sum_L += L;
    hp->max_L = L > hp->max_L ? L : hp->max_L;
    hp->max_n = n > hp->max_n ? n : hp->max_n;
    hp->score_cost += request_score_cost(L, n, G, p->num_kv_heads);
    const int64_t lb = (L + actkv::kLseKeysPerBlock - 1) / actkv::kLseKeysPerBlock;
    hp->lse_parts += n * p->num_q_heads * lb;
    hp->max_lse_blocks = lb > hp->max_lse_blocks ? lb : hp->max_lse_blocks;
  }
  hp->num_scores = hp->sum_L * p->num_kv_heads;
  hp->num_segments = (int64_t)p->num_reqs * max_chunks * p->num_kv_heads;
  if (hp->num_scores > INT64_C(1) << 40 || hp->sum_n > INT32_MAX / 2) return ACTKV_ERR_UNSUPPORTED;
  return ACTKV_OK;
}

// 64-bit FNV-1a over the problem's sizes and its host arrays: the signature a plan in the
// workspace carries (see ACTKV_FLAG_PLANNED).
struct Fnv {
  uint64_t h = 1469598103934665603ull;
  void add(const void* p, size_t n) {
    const unsigned char* b = static_cast<const unsigned char*>(p);
    for (size_t i = 0; i < n; ++i) h = (h ^ b[i]) * 1099511628211ull;
  }
  template <typename T> void add(T v) { add(&v, sizeof v); }
};

uint64_t problem_signature(const actkv_problem* p) {
  Fnv f;
  f.add(p->num_reqs); f.add(p->num_q_heads); f.add(p->num_kv_heads); f.add(p->head_dim);
  f.add(p->page_size); f.add(p->num_pages); f.add(p->bt_stride); f.add(p->pool_window);
  f.add(p->causal); f.add(p->agg);
  if (p->num_reqs > 0) {
    f.add(p->seq_lens_h, sizeof(int32_t) * (size_t)p->num_reqs);
    f.add(p->q_lens_h, sizeof(int32_t) * (size_t)p->num_reqs);
    f.add(p->budgets_h, sizeof(int32_t) * (size_t)p->num_reqs * (size_t)p->num_kv_heads);
  }
  return f.h | 1ull;   // never 0, so a zeroed workspace holds no plan
}

struct Ctx {
  HostPlan hp;
  WsLayout ws;
  DevProblem dp;
  char* base = nullptr;
};

// Common prologue of every launching entry point: validate, check the workspace, carve it
// and fill the device argument block.
actkv_status prepare(const actkv_problem* p, void* workspace, size_t workspace_bytes, Ctx* cx) {
  actkv_status st = plan_host(p, &cx->hp);
  if (st != ACTKV_OK) return st;
  if (p->num_reqs > 0 && (!p->seq_lens_d || !p->q_lens_d || !p->budgets_d))
    return ACTKV_ERR_INVALID_ARGUMENT;
  cx->ws = actkv::ws_layout(cx->hp);
  if (workspace_bytes < cx->ws.total) return ACTKV_ERR_WORKSPACE_TOO_SMALL;
  if (!workspace) return ACTKV_ERR_INVALID_ARGUMENT;
  cx->base = static_cast<char*>(workspace);
  DevProblem& d = cx->dp;
  d.R = cx->hp.R;
  d.Hq = cx->hp.Hq;
  d.Hkv = cx->hp.Hkv;
  d.G = cx->hp.G;
  d.D = cx->hp.D;
  d.num_pages = p->num_pages;
  d.bt_stride = p->bt_stride;
  d.max_chunks = cx->hp.max_chunks;
  d.pool_window = p->pool_window;
  d.causal = p->causal;
  d.agg = p->agg;
  d.sm_scale = p->sm_scale > 0.f ? p->sm_scale : 1.0f / sqrtf((float)p->head_dim);
  d.seq_lens = p->seq_lens_d;
  d.q_lens = p->q_lens_d;
  d.budgets = p->budgets_d;
  d.plan = reinterpret_cast<actkv::ReqPlan*>(cx->base + cx->ws.plan);
  d.kept_off = reinterpret_cast<int64_t*>(cx->base + cx->ws.kept_off);
  d.seg_cost = reinterpret_cast<int64_t*>(cx->base + cx->ws.seg_cost);
  d.num_segments = cx->hp.num_segments;
  d.sig = problem_signature(p);
  d.plan_sig = reinterpret_cast<uint64_t*>(cx->base + cx->ws.sig);
  d.req_done = reinterpret_cast<int32_t*>(cx->base + cx->ws.req_done);
  return ACTKV_OK;
}


actkv_status hip_status(hipError_t e) { return e == hipSuccess ? ACTKV_OK : ACTKV_ERR_HIP; }

// The plan kernel, unless the caller says the workspace already holds this problem's plan.
actkv_status plan_step(const Ctx& cx, const actkv_problem* p, hipStream_t s) {
  if (p->flags & ACTKV_FLAG_PLANNED) return ACTKV_OK;
  return hip_status(actkv::launch_plan(cx.dp, s));
}

// TopK selection of every request, on the kernel the problem's flags ask for.
hipError_t run_select(const Ctx& cx, const actkv_problem* p, const float* scores, float* pooled,
                      int32_t* kept, hipStream_t s) {
  if (p->flags & ACTKV_FLAG_SMALL_SELECT)
    return actkv::launch_select_side(cx.dp, cx.hp, 0, cx.hp.R, scores, pooled, kept, s);
  return actkv::launch_select(cx.dp, cx.hp, scores, pooled, kept, s);
}

// Selection and fresh-page compaction fused into one kernel (launch_select_compact), for
// batches whose copies are small: with several workgroups per segment when the segments fit
// its LDS form and the kept rows are few (select_compact_splits > 1), else, for at most this
// many segments keeping at most this many entries each, with one workgroup per segment that
// copies its own rows.  Measured on MI355X (Table 1 shapes: Hkv = 8, d = 128, GPU time): one
// request kept 512 of 1,024 entries in 20 against 26 us (one workgroup per segment), 1,536
// of 2,048 in 23 against 24 us and 4,096 of 6,144 in 28 against 32 us (selection, gather and
// rewrite kernels); four requests, 512 of 1,024: 25 against 34 us.  Earlier, with one
// workgroup per segment: 49 against 36 us at 8 segments of 1,536, 45 against 42 us at 128
// segments of 512.
constexpr int64_t kFusedMaxSegments = 32;
constexpr int64_t kFusedMaxKeptPerSegment = 512;

// TopK selection then fresh-page compaction of every request.
actkv_status run_select_compact(const Ctx& cx, const actkv_problem* p, const float* scores,
                                float* pooled, int32_t* kept, void* kv_cache,
                                int32_t* block_table, const int32_t* free_pages,
                                int32_t* freed_pages, int32_t* new_lens, hipStream_t s) {
  const bool small = (int64_t)cx.hp.R * cx.hp.Hkv <= kFusedMaxSegments &&
                     cx.hp.max_k <= kFusedMaxKeptPerSegment;
  const bool split = actkv::select_compact_splits(cx.hp, cx.dp.D) > 1;
  if (!(p->flags & ACTKV_FLAG_SMALL_SELECT) && (small || split))
    return hip_status(actkv::launch_select_compact(cx.dp, cx.hp, scores, pooled, kept, kv_cache,
                                                   block_table, free_pages, freed_pages,
                                                   new_lens, s));
  actkv_status st = hip_status(run_select(cx, p, scores, pooled, kept, s));
  if (st != ACTKV_OK) return st;
  return hip_status(actkv::launch_compact(cx.dp, cx.hp, kv_cache, block_table, kept, free_pages,
                                          freed_pages, new_lens, s));
}

// ---- the pipelined step ---------------------------------------------------------------
// Scoring is bound by the matrix and vector units and leaves HBM bandwidth and CU space
// (registers, LDS) idle; selection and compaction are bound by latency and HBM and leave
// the matrix units idle.  With the batch cut into request groups, group g is scored on the
// caller's stream while group g - 1 is selected (select_side_kernel, the small-budget
// selection) and compacted on a second stream, meant to run on the CUs the scoring kernel
// occupies.  The last group is selected and compacted on the caller's stream once all
// scoring is done (the whole GPU is then free for it).  Every order between the streams
// goes through an event: the side stream waits for a group's scores; the caller's stream
// waits for the side stream at the end.  Requests of different groups share no output, so
// no other order is needed.
// Measured on MI355X (32 x 35,000 tokens): the gather does run beside the scoring
// workgroups, but slows them by about as much time as it saves; the selection is not
// placed beside them at all and waits for free CUs; and scoring in several launches costs
// 5-14% over one launch.  The pipelined step came out 9-32% slower than the sequential
// one, so automatic mode does not pipeline.

constexpr int kMaxOverlapGroups = ACTKV_MAX_OVERLAP_GROUPS;
constexpr int kAutoOverlapGroups = 4;
// Automatic pipelining from this much scoring (cost units): never, for the measurements
// above.
constexpr int64_t kOverlapMinCost = INT64_MAX;
// Share of the scoring cost in the last group: its selection and compaction are not hidden.
constexpr double kOverlapLastShare = 0.125;

std::atomic<int32_t> g_overlap{0};

struct SideStream {
  hipStream_t stream = nullptr;
  hipEvent_t ev[kMaxOverlapGroups] = {};
};
constexpr int kMaxSideDevices = 64;
std::mutex g_side_mu;   // held while a pipelined step enqueues (the events are shared)
SideStream g_side[kMaxSideDevices];

// The current device's side stream and events, created on first use.  g_side_mu held.
actkv_status side_stream(SideStream** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return ACTKV_ERR_HIP;
  if (dev < 0 || dev >= kMaxSideDevices) return ACTKV_ERR_UNSUPPORTED;
  SideStream& ss = g_side[dev];
  if (!ss.stream) {
    SideStream made;
    for (hipEvent_t& e : made.ev)
      if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) return ACTKV_ERR_HIP;
    if (hipStreamCreateWithFlags(&made.stream, hipStreamNonBlocking) != hipSuccess)
      return ACTKV_ERR_HIP;
    ss = made;
  }
  *out = &ss;
  return ACTKV_OK;
}

// Request groups of a pipelined step: group g is requests [r[g], r[g + 1]), its scoring
// cost cost[g] and the most fresh pages one of its requests takes, max_x[g].
struct OverlapPlan {
  int n = 0;
  int r[kMaxOverlapGroups + 1] = {};
  int64_t cost[kMaxOverlapGroups] = {};
  int64_t max_x[kMaxOverlapGroups] = {};
};

// Whether the step is pipelined, and its groups: groups 0 .. n-2 split (1 - last share)
// of the scoring cost evenly, the last group takes the rest; every group holds at least one
// request.
bool plan_overlap(const actkv_problem* p, const HostPlan& hp, OverlapPlan* op) {
  const int32_t mode = g_overlap.load(std::memory_order_relaxed);
  if (mode == 1 || hp.R < 2 || hp.num_scores == 0) return false;
  int G = mode >= 2 ? mode : kAutoOverlapGroups;
  if (mode == 0 && hp.score_cost < kOverlapMinCost) return false;
  if (G > hp.R) G = hp.R;
  std::vector<int64_t> cost(hp.R);
  for (int r = 0; r < hp.R; ++r)
    cost[r] = request_score_cost(p->seq_lens_h[r], p->q_lens_h[r], hp.G, hp.Hkv);
  const double total = (double)hp.score_cost;
  int r = 0;
  int64_t acc = 0;
  op->n = G;
  for (int g = 0; g < G; ++g) {
    const int last_end = hp.R - (G - 1 - g);   // leave a request for every later group
    const double target = (g + 1) * (1.0 - kOverlapLastShare) / (G - 1) * total;
    int64_t gc = 0, mx = 0;
    do {
      gc += cost[r];
      acc += cost[r];
      const int64_t x = request_fresh_pages(p, r);
      mx = x > mx ? x : mx;
      ++r;
    } while (r < last_end && (g == G - 1 || (double)acc < target));
    op->r[g + 1] = r;
    op->cost[g] = gc;
    op->max_x[g] = mx;
  }
  return true;
}

actkv_status run_lse(const Ctx& cx, const void* q, const void* kv, const int32_t* bt,
                     float* lse_out, hipStream_t s) {
  float2* part = reinterpret_cast<float2*>(cx.base + cx.ws.lse_part);
  return hip_status(actkv::launch_lse(cx.dp, cx.hp, q, kv, bt, lse_out, part, s));
}

actkv_status run_score(const Ctx& cx, const void* q, const void* kv, const int32_t* bt,
                       const float* lse, float* scores, hipStream_t s) {
  if (!lse) {
    float* lse_ws = reinterpret_cast<float*>(cx.base + cx.ws.lse);
    actkv_status st = run_lse(cx, q, kv, bt, lse_ws, s);
    if (st != ACTKV_OK) return st;
    lse = lse_ws;
  }
  float* part = reinterpret_cast<float*>(cx.base + cx.ws.score_part);
  return hip_status(actkv::launch_score(cx.dp, cx.hp, q, kv, bt, lse, scores, part, s));
}

// The pipelined step's launches (the plan and the LSE, if any, already queued on s).
actkv_status run_overlapped(const Ctx& cx, const OverlapPlan& op, const void* q, void* kv,
                            int32_t* bt, const float* lse, const int32_t* free_pages,
                            float* scores, float* pooled, int32_t* kept, int32_t* freed,
                            int32_t* new_lens, hipStream_t s) {
  std::lock_guard<std::mutex> lock(g_side_mu);
  SideStream* ss = nullptr;
  actkv_status st = side_stream(&ss);
  if (st != ACTKV_OK) return st;
  const DevProblem& dp = cx.dp;
  const HostPlan& hp = cx.hp;
  float* part = reinterpret_cast<float*>(cx.base + cx.ws.score_part);
  const int G = op.n;
  hipError_t e = hipSuccess;
  for (int g = 0; g < G && e == hipSuccess; ++g) {
    e = actkv::launch_score_range(dp, hp, op.r[g], op.r[g + 1], op.cost[g], q, kv, bt, lse,
                                  scores, part, s);
    if (e != hipSuccess || g == G - 1) break;
    e = hipEventRecord(ss->ev[g], s);
    if (e == hipSuccess) e = hipStreamWaitEvent(ss->stream, ss->ev[g], 0);
    if (e == hipSuccess)
      e = actkv::launch_select_side(dp, hp, op.r[g], op.r[g + 1], scores, pooled, kept,
                                    ss->stream);
    if (e == hipSuccess)
      e = actkv::launch_compact_range(dp, hp, op.r[g], op.r[g + 1], op.max_x[g], kv, bt, kept,
                                      free_pages, freed, new_lens, ss->stream);
  }
  if (e == hipSuccess)
    e = actkv::launch_select_range(dp, hp, op.r[G - 1], op.r[G], scores, pooled, kept, s);
  if (e == hipSuccess)
    e = actkv::launch_compact_range(dp, hp, op.r[G - 1], op.r[G], op.max_x[G - 1], kv, bt, kept,
                                    free_pages, freed, new_lens, s);
  // join, also after a failed launch: nothing queued here may outlive the caller's order
  hipError_t j = hipEventRecord(ss->ev[G - 1], ss->stream);
  if (j == hipSuccess) j = hipStreamWaitEvent(s, ss->ev[G - 1], 0);
  return hip_status(e != hipSuccess ? e : j);
}

}  // namespace

extern "C" {

actkv_status actkv_query(const actkv_problem* p, size_t* workspace_bytes, int64_t* num_kept,
                         int64_t* fresh_pages_needed, int64_t* pages_freed) {
  HostPlan hp;
  actkv_status st = plan_host(p, &hp);
  if (st != ACTKV_OK) return st;
  if (workspace_bytes) *workspace_bytes = actkv::ws_layout(hp).total;
  if (num_kept) *num_kept = hp.num_kept;
  if (fresh_pages_needed) *fresh_pages_needed = hp.fresh_needed;
  if (pages_freed) *pages_freed = hp.pages_freed;
  return ACTKV_OK;
}

actkv_status actkv_plan(const actkv_problem* p, void* workspace, size_t workspace_bytes,
                        void* stream) {
  Ctx cx;
  actkv_status st = prepare(p, workspace, workspace_bytes, &cx);
  if (st != ACTKV_OK) return st;
  if (cx.hp.R == 0) return ACTKV_OK;
  return hip_status(actkv::launch_plan(cx.dp, static_cast<hipStream_t>(stream)));
}

actkv_status actkv_lse(const actkv_problem* p, const void* q, const void* kv_cache,
                       const int32_t* block_table, float* lse_out, void* workspace,
                       size_t workspace_bytes, void* stream) {
  Ctx cx;
  actkv_status st = prepare(p, workspace, workspace_bytes, &cx);
  if (st != ACTKV_OK) return st;
  if (cx.hp.sum_n > 0 && (!q || !kv_cache || !block_table || !lse_out))
    return ACTKV_ERR_INVALID_ARGUMENT;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (cx.hp.R == 0) return ACTKV_OK;
  st = plan_step(cx, p, s);
  if (st != ACTKV_OK) return st;
  return run_lse(cx, q, kv_cache, block_table, lse_out, s);
}

actkv_status actkv_score(const actkv_problem* p, const void* q, const void* kv_cache,
                         const int32_t* block_table, const float* lse, float* scores,
                         void* workspace, size_t workspace_bytes, void* stream) {
  Ctx cx;
  actkv_status st = prepare(p, workspace, workspace_bytes, &cx);
  if (st != ACTKV_OK) return st;
  if (cx.hp.num_scores > 0 && (!kv_cache || !block_table || !scores)) return ACTKV_ERR_INVALID_ARGUMENT;
  if (cx.hp.sum_n > 0 && !q) return ACTKV_ERR_INVALID_ARGUMENT;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (cx.hp.R == 0) return ACTKV_OK;
  st = plan_step(cx, p, s);
  if (st != ACTKV_OK) return st;
  return run_score(cx, q, kv_cache, block_table, lse, scores, s);
}

actkv_status actkv_score_accumulate(const actkv_problem* p, const void* q, const void* kv_cache,
                                    const int32_t* block_table, const float* lse, float* acc,
                                    void* workspace, size_t workspace_bytes, void* stream) {
  Ctx cx;
  actkv_status st = prepare(p, workspace, workspace_bytes, &cx);
  if (st != ACTKV_OK) return st;
  if (cx.hp.num_scores > 0 && (!kv_cache || !block_table || !acc)) return ACTKV_ERR_INVALID_ARGUMENT;
  if (cx.hp.sum_n > 0 && !q) return ACTKV_ERR_INVALID_ARGUMENT;
  if (acc && (reinterpret_cast<uintptr_t>(acc) & 15)) return ACTKV_ERR_INVALID_ARGUMENT;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (cx.hp.R == 0 || cx.hp.num_scores == 0) return ACTKV_OK;
  st = plan_step(cx, p, s);
  if (st != ACTKV_OK) return st;
  if (cx.hp.max_n <= 1 && cx.hp.G <= actkv::kDecodeMaxGroup) {
    // a decode step (one action query per request at most): scored and added in one pass
    if (cx.hp.sum_n == 0) return ACTKV_OK;
    if (!lse) {
      float* lse_ws = reinterpret_cast<float*>(cx.base + cx.ws.lse);
      st = run_lse(cx, q, kv_cache, block_table, lse_ws, s);
      if (st != ACTKV_OK) return st;
      lse = lse_ws;
    }
    return hip_status(actkv::launch_score_decode(cx.dp, cx.hp, q, kv_cache, block_table, lse,
                                                 acc, s));
  }
  float* step_scores = reinterpret_cast<float*>(cx.base + cx.ws.scores);
  st = run_score(cx, q, kv_cache, block_table, lse, step_scores, s);
  if (st != ACTKV_OK) return st;
  return hip_status(actkv::launch_accumulate(acc, step_scores, cx.hp.num_scores, s));
}

actkv_status actkv_select(const actkv_problem* p, const float* scores, float* pooled,
                          int32_t* kept, void* workspace, size_t workspace_bytes,
                          void* stream) {
  Ctx cx;
  actkv_status st = prepare(p, workspace, workspace_bytes, &cx);
  if (st != ACTKV_OK) return st;
  if (cx.hp.num_scores > 0 && !scores) return ACTKV_ERR_INVALID_ARGUMENT;
  if (cx.hp.num_kept > 0 && !kept) return ACTKV_ERR_INVALID_ARGUMENT;
  if (pooled && scores && pooled == scores) return ACTKV_ERR_INVALID_ARGUMENT;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (cx.hp.R == 0) return ACTKV_OK;
  if (!pooled) pooled = reinterpret_cast<float*>(cx.base + cx.ws.pooled);
  st = plan_step(cx, p, s);
  if (st != ACTKV_OK) return st;
  return hip_status(run_select(cx, p, scores, pooled, kept, s));
}

actkv_status actkv_compact(const actkv_problem* p, void* kv_cache, int32_t* block_table,
                           const int32_t* kept, const int32_t* free_pages, int64_t num_free,
                           int32_t* freed_pages, int32_t* new_lens, void* workspace,
                           size_t workspace_bytes, void* stream) {
  Ctx cx;
  actkv_status st = prepare(p, workspace, workspace_bytes, &cx);
  if (st != ACTKV_OK) return st;
  if (num_free < 0) return ACTKV_ERR_INVALID_ARGUMENT;
  if (cx.hp.R > 0 && (!block_table || !new_lens)) return ACTKV_ERR_INVALID_ARGUMENT;
  if (cx.hp.fresh_needed > 0 && (!kv_cache || !kept)) return ACTKV_ERR_INVALID_ARGUMENT;
  if (cx.hp.pages_freed > 0 && !freed_pages) return ACTKV_ERR_INVALID_ARGUMENT;
  if (num_free < cx.hp.fresh_needed) return ACTKV_ERR_OUT_OF_PAGES;
  if (cx.hp.fresh_needed > 0 && !free_pages) return ACTKV_ERR_INVALID_ARGUMENT;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (cx.hp.R == 0) return ACTKV_OK;
  st = plan_step(cx, p, s);
  if (st != ACTKV_OK) return st;
  return hip_status(actkv::launch_compact(cx.dp, cx.hp, kv_cache, block_table, kept, free_pages,
                                          freed_pages, new_lens, s));
}

actkv_status actkv_select_compact(const actkv_problem* p, const float* scores, float* pooled,
                                  int32_t* kept, void* kv_cache, int32_t* block_table,
                                  const int32_t* free_pages, int64_t num_free,
                                  int32_t* freed_pages, int32_t* new_lens, void* workspace,
                                  size_t workspace_bytes, void* stream) {
  Ctx cx;
  actkv_status st = prepare(p, workspace, workspace_bytes, &cx);
  if (st != ACTKV_OK) return st;
  if (num_free < 0) return ACTKV_ERR_INVALID_ARGUMENT;
  if (cx.hp.num_scores > 0 && !scores) return ACTKV_ERR_INVALID_ARGUMENT;
  if (pooled && scores && pooled == scores) return ACTKV_ERR_INVALID_ARGUMENT;
  if (cx.hp.R > 0 && (!block_table || !new_lens)) return ACTKV_ERR_INVALID_ARGUMENT;
  if (cx.hp.fresh_needed > 0 && !kv_cache) return ACTKV_ERR_INVALID_ARGUMENT;
  if (cx.hp.pages_freed > 0 && !freed_pages) return ACTKV_ERR_INVALID_ARGUMENT;
  if (num_free < cx.hp.fresh_needed) return ACTKV_ERR_OUT_OF_PAGES;
  if (cx.hp.fresh_needed > 0 && !free_pages) return ACTKV_ERR_INVALID_ARGUMENT;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (cx.hp.R == 0) return ACTKV_OK;
  if (!pooled) pooled = reinterpret_cast<float*>(cx.base + cx.ws.pooled);
  if (!kept) kept = reinterpret_cast<int32_t*>(cx.base + cx.ws.kept);
  st = plan_step(cx, p, s);
  if (st != ACTKV_OK) return st;
  return run_select_compact(cx, p, scores, pooled, kept, kv_cache, block_table, free_pages,
                            freed_pages, new_lens, s);
}

namespace {
actkv_status check_lrfu(const Ctx& cx, float top_p, float decay, const float* scores,
                        const float* ks, const float* pooled, const int32_t* kept,
                        const float* ks_kept) {
  if (!(top_p >= 0.0f && top_p <= 1.0f) || !(decay >= 0.0f && decay <= 1.0f))
    return ACTKV_ERR_INVALID_ARGUMENT;
  if (cx.hp.max_L > actkv::kLrfuMaxLen) return ACTKV_ERR_UNSUPPORTED;
  if (cx.hp.max_L > actkv::kLrfuLdsLen && cx.dp.pool_window > actkv::kLrfuRegMaxWindow)
    return ACTKV_ERR_UNSUPPORTED;
  if (cx.hp.num_scores > 0 && !ks) return ACTKV_ERR_INVALID_ARGUMENT;
  if (cx.hp.num_kept > 0 && (!kept || !ks_kept)) return ACTKV_ERR_INVALID_ARGUMENT;
  if (ks && (ks == scores || ks == pooled)) return ACTKV_ERR_INVALID_ARGUMENT;
  return ACTKV_OK;
}
}  // namespace

actkv_status actkv_lrfu_select(const actkv_problem* p, const float* scores, float top_p,
                               float decay, float* ks, uint8_t* hit, float* pooled,
                               int32_t* kept, float* ks_kept, void* workspace,
                               size_t workspace_bytes, void* stream) {
  Ctx cx;
  actkv_status st = prepare(p, workspace, workspace_bytes, &cx);
  if (st != ACTKV_OK) return st;
  if (cx.hp.num_scores > 0 && !scores) return ACTKV_ERR_INVALID_ARGUMENT;
  if (pooled && scores && pooled == scores) return ACTKV_ERR_INVALID_ARGUMENT;
  st = check_lrfu(cx, top_p, decay, scores, ks, pooled, kept, ks_kept);
  if (st != ACTKV_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (cx.hp.R == 0) return ACTKV_OK;
  st = plan_step(cx, p, s);
  if (st != ACTKV_OK) return st;
  return hip_status(actkv::launch_lrfu_select(cx.dp, cx.hp, scores, top_p, decay, ks, hit,
                                              pooled, kept, ks_kept, s));
}

actkv_status actkv_step_lrfu(const actkv_problem* p, const void* q, void* kv_cache,
                             int32_t* block_table, const float* lse, const int32_t* free_pages,
                             int64_t num_free, float top_p, float decay, float* ks,
                             float* ks_kept, float* scores, float* pooled, uint8_t* hit,
                             int32_t* kept, int32_t* freed_pages, int32_t* new_lens,
                             void* workspace, size_t workspace_bytes, void* stream) {
  Ctx cx;
  actkv_status st = prepare(p, workspace, workspace_bytes, &cx);
  if (st != ACTKV_OK) return st;
  if (num_free < 0) return ACTKV_ERR_INVALID_ARGUMENT;
  if (cx.hp.R > 0 && (!block_table || !new_lens)) return ACTKV_ERR_INVALID_ARGUMENT;
  if (cx.hp.num_scores > 0 && !kv_cache) return ACTKV_ERR_INVALID_ARGUMENT;
  if (cx.hp.sum_n > 0 && !q) return ACTKV_ERR_INVALID_ARGUMENT;
  if (cx.hp.pages_freed > 0 && !freed_pages) return ACTKV_ERR_INVALID_ARGUMENT;
  if (num_free < cx.hp.fresh_needed) return ACTKV_ERR_OUT_OF_PAGES;
  if (cx.hp.fresh_needed > 0 && !free_pages) return ACTKV_ERR_INVALID_ARGUMENT;
  if (scores && pooled && scores == pooled) return ACTKV_ERR_INVALID_ARGUMENT;
  if (!scores) scores = reinterpret_cast<float*>(cx.base + cx.ws.scores);
  if (!pooled) pooled = reinterpret_cast<float*>(cx.base + cx.ws.pooled);
  if (!kept) kept = reinterpret_cast<int32_t*>(cx.base + cx.ws.kept);
  st = check_lrfu(cx, top_p, decay, scores, ks, pooled, kept, ks_kept);
  if (st != ACTKV_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (cx.hp.R == 0) return ACTKV_OK;
  st = plan_step(cx, p, s);
  if (st != ACTKV_OK) return st;
  st = run_score(cx, q, kv_cache, block_table, lse, scores, s);
  if (st != ACTKV_OK) return st;
  st = hip_status(actkv::launch_lrfu_select(cx.dp, cx.hp, scores, top_p, decay, ks, hit, pooled,
                                            kept, ks_kept, s));
  if (st != ACTKV_OK) return st;
  return hip_status(actkv::launch_compact(cx.dp, cx.hp, kv_cache, block_table, kept, free_pages,
                                          freed_pages, new_lens, s));
}

actkv_status actkv_step(const actkv_problem* p, const void* q, void* kv_cache,
                        int32_t* block_table, const float* lse, const int32_t* free_pages,
                        int64_t num_free, float* scores, float* pooled, int32_t* kept,
                        int32_t* freed_pages, int32_t* new_lens, void* workspace,
                        size_t workspace_bytes, void* stream) {
  return actkv::step_impl(p, q, kv_cache, block_table, lse, free_pages, num_free, scores, pooled,
                          kept, freed_pages, new_lens, workspace, workspace_bytes, stream, true);
}

actkv_status actkv_check_pages(const actkv_problem* p, const int32_t* block_table,
                               const int32_t* free_pages, int64_t num_free, uint32_t* status,
                               void* scratch, size_t scratch_bytes, void* stream) {
  HostPlan hp;
  actkv_status st = plan_host(p, &hp);
  if (st != ACTKV_OK) return st;
  if (!status || !scratch || num_free < 0) return ACTKV_ERR_INVALID_ARGUMENT;
  if (hp.R > 0 && (!p->seq_lens_d || !p->q_lens_d || !p->budgets_d || !block_table))
    return ACTKV_ERR_INVALID_ARGUMENT;
  if (scratch_bytes < ACTKV_CHECK_SCRATCH_BYTES(p->num_pages)) return ACTKV_ERR_WORKSPACE_TOO_SMALL;
  if (num_free < hp.fresh_needed) return ACTKV_ERR_OUT_OF_PAGES;
  if (hp.fresh_needed > 0 && !free_pages) return ACTKV_ERR_INVALID_ARGUMENT;
  uint64_t want[3] = {0, 0, 0};
  for (int r = 0; r < hp.R; ++r) {
    want[0] += actkv::mirror_term(r, p->seq_lens_h[r]);
    want[1] += actkv::mirror_term(r, p->q_lens_h[r]);
  }
  for (int64_t i = 0; i < (int64_t)hp.R * hp.Hkv; ++i)
    want[2] += actkv::mirror_term(i, p->budgets_h[i]);
  return hip_status(actkv::launch_check_pages(
      p->seq_lens_d, p->q_lens_d, p->budgets_d, hp.R, hp.Hkv, block_table, p->bt_stride,
      p->num_pages, free_pages, hp.fresh_needed, want, status, static_cast<uint32_t*>(scratch),
      static_cast<hipStream_t>(stream)));
}

actkv_status actkv_set_overlap(int32_t groups) {
  if (groups < 0 || groups > ACTKV_MAX_OVERLAP_GROUPS) return ACTKV_ERR_INVALID_ARGUMENT;
  g_overlap.store(groups, std::memory_order_relaxed);
  return ACTKV_OK;
}

int32_t actkv_get_overlap(void) { return g_overlap.load(std::memory_order_relaxed); }

}  // extern "C"

// The body of actkv_step, shared with actkv_step_noalloc (which passes its static scratch
// array as the workspace).
actkv_status actkv::step_impl(const actkv_problem* p, const void* q, void* kv_cache,
                              int32_t* block_table, const float* lse, const int32_t* free_pages,
                              int64_t num_free, float* scores, float* pooled, int32_t* kept,
                              int32_t* freed_pages, int32_t* new_lens, void* workspace,
                              size_t workspace_bytes, void* stream, bool may_overlap) {
  Ctx cx;
  actkv_status st = prepare(p, workspace, workspace_bytes, &cx);
  if (st != ACTKV_OK) return st;
  if (num_free < 0) return ACTKV_ERR_INVALID_ARGUMENT;
  if (cx.hp.R > 0 && (!block_table || !new_lens)) return ACTKV_ERR_INVALID_ARGUMENT;
  if (cx.hp.num_scores > 0 && !kv_cache) return ACTKV_ERR_INVALID_ARGUMENT;
  if (cx.hp.sum_n > 0 && !q) return ACTKV_ERR_INVALID_ARGUMENT;
  if (cx.hp.pages_freed > 0 && !freed_pages) return ACTKV_ERR_INVALID_ARGUMENT;
  if (num_free < cx.hp.fresh_needed) return ACTKV_ERR_OUT_OF_PAGES;
  if (cx.hp.fresh_needed > 0 && !free_pages) return ACTKV_ERR_INVALID_ARGUMENT;
  if (scores && pooled && scores == pooled) return ACTKV_ERR_INVALID_ARGUMENT;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (cx.hp.R == 0) return ACTKV_OK;
  if (!scores) scores = reinterpret_cast<float*>(cx.base + cx.ws.scores);
  if (!pooled) pooled = reinterpret_cast<float*>(cx.base + cx.ws.pooled);
  if (!kept) kept = reinterpret_cast<int32_t*>(cx.base + cx.ws.kept);
  st = plan_step(cx, p, s);
  if (st != ACTKV_OK) return st;
  OverlapPlan op;
  if (may_overlap && plan_overlap(p, cx.hp, &op)) {
    if (!lse) {
      float* lse_ws = reinterpret_cast<float*>(cx.base + cx.ws.lse);
      st = run_lse(cx, q, kv_cache, block_table, lse_ws, s);
      if (st != ACTKV_OK) return st;
      lse = lse_ws;
    }
    return run_overlapped(cx, op, q, kv_cache, block_table, lse, free_pages, scores, pooled,
                          kept, freed_pages, new_lens, s);
  }
  st = run_score(cx, q, kv_cache, block_table, lse, scores, s);
  if (st != ACTKV_OK) return st;
  return run_select_compact(cx, p, scores, pooled, kept, kv_cache, block_table, free_pages,
                            freed_pages, new_lens, s);
}

extern "C" {

actkv_status actkv_query_inplace(const actkv_problem* p, int64_t* pages_freed) {
  HostPlan hp;
  actkv_status st = plan_host(p, &hp);
  if (st != ACTKV_OK) return st;
  if (pages_freed) *pages_freed = hp.pages_freed_inplace;
  return ACTKV_OK;
}

namespace {
actkv_status run_compact_inplace(const Ctx& cx, void* kv_cache, int32_t* block_table,
                                 const int32_t* kept, int32_t* freed_pages, int32_t* new_lens,
                                 int32_t* new_order, hipStream_t s) {
  int32_t* src_rank = reinterpret_cast<int32_t*>(cx.base + cx.ws.ip_src);
  if (!new_order) new_order = reinterpret_cast<int32_t*>(cx.base + cx.ws.ip_order);
  return hip_status(actkv::launch_compact_inplace(cx.dp, cx.hp, kv_cache, block_table, kept,
                                                  src_rank, freed_pages, new_lens, new_order,
                                                  s));
}

actkv_status check_compact_inplace(const Ctx& cx, const void* kv_cache, const int32_t* block_table,
                                   const int32_t* freed_pages, const int32_t* new_lens) {
  if (cx.hp.R > 0 && (!block_table || !new_lens)) return ACTKV_ERR_INVALID_ARGUMENT;
  if (cx.hp.num_kept > 0 && !kv_cache) return ACTKV_ERR_INVALID_ARGUMENT;
  if (cx.hp.pages_freed_inplace > 0 && !freed_pages) return ACTKV_ERR_INVALID_ARGUMENT;
  return ACTKV_OK;
}
}  // namespace

actkv_status actkv_compact_inplace(const actkv_problem* p, void* kv_cache, int32_t* block_table,
                                   const int32_t* kept, int32_t* freed_pages, int32_t* new_lens,
                                   int32_t* new_order, void* workspace, size_t workspace_bytes,
                                   void* stream) {
  Ctx cx;
  actkv_status st = prepare(p, workspace, workspace_bytes, &cx);
  if (st != ACTKV_OK) return st;
  st = check_compact_inplace(cx, kv_cache, block_table, freed_pages, new_lens);
  if (st != ACTKV_OK) return st;
  if (cx.hp.num_kept > 0 && !kept) return ACTKV_ERR_INVALID_ARGUMENT;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (cx.hp.R == 0) return ACTKV_OK;
  st = plan_step(cx, p, s);
  if (st != ACTKV_OK) return st;
  return run_compact_inplace(cx, kv_cache, block_table, kept, freed_pages, new_lens, new_order,
                             s);
}

actkv_status actkv_step_inplace(const actkv_problem* p, const void* q, void* kv_cache,
                                int32_t* block_table, const float* lse, float* scores,
                                float* pooled, int32_t* kept, int32_t* freed_pages,
                                int32_t* new_lens, int32_t* new_order, void* workspace,
                                size_t workspace_bytes, void* stream) {
  Ctx cx;
  actkv_status st = prepare(p, workspace, workspace_bytes, &cx);
  if (st != ACTKV_OK) return st;
  st = check_compact_inplace(cx, kv_cache, block_table, freed_pages, new_lens);
  if (st != ACTKV_OK) return st;
  if (cx.hp.num_scores > 0 && !kv_cache) return ACTKV_ERR_INVALID_ARGUMENT;
  if (cx.hp.sum_n > 0 && !q) return ACTKV_ERR_INVALID_ARGUMENT;
  if (scores && pooled && scores == pooled) return ACTKV_ERR_INVALID_ARGUMENT;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (cx.hp.R == 0) return ACTKV_OK;
  if (!scores) scores = reinterpret_cast<float*>(cx.base + cx.ws.scores);
  if (!pooled) pooled = reinterpret_cast<float*>(cx.base + cx.ws.pooled);
  if (!kept) kept = reinterpret_cast<int32_t*>(cx.base + cx.ws.kept);
  st = plan_step(cx, p, s);
  if (st != ACTKV_OK) return st;
  st = run_score(cx, q, kv_cache, block_table, lse, scores, s);
  if (st != ACTKV_OK) return st;
  st = hip_status(run_select(cx, p, scores, pooled, kept, s));
  if (st != ACTKV_OK) return st;
  return run_compact_inplace(cx, kv_cache, block_table, kept, freed_pages, new_lens, new_order,
                             s);
}

namespace {
size_t token_conf_ws(int64_t rows, int64_t vocab, int32_t top_k) {
  const int64_t parts = rows * actkv::conf_splits(vocab);
  return actkv::align256(sizeof(float2) * (size_t)parts) +
         actkv::align256(sizeof(float) * (size_t)(parts * top_k));
}
actkv_status check_token_conf(int64_t rows, int64_t vocab, int32_t top_k) {
  if (rows < 0 || vocab < 1 || top_k < 1) return ACTKV_ERR_INVALID_ARGUMENT;
  if (top_k > actkv::kConfMaxTopK) return ACTKV_ERR_UNSUPPORTED;
  if (vocab > (int64_t)actkv::kConfMaxSplits * actkv::kConfChunkLogits) return ACTKV_ERR_UNSUPPORTED;
  if (rows > INT32_MAX / actkv::kConfMaxSplits) return ACTKV_ERR_UNSUPPORTED;
  return ACTKV_OK;
}
}  // namespace

actkv_status actkv_token_confidence_workspace(int64_t rows, int64_t vocab, int32_t top_k,
                                              size_t* workspace_bytes) {
  actkv_status st = check_token_conf(rows, vocab, top_k);
  if (st != ACTKV_OK) return st;
  if (workspace_bytes) *workspace_bytes = token_conf_ws(rows, vocab, top_k);
  return ACTKV_OK;
}

actkv_status actkv_token_confidence(const float* logits, int64_t rows, int64_t vocab,
                                    int64_t row_stride, int32_t top_k, float* conf,
                                    void* workspace, size_t workspace_bytes, void* stream) {
  actkv_status st = check_token_conf(rows, vocab, top_k);
  if (st != ACTKV_OK) return st;
  if (row_stride < vocab) return ACTKV_ERR_INVALID_ARGUMENT;
  if (rows == 0) return ACTKV_OK;
  if (!logits || !conf) return ACTKV_ERR_INVALID_ARGUMENT;
  const size_t need = token_conf_ws(rows, vocab, top_k);
  if (workspace_bytes < need) return ACTKV_ERR_WORKSPACE_TOO_SMALL;
  if (!workspace) return ACTKV_ERR_INVALID_ARGUMENT;
  char* base = static_cast<char*>(workspace);
  const int64_t parts = rows * actkv::conf_splits(vocab);
  float2* ms = reinterpret_cast<float2*>(base);
  float* top = reinterpret_cast<float*>(base + actkv::align256(sizeof(float2) * (size_t)parts));
  return hip_status(actkv::launch_token_confidence(logits, rows, vocab, row_stride, top_k, ms,
                                                   top, conf, static_cast<hipStream_t>(stream)));
}

actkv_status actkv_budget_update(const float* token_conf, const int64_t* offsets_h,
                                 const int64_t* offsets_d, int32_t num_reqs, int32_t window,
                                 int32_t stride, float bottom_pct, float scale_up,
                                 int32_t budget_upper, const int32_t* budgets_in,
                                 int32_t* budgets_out, double* slopes, double* thresholds,
                                 int32_t* retained, void* stream) {
  if (num_reqs < 0 || window < 1 || stride < 1 || budget_upper < 0)
    return ACTKV_ERR_INVALID_ARGUMENT;
  if (!(bottom_pct >= 0.0f && bottom_pct <= 100.0f) || !(scale_up >= 1.0f) || !isfinite(scale_up))
    return ACTKV_ERR_INVALID_ARGUMENT;
  if (num_reqs == 0) return ACTKV_OK;
  if (!offsets_h || !offsets_d || !budgets_in || !budgets_out) return ACTKV_ERR_INVALID_ARGUMENT;
  if (offsets_h[0] < 0) return ACTKV_ERR_INVALID_ARGUMENT;
  for (int r = 0; r < num_reqs; ++r) {
    const int64_t n = offsets_h[r + 1] - offsets_h[r];
    if (n < 0) return ACTKV_ERR_INVALID_ARGUMENT;
    if (n >= window && (n - window) / stride + 1 > actkv::kMaxBudgetWindows)
      return ACTKV_ERR_UNSUPPORTED;
  }
  if (offsets_h[num_reqs] > offsets_h[0] && !token_conf) return ACTKV_ERR_INVALID_ARGUMENT;
  return hip_status(actkv::launch_budget_update(
      token_conf, offsets_d, num_reqs, window, stride, bottom_pct, scale_up, budget_upper,
      budgets_in, budgets_out, slopes, thresholds, retained, static_cast<hipStream_t>(stream)));
}

const char* actkv_status_str(actkv_status status) {
  switch (status) {
    case ACTKV_OK: return "ok";
    case ACTKV_ERR_INVALID_ARGUMENT: return "invalid argument";
    case ACTKV_ERR_UNSUPPORTED: return "unsupported";
    case ACTKV_ERR_WORKSPACE_TOO_SMALL: return "workspace too small";
    case ACTKV_ERR_OUT_OF_PAGES: return "free list shorter than the fresh pages needed";
    case ACTKV_ERR_HIP: return "HIP launch or runtime error";
  }
  return "unknown status";
}

}  // extern "C"
