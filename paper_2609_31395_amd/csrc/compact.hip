// Fresh-page compaction: the kept K/V rows of every (request, KV head) are gathered, in
// ascending token order, into pages popped from the caller's free list; the block table
// row is then rewritten and the old pages returned (Sec. 7.2: freed blocks go back to the
// serving system).
//
// compact_gather_kernel: one 256-thread workgroup per group of destination (fresh) pages of
// one request (grid: page groups of the longest request x requests; the workgroups past a
// request's own pages return at once).  It first resolves every (page, slot, head) to its
// source row through the kept indices and the OLD block table (one lookup per thread, into
// LDS), then streams the rows: each destination page is written contiguously
// ([slot][head][D] rows, 16 bytes per lane) and each source row is read as one contiguous
// run.  Destination pages are disjoint from every live page, so all copies are independent
// and need no ordering among themselves.
// compact_rewrite_kernel (runs after the gather, same stream): copies the old block-table
// row into freed_pages and writes the new row, so the gather never races the rewrite.
#include "device_common.hpp"

namespace actkv {

constexpr int kCompactThreads = 256;
// at most 72 registers: two of its waves fit on a SIMD beside a resident scoring wave
constexpr int kCompactMinWaves = 7;
constexpr int kCompactTable = 1024;   // (page, slot, head) source entries per workgroup
constexpr int kCompactBatch = 8;      // 16-byte loads of a thread in flight together
constexpr int kRewriteBatch = 8;      // block-table entries a rewrite thread reads together

// Fresh pages handled by one workgroup: enough (page, slot, head) rows to give every
// thread one source lookup, at least one page.
__host__ __device__ inline int compact_pages_per_wg(int Hkv) {
  const int p = kCompactThreads / (kPageSize * Hkv);
  return p < 1 ? 1 : p;
}

// The copies of destination pages q0 .. of request r (see compact_gather_kernel).
template <int D, bool kInPlace>
__device__ __forceinline__ void gather_pages(const DevProblem& dp, int r, const ReqPlan& pl, int q0,
                                             uint16_t* kv, const int32_t* __restrict__ bt,
                                             const int32_t* __restrict__ kept,
                                             const int32_t* __restrict__ free_pages) {
  constexpr int CH = D / 8;                 // 16-byte chunks per row
  static_assert((CH & (CH - 1)) == 0, "chunks per row: a power of two");
  // per (page, slot, head) entry: the source row's element offset in the K plane (-1:
  // nothing to copy); compacted in place into the live entries' source offsets below
  __shared__ int64_t src_off[kCompactTable];
  __shared__ int64_t dst_off[kCompactTable];    // the live entries' destination offsets
  __shared__ int64_t dst_page[kCompactTable / kPageSize];
  __shared__ int wave_live[kCompactThreads / 64];
  const int Hkv = dp.Hkv;
  const int ppw = compact_pages_per_wg(Hkv);
  const int npages = pl.X - q0 < ppw ? pl.X - q0 : ppw;
  const int entries = npages * kPageSize * Hkv;
  const int start = (pl.Y - pl.X) * kPageSize;   // in place: logical slot of new slot 0

  // ---- resolve every (page, slot, head) of this workgroup to its source row once
  for (int e = threadIdx.x; e < entries; e += kCompactThreads) {
    const int p = e / (kPageSize * Hkv), s = (e / Hkv) % kPageSize, h = e % Hkv;
    const int j = (q0 + p) * kPageSize + s;
    const int bh = dp.budgets[r * Hkv + h];
    const int kh = bh < pl.L ? bh : pl.L;
    int64_t src = -1;
    if (j < kh) {
      const int t = kept[dp.kept_off[r * Hkv + h] + j];
      if (t >= 0 && t < pl.L && !(kInPlace && t == start + j)) {
        const int64_t page = bt[(int64_t)r * dp.bt_stride + t / kPageSize];
        // pages outside the pool are never dereferenced (the slot is left unwritten)
        if (page >= 0 && page < dp.num_pages)
          src = ((page * kPageSize + t % kPageSize) * Hkv + h) * (int64_t)D;
      }
    }
    src_off[e] = src;
    if (s == 0 && h == 0) {
      const int64_t dpg = kInPlace
          ? (int64_t)bt[(int64_t)r * dp.bt_stride + (pl.Y - pl.X) + q0 + p]
          : (int64_t)free_pages[pl.fresh_off + q0 + p];
      dst_page[p] = (dpg >= 0 && dpg < dp.num_pages) ? dpg : -1;
    }
  }
  __syncthreads();

  // ---- the entries that copy a row, in ascending order (with unequal head budgets or in
  // place, many slots of a destination page receive nothing; the copy loop skips them):
  // their (source, destination) offsets, packed to the front.  An entry's packed position
  // is at most its own, and every entry of a pass is read before any is written.
  int n_live = 0;   // uniform
  for (int e0 = 0; e0 < entries; e0 += kCompactThreads) {
    const int e = e0 + (int)threadIdx.x, w = threadIdx.x >> 6;
    int64_t src = -1, dst = -1;
    if (e < entries) {
      const int p = e / (kPageSize * Hkv), s = (e / Hkv) % kPageSize, h = e % Hkv;
      src = src_off[e];
      if (dst_page[p] >= 0) dst = ((dst_page[p] * kPageSize + s) * Hkv + h) * (int64_t)D;
    }
    const bool has = src >= 0 && dst >= 0;
    const uint64_t bal = __ballot(has);
    if ((threadIdx.x & 63) == 0) wave_live[w] = __popcll(bal);
    __syncthreads();
    int before = n_live, total = 0;
    for (int i = 0; i < kCompactThreads / 64; ++i) {
      before += i < w ? wave_live[i] : 0;
      total += wave_live[i];
    }
    if (has) {
      const int at = before + (int)__builtin_amdgcn_mbcnt_hi(
                                  (uint32_t)(bal >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u));
      src_off[at] = src;
      dst_off[at] = dst;
    }
    n_live += total;
    __syncthreads();
  }

  // ---- copy: consecutive threads move consecutive 16-byte chunks of the live rows (K rows,
  // then V rows), so the stores of a destination page form contiguous runs.  Every row is
  // read and written once: non-temporal loads and stores (a plain 1 GiB device copy measured
  // 5.5 TB/s with ordinary and 5.9 TB/s with non-temporal accesses on MI355X).
  const int64_t plane = dp.num_pages * kPageSize * Hkv * (int64_t)D;   // K -> V offset
  const int half = n_live * CH, items = 2 * half;
  constexpr int kBatch = kCompactBatch, kStep = kCompactThreads * kBatch;
  auto chunk_of = [&](int it, int64_t* src, int64_t* dst) {
    const bool v_plane = it >= half;
    const int i = v_plane ? it - half : it;
    const int row = i / CH, ch = i % CH;
    const int64_t add = (v_plane ? plane : 0) + ch * 8;
    *src = src_off[row] + add;
    *dst = dst_off[row] + add;
  };
  // whole batches: every item is a live row, so the loads and stores carry no condition and
  // all kBatch loads of a thread are in flight together (a condition per item made the
  // compiler wait for every outstanding access before each load and store)
  const int full = items / kStep * kStep;
  for (int base = 0; base < full; base += kStep) {
    u32x4 v[kBatch];
    int64_t dst[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      int64_t src;
      chunk_of(base + kCompactThreads * u + (int)threadIdx.x, &src, &dst[u]);
      v[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(kv + src));
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u)
      __builtin_nontemporal_store(v[u], reinterpret_cast<u32x4*>(kv + dst[u]));
  }
  // the last, partial batch: items past the end repeat the last one (the same bytes to the
  // same place), so this batch carries no condition either
  if (full < items) {
    u32x4 v[kBatch];
    int64_t dst[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int it = full + kCompactThreads * u + (int)threadIdx.x;
      int64_t src;
      chunk_of(it < items ? it : items - 1, &src, &dst[u]);
      v[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(kv + src));
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u)
      __builtin_nontemporal_store(v[u], reinterpret_cast<u32x4*>(kv + dst[u]));
  }
}

// Request r's block-table rewrite: new lengths, the old row to the freed list, the fresh
// pages (then -1) into the row.  Runs after every read of the old row.
__device__ __forceinline__ void rewrite_row(const DevProblem& dp, int r, const ReqPlan& pl,
                                            int32_t* bt, const int32_t* __restrict__ free_pages,
                                            int32_t* __restrict__ freed,
                                            int32_t* __restrict__ new_lens) {
  const int Hkv = dp.Hkv;
  for (int h = threadIdx.x; h < Hkv; h += blockDim.x) {
    const int b = dp.budgets[r * Hkv + h];
    new_lens[r * Hkv + h] = pl.skip ? pl.L : (b < pl.L ? b : pl.L);
  }
  if (pl.skip || pl.Y <= 0) return;
  // batches of kRewriteBatch entries per thread: every load of a batch is issued before its
  // stores (an entry is read and written by the same thread only), and the loads carry no
  // condition (indices past the row re-read its last entry, values unused), so they are in
  // flight together instead of one round trip per entry
  int32_t* row = bt + (int64_t)r * dp.bt_stride;
  const int last = pl.Y - 1;
  // the fresh page ids (a request that takes none, every head keeping nothing, reads its own
  // row instead and writes -1)
  const int32_t* fresh = pl.X > 0 ? free_pages + pl.fresh_off : row;
  const int fresh_last = pl.X > 0 ? pl.X - 1 : last;
  for (int i0 = threadIdx.x; i0 < pl.Y; i0 += kRewriteBatch * (int)blockDim.x) {
    int32_t old[kRewriteBatch], now[kRewriteBatch];
#pragma unroll
    for (int u = 0; u < kRewriteBatch; ++u) {
      const int i = i0 + u * (int)blockDim.x;
      old[u] = row[i < last ? i : last];
      now[u] = fresh[i < fresh_last ? i : fresh_last];
    }
#pragma unroll
    for (int u = 0; u < kRewriteBatch; ++u) {
      const int i = i0 + u * (int)blockDim.x;
      if (i < pl.Y) {
        freed[pl.freed_off + i] = old[u];
        row[i] = i < pl.X ? now[u] : -1;
      }
    }
  }
}

// kInPlace = false: destination page q of request r is free_pages[fresh_off + q] and new
// slot j gets token kept[j].  kInPlace = true (Alg. 4): destination page q is the request's
// own page bt[r, Y - X + q] and new slot j gets token new_order[j] (`kept` below), a copy
// only where that token is not already there.
template <int D, bool kInPlace>
__global__ __launch_bounds__(kCompactThreads, kCompactMinWaves) void compact_gather_kernel(
    DevProblem dp, int r0, uint16_t* kv, const int32_t* __restrict__ bt,
    const int32_t* __restrict__ kept, const int32_t* __restrict__ free_pages) {
  if (!plan_ok(dp)) return;   // the workspace holds another problem's plan
  const int ppw = compact_pages_per_wg(dp.Hkv);
  // request r's destination pages q0 .. q0 + npages - 1 (of its X)
  const int r = r0 + (int)blockIdx.y;
  const ReqPlan pl = dp.plan[r];
  const int q0 = (int)blockIdx.x * ppw;
  if (q0 >= pl.X) return;   // the request has fewer pages than the grid's longest
  gather_pages<D, kInPlace>(dp, r, pl, q0, kv, bt, kept, free_pages);
}

// After the gather on the same stream, so the gather always reads the old row.  (Fused
// into the gather's tail -- the last workgroup of a request, found by a per-request counter,
// rewriting its row -- the counter's atomics cost more than this launch: 1169 against 1076
// us per layer of the 48-layer model, 240 against 199 us for the adaptive batch.)
__global__ __launch_bounds__(256) void compact_rewrite_kernel(DevProblem dp, int r0, int32_t* bt,
                                                              const int32_t* __restrict__ free_pages,
                                                              int32_t* __restrict__ freed,
                                                              int32_t* __restrict__ new_lens) {
  if (!plan_ok(dp)) return;   // the workspace holds another problem's plan
  const int r = r0 + (int)blockIdx.x;
  rewrite_row(dp, r, dp.plan[r], bt, free_pages, freed, new_lens);
}

hipError_t launch_compact_range(const DevProblem& dp, const HostPlan& hp, int r0, int r1,
                                int64_t max_x, void* kv, int32_t* bt, const int32_t* kept,
                                const int32_t* free_pages, int32_t* freed, int32_t* new_lens,
                                hipStream_t s) {
  if (r0 >= r1) return hipSuccess;
  if (max_x > 0) {
    const int ppw = compact_pages_per_wg(hp.Hkv);
    const dim3 grid((unsigned)((max_x + ppw - 1) / ppw), (unsigned)(r1 - r0));
    if (dp.D == 128)
      hipLaunchKernelGGL((compact_gather_kernel<128, false>), grid, dim3(kCompactThreads), 0, s,
                         dp, r0, static_cast<uint16_t*>(kv), bt, kept, free_pages);
    else
      hipLaunchKernelGGL((compact_gather_kernel<64, false>), grid, dim3(kCompactThreads), 0, s,
                         dp, r0, static_cast<uint16_t*>(kv), bt, kept, free_pages);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(compact_rewrite_kernel, dim3(r1 - r0), dim3(256), 0, s, dp, r0, bt,
                     free_pages, freed, new_lens);
  return hipGetLastError();
}

hipError_t launch_compact(const DevProblem& dp, const HostPlan& hp, void* kv, int32_t* bt,
                          const int32_t* kept, const int32_t* free_pages, int32_t* freed,
                          int32_t* new_lens, hipStream_t s) {
  return launch_compact_range(dp, hp, 0, hp.R, hp.max_fresh, kv, bt, kept, free_pages, freed,
                              new_lens, s);
}

// ---- in-place compaction (Alg. 4) --------------------------------------------------------
//
// Per compacted request, with Y = ceil(L / 16) and X = ceil(max_h k_h / 16) (shared by the
// heads: a page holds every head's row of a slot), each head h has the tail region
// [Start, End) = [(Y - X) * 16, (Y - X) * 16 + k_h).  Its destinations are the slots of the
// region that hold no kept entry (slots at or past L included: they exist in the last
// page), its sources the kept entries outside the region, both ascending; the i-th source
// is copied to the i-th destination (Alg. 4 steps 2-6).  Sources are kept and destinations
// are not, so no copy reads a slot another copy writes: one pass, no staging buffer.
//
// inplace_plan_kernel: one 1024-thread workgroup per (request, KV head).  With the kept
//   indices ascending, the sources are kept[0, a) and kept[b, k), a and b the counts of kept
//   entries below Start and below End (one workgroup sum); the destinations are the zero
//   bits of a bitmap of the region (kept[a, b) set), ranked by one workgroup scan per
//   32768 slots.  The plan is written as new_order: the token that new slot j = d - Start
//   receives (the i-th source for the i-th destination d, the token itself for a survivor
//   already in place).
// compact_gather_kernel<D, true>: the copies, organised by destination page exactly like
//   the fresh-page gather (the last X pages of every request in place of fresh pages),
//   skipping the slots whose token is already there.
// inplace_rewrite_kernel: per request, the first Y - X pages to the freed list, then the
//   block-table row shifted left by Y - X (read before write within each chunk of 256
//   entries) and -1 past X.
constexpr int kIpPlanThreads = 1024;
constexpr int kIpBitmapSlots = 32 * kIpPlanThreads;   // region slots per bitmap pass

__global__ __launch_bounds__(kIpPlanThreads) void inplace_plan_kernel(
    DevProblem dp, const int32_t* __restrict__ kept, int32_t* src_rank, int32_t* new_order) {
  if (!plan_ok(dp)) return;   // the workspace holds another problem's plan
  __shared__ uint32_t bits[kIpBitmapSlots / 32];
  __shared__ int64_t scan_tmp[17];
  const int seg = blockIdx.x, tid = threadIdx.x, Hkv = dp.Hkv;
  const int r = seg / Hkv;
  const ReqPlan pl = dp.plan[r];
  const int L = pl.L;
  const int bud = dp.budgets[seg];
  const int k = bud < L ? bud : L;
  const int64_t ko = dp.kept_off[seg];
  const int32_t* kk = kept + ko;
  int32_t* ps = src_rank + ko;
  int32_t* no = new_order + ko;
  if (pl.skip) {   // untouched request: nothing moves
    for (int j = tid; j < k; j += kIpPlanThreads) no[j] = kk[j];
    return;
  }
  const int start = (pl.Y - pl.X) * kPageSize, end = start + k;
  // a = kept entries below Start, b = below End (each count < 2^31: one packed sum)
  int64_t cnt = 0;
  for (int j = tid; j < k; j += kIpPlanThreads) {
    const int t = kk[j];
    cnt += ((int64_t)(t < start) << 32) + (t < end);
  }
  int64_t tot;
  block_excl_scan_i64(cnt, scan_tmp, &tot);
  const int a = (int)(tot >> 32), b = (int)(tot & 0xFFFFFFFFll);
  const int npairs = a + (k - b);
  // sources in ascending order; survivors inside the region stay where they are
  for (int j = tid; j < k; j += kIpPlanThreads) {
    const int t = kk[j];
    if (j < a) ps[j] = t;
    else if (j >= b) ps[j - (b - a)] = t;
    else if (t >= start && t < end) no[t - start] = t;
  }
  __syncthreads();   // the sources are read back below
  // destinations: the holes of [start, end), ranked in ascending order
  int64_t rank_base = 0;
  for (int c0 = 0; c0 < k; c0 += kIpBitmapSlots) {
    const int span = k - c0 < kIpBitmapSlots ? k - c0 : kIpBitmapSlots;
    bits[tid] = 0;
    __syncthreads();
    for (int j = a + tid; j < b; j += kIpPlanThreads) {
      const int off = kk[j] - start - c0;
      if (off >= 0 && off < span) atomicOr(&bits[off >> 5], 1u << (off & 31));
    }
    __syncthreads();
    const int valid = span - tid * 32;   // slots of this thread's word inside the span
    uint32_t holes = valid <= 0 ? 0u : ~bits[tid];
    if (valid > 0 && valid < 32) holes &= (1u << valid) - 1u;
    int64_t rank = rank_base + block_excl_scan_i64(__popc(holes), scan_tmp, &tot);
    while (holes) {
      const int j = c0 + tid * 32 + __builtin_ctz(holes);   // new slot (destination - Start)
      if (rank < npairs) no[j] = ps[rank];
      ++rank;
      holes &= holes - 1u;
    }
    rank_base += tot;
    __syncthreads();   // the bitmap is cleared again by the next pass
  }
}

__global__ __launch_bounds__(256) void inplace_rewrite_kernel(DevProblem dp, int32_t* bt,
                                                              int32_t* __restrict__ freed,
                                                              int32_t* __restrict__ new_lens) {
  if (!plan_ok(dp)) return;   // the workspace holds another problem's plan
  const int r = blockIdx.x, Hkv = dp.Hkv, tid = threadIdx.x;
  const ReqPlan pl = dp.plan[r];
  for (int h = tid; h < Hkv; h += 256) {
    const int b = dp.budgets[r * Hkv + h];
    new_lens[r * Hkv + h] = pl.skip ? pl.L : (b < pl.L ? b : pl.L);
  }
  if (pl.skip) return;
  int32_t* row = bt + (int64_t)r * dp.bt_stride;
  const int X = pl.X, F = pl.Y - pl.X;
  for (int i = tid; i < F; i += 256) freed[pl.ip_freed_off + i] = row[i];
  __syncthreads();   // every freed page read before the row is overwritten
  for (int base = 0; base < X; base += 256) {
    const int i = base + tid;
    const int32_t v = i < X ? row[F + i] : 0;
    __syncthreads();   // this chunk's reads before its writes (the ranges overlap if F < 256)
    if (i < X) row[i] = v;
    __syncthreads();
  }
  for (int i = X + tid; i < pl.Y; i += 256) row[i] = -1;
}

hipError_t launch_compact_inplace(const DevProblem& dp, const HostPlan& hp, void* kv,
                                  int32_t* bt, const int32_t* kept, int32_t* src_rank,
                                  int32_t* freed, int32_t* new_lens, int32_t* new_order,
                                  hipStream_t s) {
  if (hp.R == 0) return hipSuccess;
  hipLaunchKernelGGL(inplace_plan_kernel, dim3((unsigned)(hp.R * hp.Hkv)), dim3(kIpPlanThreads),
                     0, s, dp, kept, src_rank, new_order);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // the destination pages are the last X pages of every compacted request: as many, and at
  // the same offsets, as the fresh pages of the other form
  if (hp.max_fresh > 0) {
    const int ppw = compact_pages_per_wg(hp.Hkv);
    const dim3 grid((unsigned)((hp.max_fresh + ppw - 1) / ppw), (unsigned)hp.R);
    if (dp.D == 128)
      hipLaunchKernelGGL((compact_gather_kernel<128, true>), grid, dim3(kCompactThreads), 0, s,
                         dp, 0, static_cast<uint16_t*>(kv), bt, new_order, nullptr);
    else
      hipLaunchKernelGGL((compact_gather_kernel<64, true>), grid, dim3(kCompactThreads), 0, s,
                         dp, 0, static_cast<uint16_t*>(kv), bt, new_order, nullptr);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(inplace_rewrite_kernel, dim3(hp.R), dim3(256), 0, s, dp, bt, freed,
                     new_lens);
  return hipGetLastError();
}

}  // namespace actkv
