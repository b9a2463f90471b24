// Fresh-page compaction: the kept K/V rows of every (request, KV head) are gathered, in
// ascending token order, into pages popped from the caller's free list; the block table
// row is then rewritten and the old pages returned (Sec. 7.2: freed blocks go back to the
// serving system).
//
// compact_gather_kernel: one 256-thread workgroup per group of destination (fresh) pages.
// It first resolves every (page, slot, head) to its source slot through the kept indices
// and the OLD block table (one lookup per thread, into LDS), then streams the rows: each
// destination page is written contiguously ([slot][head][D] rows, 16 bytes per lane) and
// each source row is read as one contiguous run.  Destination pages are disjoint from
// every live page, so all copies are independent and need no ordering among themselves.
// compact_rewrite_kernel (runs after the gather, same stream): copies the old block-table
// row into freed_pages and writes the new row, so the gather never races the rewrite.
#include "device_common.hpp"

namespace actkv {

constexpr int kCompactThreads = 256;
constexpr int kCompactTable = 1024;   // (page, slot, head) source entries per workgroup

// Fresh pages handled by one workgroup: enough (page, slot, head) rows to give every
// thread one source lookup, at least one page.
__host__ __device__ inline int compact_pages_per_wg(int Hkv) {
  const int p = kCompactThreads / (kPageSize * Hkv);
  return p < 1 ? 1 : p;
}

template <int D>
__global__ __launch_bounds__(kCompactThreads) void compact_gather_kernel(
    DevProblem dp, uint16_t* kv, const int32_t* __restrict__ bt, const int32_t* __restrict__ kept,
    const int32_t* __restrict__ free_pages, int64_t num_fresh) {
  constexpr int CH = D / 8;                 // 16-byte chunks per row
  __shared__ int64_t src_slot[kCompactTable];   // flat source slot, -1: nothing to copy
  __shared__ int64_t dst_page[kCompactTable / kPageSize];
  const int Hkv = dp.Hkv;
  const int ppw = compact_pages_per_wg(Hkv);
  const int64_t f0 = (int64_t)blockIdx.x * ppw;
  const int npages = (int)(num_fresh - f0 < ppw ? num_fresh - f0 : ppw);
  const int entries = npages * kPageSize * Hkv;

  // ---- resolve every (page, slot, head) of this workgroup to its source slot once
  for (int e = threadIdx.x; e < entries; e += kCompactThreads) {
    const int p = e / (kPageSize * Hkv), s = (e / Hkv) % kPageSize, h = e % Hkv;
    const int64_t f = f0 + p;
    // request owning fresh page f: the largest r with fresh_off[r] <= f
    int lo = 0, hi = dp.R - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) / 2;
      if (dp.plan[mid].fresh_off <= f) lo = mid; else hi = mid - 1;
    }
    const ReqPlan pl = dp.plan[lo];
    const int j = (int)(f - pl.fresh_off) * kPageSize + s;
    const int bh = dp.budgets[lo * Hkv + h];
    const int kh = bh < pl.L ? bh : pl.L;
    int64_t src = -1;
    if (j < kh) {
      const int t = kept[dp.kept_off[lo * Hkv + h] + j];
      if (t >= 0 && t < pl.L) {
        const int64_t page = bt[(int64_t)lo * dp.bt_stride + t / kPageSize];
        // pages outside the pool are never dereferenced (the slot is left unwritten)
        if (page >= 0 && page < dp.num_pages) src = page * kPageSize + t % kPageSize;
      }
    }
    src_slot[e] = src;
    if (s == 0 && h == 0) {
      const int64_t dpg = free_pages[f];
      dst_page[p] = (dpg >= 0 && dpg < dp.num_pages) ? dpg : -1;
    }
  }
  __syncthreads();

  // ---- copy: consecutive threads move consecutive 16-byte chunks of the destination pages
  // (K half, then V half), so every store is part of a contiguous run
  const int64_t plane = dp.num_pages * kPageSize * Hkv * (int64_t)D;   // K -> V offset
  const int rows = 2 * entries;
  const int items = rows * CH;
  constexpr int kBatch = 16;
  for (int base = 0; base < items; base += kCompactThreads * kBatch) {
    u32x4 v[kBatch];
    int64_t dst[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      dst[u] = -1;
      const int it = base + kCompactThreads * u + threadIdx.x;
      if (it >= items) continue;
      const int row = it / CH, ch = it % CH;
      const int which = row / entries, e = row % entries;
      const int p = e / (kPageSize * Hkv), s = (e / Hkv) % kPageSize, h = e % Hkv;
      const int64_t src = src_slot[e], dpg = dst_page[p];
      if (src < 0 || dpg < 0) continue;
      dst[u] = which * plane + ((dpg * kPageSize + s) * Hkv + h) * (int64_t)D + ch * 8;
      v[u] = *reinterpret_cast<const u32x4*>(kv + which * plane + (src * Hkv + h) * (int64_t)D + ch * 8);
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u)
      if (dst[u] >= 0) *reinterpret_cast<u32x4*>(kv + dst[u]) = v[u];
  }
}

__global__ __launch_bounds__(256) void compact_rewrite_kernel(DevProblem dp, int32_t* bt,
                                                              const int32_t* __restrict__ free_pages,
                                                              int32_t* __restrict__ freed,
                                                              int32_t* __restrict__ new_lens) {
  const int r = blockIdx.x, Hkv = dp.Hkv;
  const ReqPlan pl = dp.plan[r];
  for (int h = threadIdx.x; h < Hkv; h += 256) {
    const int b = dp.budgets[r * Hkv + h];
    new_lens[r * Hkv + h] = pl.skip ? pl.L : (b < pl.L ? b : pl.L);
  }
  if (pl.skip) return;
  int32_t* row = bt + (int64_t)r * dp.bt_stride;
  for (int i = threadIdx.x; i < pl.Y; i += 256) {
    const int32_t old = row[i];
    freed[pl.freed_off + i] = old;
    row[i] = i < pl.X ? free_pages[pl.fresh_off + i] : -1;
  }
}

hipError_t launch_compact(const DevProblem& dp, const HostPlan& hp, void* kv, int32_t* bt,
                          const int32_t* kept, const int32_t* free_pages, int32_t* freed,
                          int32_t* new_lens, hipStream_t s) {
  if (hp.R == 0) return hipSuccess;
  if (hp.fresh_needed > 0) {
    const int ppw = compact_pages_per_wg(hp.Hkv);
    const unsigned grid = (unsigned)((hp.fresh_needed + ppw - 1) / ppw);
    if (dp.D == 128)
      hipLaunchKernelGGL(compact_gather_kernel<128>, dim3(grid), dim3(kCompactThreads), 0, s, dp,
                         static_cast<uint16_t*>(kv), bt, kept, free_pages, hp.fresh_needed);
    else
      hipLaunchKernelGGL(compact_gather_kernel<64>, dim3(grid), dim3(kCompactThreads), 0, s, dp,
                         static_cast<uint16_t*>(kv), bt, kept, free_pages, hp.fresh_needed);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(compact_rewrite_kernel, dim3(hp.R), dim3(256), 0, s, dp, bt, free_pages,
                     freed, new_lens);
  return hipGetLastError();
}

}  // namespace actkv
