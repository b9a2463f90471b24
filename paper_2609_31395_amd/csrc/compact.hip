// Fresh-page compaction: the kept K/V rows of every (request, KV head) are gathered, in
// ascending token order, into pages popped from the caller's free list; the block table
// row is then rewritten and the old pages returned (Sec. 7.2: freed blocks go back to the
// serving system).
//
// compact_gather_kernel: one 256-thread workgroup per destination (fresh) page.  It writes
// the page's K half and V half contiguously ([slot][head][D] rows, 16 bytes per lane, one
// 256-byte row per 16 lanes) and reads each source row as one contiguous 256-byte run
// through the OLD block table.  Destination pages are disjoint from every live page, so
// all copies are independent and need no ordering among themselves.
// compact_rewrite_kernel (runs after the gather, same stream): copies the old block-table
// row into freed_pages and writes the new row, so the gather never races the rewrite.
#include "device_common.hpp"

namespace actkv {

template <int D>
__global__ __launch_bounds__(256) void compact_gather_kernel(DevProblem dp, uint16_t* kv,
                                                             const int32_t* __restrict__ bt,
                                                             const int32_t* __restrict__ kept,
                                                             const int32_t* __restrict__ free_pages) {
  constexpr int CH = D / 8;                 // 16-byte chunks per row
  const int Hkv = dp.Hkv;
  const int64_t f = blockIdx.x;
  // request owning fresh page f: the largest r with fresh_off[r] <= f
  int lo = 0, hi = dp.R - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) / 2;
    if (dp.plan[mid].fresh_off <= f) lo = mid; else hi = mid - 1;
  }
  const int r = lo;
  const ReqPlan pl = dp.plan[r];
  const int p = (int)(f - pl.fresh_off);
  const int64_t dst_page = free_pages[f];
  const int32_t* bt_row = bt + (int64_t)r * dp.bt_stride;
  const int64_t plane = dp.num_pages * kPageSize * Hkv * (int64_t)D;   // K -> V offset
  const int items = 2 * kPageSize * Hkv * CH;
  constexpr int kBatch = 8;
  for (int base = 0; base < items; base += 256 * kBatch) {
    u32x4 v[kBatch];
    int64_t dst[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      dst[u] = -1;
      const int it = base + 256 * u + threadIdx.x;
      if (it >= items) continue;
      const int which = it / (kPageSize * Hkv * CH);
      const int rem = it % (kPageSize * Hkv * CH);
      const int s = rem / (Hkv * CH), h = (rem / CH) % Hkv, ch = rem % CH;
      const int j = p * kPageSize + s;
      const int bh = dp.budgets[r * Hkv + h];
      const int kh = bh < pl.L ? bh : pl.L;
      if (j >= kh) continue;
      const int t = kept[dp.kept_off[r * Hkv + h] + j];
      if (t < 0 || t >= pl.L) continue;
      const int64_t src_page = bt_row[t / kPageSize];
      // pages outside the pool are never dereferenced (the slot is left unwritten)
      if (src_page < 0 || src_page >= dp.num_pages || dst_page < 0 || dst_page >= dp.num_pages)
        continue;
      const int64_t src = which * plane + ((src_page * kPageSize + t % kPageSize) * Hkv + h) * (int64_t)D + ch * 8;
      dst[u] = which * plane + ((dst_page * kPageSize + s) * Hkv + h) * (int64_t)D + ch * 8;
      v[u] = *reinterpret_cast<const u32x4*>(kv + src);
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
    if (dp.D == 128)
      hipLaunchKernelGGL(compact_gather_kernel<128>, dim3((unsigned)hp.fresh_needed), dim3(256), 0, s,
                         dp, static_cast<uint16_t*>(kv), bt, kept, free_pages);
    else
      hipLaunchKernelGGL(compact_gather_kernel<64>, dim3((unsigned)hp.fresh_needed), dim3(256), 0, s,
                         dp, static_cast<uint16_t*>(kv), bt, kept, free_pages);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(compact_rewrite_kernel, dim3(hp.R), dim3(256), 0, s, dp, bt, free_pages,
                     freed, new_lens);
  return hipGetLastError();
}

}  // namespace actkv
