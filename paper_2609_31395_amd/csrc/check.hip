// Device-side check of what the fresh-page compaction takes on trust (the caller's guarantee
// to actkv_compact and actkv_step; the paper's compaction is correct only when no copy writes
// a slot another copy reads, Sec. 7.2): the pages the step takes from the free list lie in
// the pool, appear once and are not live; live block-table entries lie in the pool; the
// device mirrors of the lengths, query counts and budgets hold the host's values.  Every
// kernel here only reads its inputs and bounds-checks a page before using it as an index;
// findings are OR-ed into one status word.
#include "device_common.hpp"

namespace actkv {

namespace {

constexpr int kCheckThreads = 256;

__device__ __forceinline__ void flag(uint32_t* status, uint32_t bit) { atomicOr(status, bit); }

// Both bitmaps and the status word to zero (a kernel, so that a captured graph holds no
// memset node).
__global__ __launch_bounds__(kCheckThreads) void check_clear_kernel(uint32_t* bits, int64_t words,
                                                                    uint32_t* status) {
  for (int64_t i = (int64_t)blockIdx.x * kCheckThreads + threadIdx.x; i < words;
       i += (int64_t)gridDim.x * kCheckThreads)
    bits[i] = 0u;
  if (blockIdx.x == 0 && threadIdx.x == 0) *status = 0u;
}

// Every live page, bt[r, 0 .. ceil(L_r / 16)) with L_r from the device mirror (clamped to the
// row), into `live`; entries outside the pool are flagged instead.
__global__ __launch_bounds__(kCheckThreads) void check_live_kernel(
    const int32_t* __restrict__ seq_lens, const int32_t* __restrict__ bt, int bt_stride,
    int64_t num_pages, uint32_t* live, uint32_t* status) {
  const int r = blockIdx.y;
  const int64_t L = seq_lens[r];
  int64_t Y = L > 0 ? (L + kPageSize - 1) / kPageSize : 0;
  Y = Y < bt_stride ? Y : bt_stride;
  for (int64_t i = (int64_t)blockIdx.x * kCheckThreads + threadIdx.x; i < Y;
       i += (int64_t)gridDim.x * kCheckThreads) {
    const int64_t page = bt[(int64_t)r * bt_stride + i];
    if (page < 0 || page >= num_pages)
      flag(status, ACTKV_CHECK_TABLE_RANGE);
    else
      atomicOr(&live[page >> 5], 1u << (page & 31));
  }
}

// The fresh pages free_pages[0 .. n_fresh): in the pool, not live, not repeated.
__global__ __launch_bounds__(kCheckThreads) void check_fresh_kernel(
    const int32_t* __restrict__ free_pages, int64_t n_fresh, int64_t num_pages,
    const uint32_t* __restrict__ live, uint32_t* seen, uint32_t* status) {
  for (int64_t f = (int64_t)blockIdx.x * kCheckThreads + threadIdx.x; f < n_fresh;
       f += (int64_t)gridDim.x * kCheckThreads) {
    const int64_t page = free_pages[f];
    if (page < 0 || page >= num_pages) {
      flag(status, ACTKV_CHECK_FREE_RANGE);
      continue;
    }
    const uint32_t bit = 1u << (page & 31);
    if (live[page >> 5] & bit) flag(status, ACTKV_CHECK_FRESH_LIVE);
    if (atomicOr(&seen[page >> 5], bit) & bit) flag(status, ACTKV_CHECK_FRESH_DUP);
  }
}

// One workgroup: the mirrors' checksums against the host's.
__global__ __launch_bounds__(kCheckThreads) void check_mirrors_kernel(
    const int32_t* __restrict__ seq_lens, const int32_t* __restrict__ q_lens,
    const int32_t* __restrict__ budgets, int R, int Hkv, uint64_t want_lens, uint64_t want_q,
    uint64_t want_budgets, uint32_t* status) {
  __shared__ uint64_t part[3][kCheckThreads];
  uint64_t a = 0, b = 0, c = 0;
  for (int i = threadIdx.x; i < R; i += kCheckThreads) {
    a += mirror_term(i, seq_lens[i]);
    b += mirror_term(i, q_lens[i]);
  }
  for (int64_t i = threadIdx.x; i < (int64_t)R * Hkv; i += kCheckThreads)
    c += mirror_term(i, budgets[i]);
  part[0][threadIdx.x] = a;
  part[1][threadIdx.x] = b;
  part[2][threadIdx.x] = c;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t s[3] = {0, 0, 0};
    for (int t = 0; t < kCheckThreads; ++t)
      for (int k = 0; k < 3; ++k) s[k] += part[k][t];
    if (s[0] != want_lens || s[1] != want_q || s[2] != want_budgets)
      flag(status, ACTKV_CHECK_MIRRORS);
  }
}

}  // namespace

hipError_t launch_check_pages(const int32_t* seq_lens, const int32_t* q_lens,
                              const int32_t* budgets, int R, int Hkv, const int32_t* bt,
                              int bt_stride, int64_t num_pages, const int32_t* free_pages,
                              int64_t n_fresh, const uint64_t want[3], uint32_t* status,
                              uint32_t* scratch, hipStream_t s) {
  const int64_t words = check_bitmap_words(num_pages);
  uint32_t* live = scratch;
  uint32_t* seen = scratch + words;
  const int64_t clear_blocks = (2 * words + kCheckThreads - 1) / kCheckThreads;
  hipLaunchKernelGGL(check_clear_kernel,
                     dim3((unsigned)(clear_blocks < 4096 ? (clear_blocks > 0 ? clear_blocks : 1)
                                                         : 4096)),
                     dim3(kCheckThreads), 0, s, scratch, 2 * words, status);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (R > 0) {
    const int64_t xb = ((int64_t)bt_stride + kCheckThreads - 1) / kCheckThreads;
    hipLaunchKernelGGL(check_live_kernel, dim3((unsigned)(xb < 64 ? xb : 64), (unsigned)R),
                       dim3(kCheckThreads), 0, s, seq_lens, bt, bt_stride, num_pages, live,
                       status);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(check_mirrors_kernel, dim3(1), dim3(kCheckThreads), 0, s, seq_lens,
                       q_lens, budgets, R, Hkv, want[0], want[1], want[2], status);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (n_fresh > 0) {
    const int64_t fb = (n_fresh + kCheckThreads - 1) / kCheckThreads;
    hipLaunchKernelGGL(check_fresh_kernel, dim3((unsigned)(fb < 4096 ? fb : 4096)),
                       dim3(kCheckThreads), 0, s, free_pages, n_fresh, num_pages, live, seen,
                       status);
    e = hipGetLastError();
  }
  return e;
}

}  // namespace actkv
