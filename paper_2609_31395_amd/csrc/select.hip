// Eviction: per (request, KV head) keep the k = min(budget, L) entries with the largest
// max-pooled score, ties to the lower token index (Alg. 1 step 5, TopK), emitted in
// ascending token order.
//
// One 1024-thread workgroup per (request, KV head).  Every decision below is made on an
// unsigned key derived from the fp32 bit pattern that orders exactly like the float, so the
// result is exact and deterministic.
//   pool    the raw scores of the segment are staged in LDS (coalesced), max-pooled over
//           the window (clipped at the ends) and written back in place; the pooled scores
//           also go to `pooled` in global memory.  Segments longer than the LDS capacity
//           run the same passes on `pooled` itself.
//   radix   four 8-bit digit passes (LDS histogram, most significant first) find the bit
//           pattern tau of the k-th largest key and how many keys equal to tau to take.
//   emit    each thread owns a contiguous run of the segment; two workgroup prefix sums
//           (equal-to-tau counts, then kept counts) give every thread its output offset,
//           so the kept indices come out in ascending order.
#include "device_common.hpp"

namespace actkv {

namespace {

constexpr int kSelectThreads = 1024;
constexpr int kSelectLdsKeys = 40000;     // segment length kept in LDS (160,000 bytes)
constexpr int kMaxPerThread = (kSelectLdsKeys + kSelectThreads - 1) / kSelectThreads;   // 40

// Unsigned key that orders exactly like the float (negative values included; -0 == +0).
__device__ __forceinline__ uint32_t order_key(float v) {
  const uint32_t u = __float_as_uint(v == 0.0f ? 0.0f : v);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Among bins [0, 256) (higher bin = larger key), find the bin b holding the need-th largest
// element: sum_{b' > b} hist[b'] < need <= sum_{b' >= b} hist[b'].  Returns b and the count
// strictly above it through LDS.
__device__ void find_bin(const uint32_t* hist, uint32_t need, int64_t* scan_tmp, int* bin_out,
                         uint32_t* above_out) {
  const int t = threadIdx.x;
  const uint32_t s = t < 256 ? hist[255 - t] : 0u;   // thread t covers bin 255 - t
  int64_t total;
  const int64_t ex = block_excl_scan_i64(s, scan_tmp, &total);
  if (t < 256 && (uint64_t)ex < need && need <= (uint64_t)(ex + s)) {
    *bin_out = 255 - t;
    *above_out = (uint32_t)ex;
  }
  __syncthreads();
}

}  // namespace

__global__ __launch_bounds__(kSelectThreads) void select_kernel(DevProblem dp,
                                                                const float* __restrict__ scores,
                                                                float* pooled,
                                                                int32_t* __restrict__ kept) {
  extern __shared__ float lds_vals[];
  __shared__ uint32_t hist[256];
  __shared__ int64_t scan_tmp[17];
  __shared__ int s_bin;
  __shared__ uint32_t s_above;

  const int h = blockIdx.x, r = blockIdx.y, Hkv = dp.Hkv;
  const ReqPlan pl = dp.plan[r];
  const int L = pl.L;
  const int b = dp.budgets[r * Hkv + h];
  const int k = b < L ? b : L;
  const float* in = scores + pl.seg_off + (int64_t)h * L;
  float* pout = pooled + pl.seg_off + (int64_t)h * L;
  int32_t* kout = kept + dp.kept_off[r * Hkv + h];
  const int hw = dp.pool_window / 2;
  const int tid = threadIdx.x;
  const bool in_lds = L <= kSelectLdsKeys;
  float* vals = in_lds ? lds_vals : pout;   // pooled scores of the segment

  // ---- pool
  if (in_lds) {
    float* raw = lds_vals;
    for (int t = tid; t < L; t += kSelectThreads) raw[t] = in[t];
    __syncthreads();
    float pv[kMaxPerThread];
#pragma unroll
    for (int u = 0; u < kMaxPerThread; ++u) {
      const int t = tid + u * kSelectThreads;
      if (t < L) {
        const int lo = t - hw < 0 ? 0 : t - hw, hi = t + hw >= L ? L - 1 : t + hw;
        float m = raw[t];
        for (int x = lo; x <= hi; ++x) m = fmaxf(m, raw[x]);
        pv[u] = m;
      }
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < kMaxPerThread; ++u) {
      const int t = tid + u * kSelectThreads;
      if (t < L) {
        pout[t] = pv[u];
        vals[t] = pv[u];
      }
    }
  } else {
    for (int t = tid; t < L; t += kSelectThreads) {
      const int lo = t - hw < 0 ? 0 : t - hw, hi = t + hw >= L ? L - 1 : t + hw;
      float m = in[t];
      for (int x = lo; x <= hi; ++x) m = fmaxf(m, in[x]);
      pout[t] = m;
    }
  }
  __syncthreads();
  if (k <= 0) return;
  if (k >= L) {
    for (int t = tid; t < L; t += kSelectThreads) kout[t] = t;
    return;
  }

  // ---- radix select: four 8-bit digits, most significant first
  uint32_t need = (uint32_t)k, prefix = 0;
#pragma unroll 1
  for (int pass = 0; pass < 4; ++pass) {
    const int sh = 24 - 8 * pass;
    if (tid < 256) hist[tid] = 0;
    __syncthreads();
    for (int t = tid; t < L; t += kSelectThreads) {
      const uint32_t key = order_key(vals[t]);
      // keys whose higher digits match the prefix found so far
      if (pass == 0 || (key >> (sh + 8)) == prefix) atomicAdd(&hist[(key >> sh) & 255u], 1u);
    }
    __syncthreads();
    find_bin(hist, need, scan_tmp, &s_bin, &s_above);
    need -= s_above;
    prefix = (prefix << 8) | (uint32_t)s_bin;
  }
  const uint32_t tau = prefix;   // order key of the k-th largest pooled score

  // ---- emit: all keys > tau, then the first `need` keys == tau, in index order
  const int per = (L + kSelectThreads - 1) / kSelectThreads;
  const int t0 = tid * per < L ? tid * per : L, t1 = t0 + per < L ? t0 + per : L;
  uint32_t n_gt = 0, n_eq = 0;
  for (int t = t0; t < t1; ++t) {
    const uint32_t key = order_key(vals[t]);
    n_gt += key > tau;
    n_eq += key == tau;
  }
  int64_t tot;
  const int64_t eq_before = block_excl_scan_i64(n_eq, scan_tmp, &tot);
  int64_t eq_take = (int64_t)need - eq_before;
  eq_take = eq_take < 0 ? 0 : (eq_take > n_eq ? n_eq : eq_take);
  const int64_t at0 = block_excl_scan_i64(n_gt + eq_take, scan_tmp, &tot);
  int32_t* o = kout + at0;
  int64_t taken = 0;
  for (int t = t0; t < t1; ++t) {
    const uint32_t key = order_key(vals[t]);
    if (key > tau) {
      *o++ = t;
    } else if (key == tau && taken < eq_take) {
      *o++ = t;
      ++taken;
    }
  }
}

hipError_t launch_select(const DevProblem& dp, const HostPlan& hp, const float* scores,
                         float* pooled, int32_t* kept, hipStream_t s) {
  if (hp.R == 0) return hipSuccess;
  const int64_t keys = hp.max_L < kSelectLdsKeys ? hp.max_L : kSelectLdsKeys;
  const size_t lds = (size_t)(keys > 0 ? keys : 1) * sizeof(uint32_t);
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void*)select_kernel,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(select_kernel, dim3(hp.Hkv, hp.R), dim3(kSelectThreads), lds, s, dp, scores,
                     pooled, kept);
  return hipGetLastError();
}

}  // namespace actkv
