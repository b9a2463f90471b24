// Eviction: per (request, KV head) keep the k = min(budget, L) entries with the largest
// max-pooled score, ties to the lower token index (Alg. 1 step 5, TopK), emitted in
// ascending token order.
//
// One 1024-thread workgroup per (request, KV head).  Every decision below is made on an
// unsigned key derived from the fp32 bit pattern that orders exactly like the float, so the
// result is exact and deterministic.
//   pool    the raw scores of the segment are staged in LDS (coalesced loads, all in
//           flight at once) and max-pooled over the window (clipped at the ends); the
//           pooled scores go to `pooled` in global memory and their order keys stay in
//           registers, then replace the raw scores in LDS.  Segments longer than the LDS
//           capacity run the same passes on `pooled` itself.
//   radix   three digit passes of 11, 11 and 10 bits over the register-resident keys (LDS
//           histogram, most significant first) find the bit pattern tau of the k-th largest key and how many keys equal
//           to tau to take.  The first digit spans the exponent and two mantissa bits, so
//           even densely packed scores spread over many bins (few atomic collisions).
//   emit    each thread owns a contiguous run of the segment; two workgroup prefix sums
//           (equal-to-tau counts, then kept counts) give every thread its output offset,
//           so the kept indices come out in ascending order.
#include "device_common.hpp"

namespace actkv {

namespace {

constexpr int kSelectThreads = 1024;
constexpr int kSelectLdsKeys = 38400;     // segment length kept in LDS (153,600 bytes)
constexpr int kMaxBins = 2048;            // largest digit: 11 bits
constexpr int kDigits = 3;                // bits 31..21, 20..10, 9..0
constexpr int kMaxPerThread = (kSelectLdsKeys + kSelectThreads - 1) / kSelectThreads;   // 38

// Unsigned key that orders exactly like the float (negative values included; -0 == +0).
__device__ __forceinline__ uint32_t order_key(float v) {
  const uint32_t u = __float_as_uint(v == 0.0f ? 0.0f : v);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Among bins [0, nbins) (higher bin = larger key), find the bin b holding the need-th
// largest element: sum_{b' > b} hist[b'] < need <= sum_{b' >= b} hist[b'].  Thread t covers
// the nbins / kSelectThreads bins counted down from the top.  Returns b and the count
// strictly above it through LDS.
__device__ void find_bin(const uint32_t* hist, int nbins, uint32_t need, int64_t* scan_tmp,
                         int* bin_out, uint32_t* above_out) {
  const int t = threadIdx.x, per = nbins / kSelectThreads;   // 1 or 2
  const int top = nbins - 1 - t * per;                        // this thread's highest bin
  uint32_t s = 0;
  for (int u = 0; u < per; ++u) s += hist[top - u];
  int64_t total;
  const int64_t ex = block_excl_scan_i64(s, scan_tmp, &total);
  if ((uint64_t)ex < need && need <= (uint64_t)(ex + s)) {
    uint32_t above = (uint32_t)ex;
    for (int u = 0; u < per; ++u) {
      const uint32_t c = hist[top - u];
      if (need <= above + c) {
        *bin_out = top - u;
        *above_out = above;
        break;
      }
      above += c;
    }
  }
  __syncthreads();
}

}  // namespace

// Segments that fit in LDS: the pooled order keys stay in registers (strided ownership,
// element tid + u * kSelectThreads) through the radix passes and in LDS for the emit.
__device__ void select_lds(int L, int k, int hw, const float* __restrict__ in, float* pout,
                           int32_t* __restrict__ kout, uint32_t* lds, uint32_t* hist,
                           int64_t* scan_tmp, int* s_bin, uint32_t* s_above) {
  const int tid = threadIdx.x;
  float* raw = reinterpret_cast<float*>(lds);
  {
    // every load of this thread in flight at once, then into LDS
    float rv[kMaxPerThread];
#pragma unroll
    for (int u = 0; u < kMaxPerThread; ++u) {
      const int t = tid + u * kSelectThreads;
      rv[u] = t < L ? in[t] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < kMaxPerThread; ++u) {
      const int t = tid + u * kSelectThreads;
      if (t < L) raw[t] = rv[u];
    }
  }
  __syncthreads();

  // ---- pool: max over [t - hw, t + hw] clipped to the segment.  For hw <= 3 a fixed
  // 7-tap window whose out-of-window taps repeat the window edge (max is idempotent).
  uint32_t key[kMaxPerThread];
#pragma unroll
  for (int u = 0; u < kMaxPerThread; ++u) {
    const int t = tid + u * kSelectThreads;
    key[u] = 0u;
    if (t < L) {
      float m = raw[t];
      if (hw <= 3) {
#pragma unroll
        for (int d = 1; d <= 3; ++d) {
          const int dd = d <= hw ? d : hw;
          const int a = t - dd < 0 ? 0 : t - dd, c = t + dd >= L ? L - 1 : t + dd;
          m = fmaxf(m, fmaxf(raw[a], raw[c]));
        }
      } else {
        const int lo = t - hw < 0 ? 0 : t - hw, hi = t + hw >= L ? L - 1 : t + hw;
        for (int x = lo; x <= hi; ++x) m = fmaxf(m, raw[x]);
      }
      pout[t] = m;
      key[u] = order_key(m);
    }
  }
  __syncthreads();   // every read of the raw scores is done: LDS now holds the keys
#pragma unroll
  for (int u = 0; u < kMaxPerThread; ++u) {
    const int t = tid + u * kSelectThreads;
    if (t < L) lds[t] = key[u];
  }
  if (k <= 0) return;
  if (k >= L) {
    for (int t = tid; t < L; t += kSelectThreads) kout[t] = t;
    return;
  }

  // ---- radix select: digits of 11, 11 and 10 bits, most significant first
  uint32_t need = (uint32_t)k, prefix = 0;
#pragma unroll 1
  for (int pass = 0; pass < kDigits; ++pass) {
    const int bits = pass == 2 ? 10 : 11, sh = pass == 0 ? 21 : (pass == 1 ? 10 : 0);
    const int nbins = 1 << bits;
    for (int bb = tid; bb < nbins; bb += kSelectThreads) hist[bb] = 0;
    __syncthreads();
#pragma unroll
    for (int u = 0; u < kMaxPerThread; ++u) {
      const int t = tid + u * kSelectThreads;
      // keys whose higher digits match the prefix found so far
      if (t < L && (pass == 0 || (key[u] >> (sh + bits)) == prefix))
        atomicAdd(&hist[(key[u] >> sh) & (uint32_t)(nbins - 1)], 1u);
    }
    __syncthreads();
    find_bin(hist, nbins, need, scan_tmp, s_bin, s_above);
    need -= *s_above;
    prefix = (prefix << bits) | (uint32_t)*s_bin;
  }
  const uint32_t tau = prefix;   // order key of the k-th largest pooled score

  // ---- emit: all keys > tau, then the first `need` keys == tau, in index order.  Thread
  // tid owns the contiguous run [tid * per, tid * per + per); an odd run length keeps the
  // lanes' LDS reads on distinct banks.
  const int per = ((L + kSelectThreads - 1) / kSelectThreads) | 1;
  const int t0 = tid * per < L ? tid * per : L, t1 = t0 + per < L ? t0 + per : L;
  uint32_t rk[kMaxPerThread + 1];
  uint32_t n_gt = 0, n_eq = 0;
#pragma unroll
  for (int i = 0; i < kMaxPerThread + 1; ++i) {
    rk[i] = t0 + i < t1 ? lds[t0 + i] : 0u;
    n_gt += t0 + i < t1 && rk[i] > tau;
    n_eq += t0 + i < t1 && rk[i] == tau;
  }
  int64_t tot;
  const int64_t eq_before = block_excl_scan_i64(n_eq, scan_tmp, &tot);
  int64_t eq_take = (int64_t)need - eq_before;
  eq_take = eq_take < 0 ? 0 : (eq_take > n_eq ? n_eq : eq_take);
  const int64_t at0 = block_excl_scan_i64(n_gt + eq_take, scan_tmp, &tot);
  // branch-free positions (predicated stores, no pointer updates under divergent control)
  int pos = 0, taken = 0;
#pragma unroll
  for (int i = 0; i < kMaxPerThread + 1; ++i) {
    const bool valid = t0 + i < t1;
    const bool gt = valid && rk[i] > tau;
    const bool eq = valid && rk[i] == tau && taken < eq_take;
    taken += eq ? 1 : 0;
    if (gt || eq) kout[at0 + pos] = t0 + i;
    pos += (gt || eq) ? 1 : 0;
  }
}

// Segments longer than the LDS capacity: the same steps on the pooled scores in global
// memory.
__device__ void select_global(int L, int k, int hw, const float* __restrict__ in, float* pout,
                              int32_t* __restrict__ kout, uint32_t* hist, int64_t* scan_tmp,
                              int* s_bin, uint32_t* s_above) {
  const int tid = threadIdx.x;
  for (int t = tid; t < L; t += kSelectThreads) {
    const int lo = t - hw < 0 ? 0 : t - hw, hi = t + hw >= L ? L - 1 : t + hw;
    float m = in[t];
    for (int x = lo; x <= hi; ++x) m = fmaxf(m, in[x]);
    pout[t] = m;
  }
  __threadfence_block();
  __syncthreads();
  if (k <= 0) return;
  if (k >= L) {
    for (int t = tid; t < L; t += kSelectThreads) kout[t] = t;
    return;
  }
  uint32_t need = (uint32_t)k, prefix = 0;
#pragma unroll 1
  for (int pass = 0; pass < kDigits; ++pass) {
    const int bits = pass == 2 ? 10 : 11, sh = pass == 0 ? 21 : (pass == 1 ? 10 : 0);
    const int nbins = 1 << bits;
    for (int bb = tid; bb < nbins; bb += kSelectThreads) hist[bb] = 0;
    __syncthreads();
    for (int t = tid; t < L; t += kSelectThreads) {
      const uint32_t key = order_key(pout[t]);
      if (pass == 0 || (key >> (sh + bits)) == prefix)
        atomicAdd(&hist[(key >> sh) & (uint32_t)(nbins - 1)], 1u);
    }
    __syncthreads();
    find_bin(hist, nbins, need, scan_tmp, s_bin, s_above);
    need -= *s_above;
    prefix = (prefix << bits) | (uint32_t)*s_bin;
  }
  const uint32_t tau = prefix;
  const int per = (L + kSelectThreads - 1) / kSelectThreads;
  const int t0 = tid * per < L ? tid * per : L, t1 = t0 + per < L ? t0 + per : L;
  uint32_t n_gt = 0, n_eq = 0;
  for (int t = t0; t < t1; ++t) {
    const uint32_t key = order_key(pout[t]);
    n_gt += key > tau;
    n_eq += key == tau;
  }
  int64_t tot;
  const int64_t eq_before = block_excl_scan_i64(n_eq, scan_tmp, &tot);
  int64_t eq_take = (int64_t)need - eq_before;
  eq_take = eq_take < 0 ? 0 : (eq_take > n_eq ? n_eq : eq_take);
  const int64_t at0 = block_excl_scan_i64(n_gt + eq_take, scan_tmp, &tot);
  int pos = 0, taken = 0;
  for (int t = t0; t < t1; ++t) {
    const uint32_t key = order_key(pout[t]);
    const bool gt = key > tau, eq = key == tau && taken < eq_take;
    taken += eq ? 1 : 0;
    if (gt || eq) kout[at0 + pos] = t;
    pos += (gt || eq) ? 1 : 0;
  }
}

__global__ __launch_bounds__(kSelectThreads) void select_kernel(DevProblem dp,
                                                                const float* __restrict__ scores,
                                                                float* pooled,
                                                                int32_t* __restrict__ kept) {
  extern __shared__ uint32_t lds_keys[];
  __shared__ uint32_t hist[kMaxBins];
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
  if (L <= kSelectLdsKeys)
    select_lds(L, k, hw, in, pout, kout, lds_keys, hist, scan_tmp, &s_bin, &s_above);
  else
    select_global(L, k, hw, in, pout, kout, hist, scan_tmp, &s_bin, &s_above);
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
