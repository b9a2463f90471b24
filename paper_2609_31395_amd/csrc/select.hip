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

// The float whose order_key is k.
__device__ __forceinline__ float key_value(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

// Among bins [0, nbins) (higher bin = larger key), find the bin b holding the need-th
// largest element: sum_{b' > b} hist[b'] < need <= sum_{b' >= b} hist[b'].  Thread t covers
// max(1, nbins / kSelectThreads) bins counted down from the top.  Returns b and the count
// strictly above it through LDS.
__device__ void find_bin(const uint32_t* hist, int nbins, uint32_t need, int64_t* scan_tmp,
                         int* bin_out, uint32_t* above_out) {
  // 1 or 2 bins per thread; threads past the bins of a small histogram hold none
  const int t = threadIdx.x, per = nbins > kSelectThreads ? nbins / kSelectThreads : 1;
  const int top = nbins - 1 - t * per;                        // this thread's highest bin
  uint32_t s = 0;
  for (int u = 0; u < per; ++u) s += top - u >= 0 ? hist[top - u] : 0u;
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

// Block-wide min and max of a per-thread value (every thread gets both).
__device__ __forceinline__ void block_min_max(uint32_t lo, uint32_t hi, uint32_t* tmp,
                                              uint32_t* out_lo, uint32_t* out_hi) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) {
    lo = min(lo, (uint32_t)__shfl_xor((int)lo, d, 64));
    hi = max(hi, (uint32_t)__shfl_xor((int)hi, d, 64));
  }
  if (lane == 0) { tmp[w] = lo; tmp[16 + w] = hi; }
  __syncthreads();
  lo = tmp[0];
  hi = tmp[16];
  for (int i = 1; i < kSelectThreads / 64; ++i) { lo = min(lo, tmp[i]); hi = max(hi, tmp[16 + i]); }
  *out_lo = lo;
  *out_hi = hi;
  __syncthreads();
}

// Segments that fit in LDS.  Thread tid owns the contiguous run [tid * per, tid * per + per)
// (per odd: the lanes' LDS accesses fall on distinct banks); its pooled order keys stay in
// registers from the pool to the emit.
__device__ void select_lds(int L, int k, int hw, const float* __restrict__ in, float* pout,
                           int32_t* __restrict__ kout, uint32_t* lds, uint32_t* hist,
                           int64_t* scan_tmp, uint32_t* mm_tmp, int* s_bin, uint32_t* s_above) {
  constexpr int kRun = kMaxPerThread + 1;   // longest run: odd >= ceil(kSelectLdsKeys / threads)
  const int tid = threadIdx.x;
  float* vals = reinterpret_cast<float*>(lds);
  int32_t* idx = reinterpret_cast<int32_t*>(lds);
  {
    // coalesced staging, every load of this thread in flight at once
    float rv[kMaxPerThread];
#pragma unroll
    for (int u = 0; u < kMaxPerThread; ++u) {
      const int t = tid + u * kSelectThreads;
      rv[u] = t < L ? in[t] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < kMaxPerThread; ++u) {
      const int t = tid + u * kSelectThreads;
      if (t < L) vals[t] = rv[u];
    }
  }
  __syncthreads();

  const int per = ((L + kSelectThreads - 1) / kSelectThreads) | 1;
  const int t0 = tid * per < L ? tid * per : L, t1 = t0 + per < L ? t0 + per : L;
  const int n = t1 - t0;

  // ---- pool: max over [t - hw, t + hw] clipped to the segment, from the run and a halo of
  // 3 on each side held in registers (hw <= 3); a general loop for wider windows
  uint32_t key[kRun];
  if (hw <= 3) {
    // in three chunks of 13 (run + halo of 3 each side in registers)
    constexpr int kHalo = 3, kChunk = kRun / 3;
    static_assert(kRun % 3 == 0, "run splits into three chunks");
#pragma unroll
    for (int c = 0; c < kRun; c += kChunk) {
      float v[kChunk + 2 * kHalo];
#pragma unroll
      for (int i = 0; i < kChunk + 2 * kHalo; ++i) {
        const int t = t0 + c - kHalo + i;
        v[i] = (t >= 0 && t < L && c + i < n + 2 * kHalo) ? vals[t] : -__builtin_inff();
      }
#pragma unroll
      for (int i = 0; i < kChunk; ++i) {
        float m = v[i + kHalo];
#pragma unroll
        for (int d = 1; d <= kHalo; ++d)
          if (d <= hw) m = fmaxf(m, fmaxf(v[i + kHalo - d], v[i + kHalo + d]));
        key[c + i] = order_key(m);
      }
    }
  } else {
#pragma unroll
    for (int i = 0; i < kRun; ++i) {
      const int t = t0 + i;
      float m = -__builtin_inff();
      if (i < n) {
        const int lo = t - hw < 0 ? 0 : t - hw, hi = t + hw >= L ? L - 1 : t + hw;
        for (int x = lo; x <= hi; ++x) m = fmaxf(m, vals[x]);
      }
      key[i] = order_key(m);
    }
  }
  uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
#pragma unroll
  for (int i = 0; i < kRun; ++i)
    if (i < n) { kmin = min(kmin, key[i]); kmax = max(kmax, key[i]); }
  __syncthreads();   // every read of the raw scores is done
  // pooled scores out through LDS, coalesced (the key maps back to the value; -0 reads +0)
#pragma unroll
  for (int i = 0; i < kRun; ++i)
    if (i < n) vals[t0 + i] = key_value(key[i]);
  __syncthreads();
  for (int t = tid; t < L; t += kSelectThreads) pout[t] = vals[t];
  if (k <= 0) return;
  if (k >= L) {
    for (int t = tid; t < L; t += kSelectThreads) kout[t] = t;
    return;
  }

  // ---- radix select on d = key - min key, over the bit width of the segment's key range
  // (digits of up to 11 bits, most significant first): concentrated scores still spread
  // over the whole first histogram.
  uint32_t lo, hi;
  block_min_max(kmin, kmax, mm_tmp, &lo, &hi);
  const uint32_t range = hi - lo;
  int rem = range == 0 ? 0 : 32 - __clz(range);
  uint32_t need = (uint32_t)k, prefix = 0;
#pragma unroll 1
  while (rem > 0) {
    const int bits = rem < 11 ? rem : 11, sh = rem - bits, nbins = 1 << bits;
    for (int bb = tid; bb < nbins; bb += kSelectThreads) hist[bb] = 0;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kRun; ++i) {
      const uint32_t d = key[i] - lo;
      // keys whose higher digits match the prefix found so far (none above the range)
      if (i < n && (uint32_t)(((uint64_t)d) >> (sh + bits)) == prefix)
        atomicAdd(&hist[(d >> sh) & (uint32_t)(nbins - 1)], 1u);
    }
    __syncthreads();
    find_bin(hist, nbins, need, scan_tmp, s_bin, s_above);
    need -= *s_above;
    prefix = (prefix << bits) | (uint32_t)*s_bin;
    rem = sh;
  }
  const uint32_t tau = lo + prefix;   // order key of the k-th largest pooled score

  // ---- emit: all keys > tau, then the first `need` keys == tau, in index order, staged in
  // LDS (positions from two workgroup prefix sums) and written out coalesced
  uint32_t n_gt = 0, n_eq = 0;
#pragma unroll
  for (int i = 0; i < kRun; ++i) {
    n_gt += i < n && key[i] > tau;
    n_eq += i < n && key[i] == tau;
  }
  int64_t tot;
  const int64_t eq_before = block_excl_scan_i64(n_eq, scan_tmp, &tot);
  int64_t eq_take = (int64_t)need - eq_before;
  eq_take = eq_take < 0 ? 0 : (eq_take > n_eq ? n_eq : eq_take);
  const int64_t at0 = block_excl_scan_i64(n_gt + eq_take, scan_tmp, &tot);
  // branch-free positions (predicated stores, no pointer updates under divergent control)
  int pos = 0, taken = 0;
#pragma unroll
  for (int i = 0; i < kRun; ++i) {
    const bool gt = i < n && key[i] > tau;
    const bool eq = i < n && key[i] == tau && taken < eq_take;
    taken += eq ? 1 : 0;
    if (gt || eq) idx[at0 + pos] = t0 + i;
    pos += (gt || eq) ? 1 : 0;
  }
  __syncthreads();
  for (int j = tid; j < k; j += kSelectThreads) kout[j] = idx[j];
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
  __shared__ uint32_t mm_tmp[32];
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
    select_lds(L, k, hw, in, pout, kout, lds_keys, hist, scan_tmp, mm_tmp, &s_bin, &s_above);
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
