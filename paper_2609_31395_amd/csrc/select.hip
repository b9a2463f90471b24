// Eviction: per (request, KV head) keep the k = min(budget, L) entries with the largest
// max-pooled score, ties to the lower token index (Alg. 1 step 5, TopK), emitted in
// ascending token order.
//
// One 1024-thread workgroup per (request, KV head):
//   pass 0  max-pool the raw scores (window w, clipped at the ends) into `pooled` and build
//           a 2048-bin LDS histogram of bits 31..21 of each score's bit pattern (scores are
//           >= 0, so the unsigned bit pattern orders like the float);
//   pass 1  histogram of bits 20..10 among entries whose top digit equals the k-th
//           largest's;  pass 2  bits 9..0 likewise -> the exact k-th largest pattern tau
//           and how many entries equal to tau must be taken;
//   emit    in index order, keep every entry > tau and the first `need` entries == tau;
//           positions come from a workgroup prefix count, so the output is ascending.
// Every decision is on the fp32 bit patterns: the result is exact and deterministic.
#include "device_common.hpp"

namespace actkv {

namespace {

__device__ __forceinline__ uint32_t order_key(float v) {
  // +0 and -0 are the same score; scores are non-negative so the bit pattern orders them
  return __float_as_uint(v == 0.0f ? 0.0f : v);
}

// Among bins [0, nbins) (higher bin = larger key), find the bin b holding the need-th
// largest element: sum_{b' > b} hist[b'] < need <= sum_{b' >= b} hist[b'].  Returns b and
// the count strictly above it.  Requires blockDim.x == 1024 and nbins in {1024, 2048}.
__device__ void find_bin(const uint32_t* hist, int nbins, uint32_t need, int64_t* scan_tmp,
                         int* bin_out, uint32_t* above_out) {
  const int per = nbins / 1024;
  const int t = threadIdx.x;
  // thread t covers bins nbins-1-per*t down to nbins-per*(t+1)
  uint32_t s = 0;
  for (int i = 0; i < per; ++i) s += hist[nbins - 1 - per * t - i];
  int64_t total;
  const int64_t ex = block_excl_scan_i64(s, scan_tmp, &total);
  if ((uint64_t)ex < need && need <= (uint64_t)(ex + s)) {
    uint32_t acc = (uint32_t)ex;
    for (int i = 0; i < per; ++i) {
      const int b = nbins - 1 - per * t - i;
      if (need <= acc + hist[b]) { *bin_out = b; *above_out = acc; break; }
      acc += hist[b];
    }
  }
  __syncthreads();
}

}  // namespace

__global__ __launch_bounds__(1024) void select_kernel(DevProblem dp, const float* __restrict__ scores,
                                                      float* pooled, int32_t* __restrict__ kept) {
  __shared__ uint32_t hist[2048];
  __shared__ int64_t scan_tmp[17];
  __shared__ uint32_t cnt_tmp[17];
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

  for (int i = tid; i < 2048; i += 1024) hist[i] = 0;
  __syncthreads();
  // pass 0: pool + top-digit histogram
  for (int t = tid; t < L; t += 1024) {
    float m = in[t];
    const int lo = t - hw < 0 ? 0 : t - hw, hi = t + hw >= L ? L - 1 : t + hw;
    for (int u = lo; u <= hi; ++u) m = fmaxf(m, in[u]);
    pout[t] = m;
    atomicAdd(&hist[order_key(m) >> 21], 1u);
  }
  __syncthreads();
  if (k <= 0) return;
  if (k >= L) {
    for (int t = tid; t < L; t += 1024) kout[t] = t;
    return;
  }
  uint32_t need = (uint32_t)k;
  uint32_t prefix = 0;
  // three radix digits: 11, 11 and 10 bits
  const int shifts[3] = {21, 10, 0};
  const int widths[3] = {11, 11, 10};
  for (int pass = 0; pass < 3; ++pass) {
    if (pass > 0) {
      for (int i = tid; i < 2048; i += 1024) hist[i] = 0;
      __syncthreads();
      const int hi_shift = shifts[pass - 1];
      const int sh = shifts[pass];
      const uint32_t mask = (1u << widths[pass]) - 1u;
      for (int t = tid; t < L; t += 1024) {
        const uint32_t key = order_key(pout[t]);
        if ((key >> hi_shift) == prefix) atomicAdd(&hist[(key >> sh) & mask], 1u);
      }
      __syncthreads();
    }
    find_bin(hist, 1 << widths[pass], need, scan_tmp, &s_bin, &s_above);
    need -= s_above;
    prefix = (prefix << widths[pass]) | (uint32_t)s_bin;
    __syncthreads();
  }
  const uint32_t tau = prefix;   // bit pattern of the k-th largest pooled score
  // emit: all > tau, then the first `need` entries equal to tau, in index order
  uint32_t eq_seen = 0, kept_so_far = 0;
  for (int base = 0; base < L; base += 1024) {
    const int t = base + tid;
    const uint32_t key = t < L ? order_key(pout[t]) : 0u;
    const bool gt = t < L && key > tau;
    const bool eq = t < L && key == tau;
    uint32_t eq_tot, keep_tot;
    const uint32_t eq_rank = eq_seen + block_excl_count(eq, cnt_tmp, &eq_tot);
    const bool keep = gt || (eq && eq_rank < need);
    const uint32_t at = kept_so_far + block_excl_count(keep, cnt_tmp, &keep_tot);
    if (keep) kout[at] = t;
    eq_seen += eq_tot;
    kept_so_far += keep_tot;
  }
}

hipError_t launch_select(const DevProblem& dp, const HostPlan& hp, const float* scores,
                         float* pooled, int32_t* kept, hipStream_t s) {
  if (hp.R == 0) return hipSuccess;
  hipLaunchKernelGGL(select_kernel, dim3(hp.Hkv, hp.R), dim3(1024), 0, s, dp, scores, pooled,
                     kept);
  return hipGetLastError();
}

}  // namespace actkv
