// Confidence-driven budget allocation (Sec. 6.1 confidence monitor; Alg. 2).
//
// Token confidence (Alg. 2 step 1, GetTokenConf): for one row of logits x over the
// vocabulary, T = -(1/k) sum_{j<=k} log P(j) = LSE(x) - (1/k) sum of the k largest logits.
//   token_conf_partial_kernel  one 256-thread workgroup per (row, chunk of <= 16384 logits):
//                              an online (max, sum of exp) over the chunk, and the chunk's
//                              k largest logits by a 4-pass radix select on order keys
//                              staged in LDS (exact; emitted as a multiset)
//   token_conf_merge_kernel    one workgroup per row: the chunks' (max, sum) combined in chunk
//                              order, the candidates sorted (bitonic, LDS), the k largest
//                              summed in fp64 in sorted order, T written as fp32
// Trace confidence, trend and budget (Alg. 2 steps 2-4): budget_kernel, one 1024-thread
// workgroup per request: min-pooled windows into LDS, the two order statistics of the
// percentile by radix select, the retained windows compacted in window order (in place),
// then one thread sums them in that order in fp64 with every operation rounded on its own,
// so the slope -- and the integer decision it drives -- is reproducible bit for bit.
#include "device_common.hpp"

namespace actkv {

namespace {

constexpr int kConfThreads = 256;
constexpr int kConfChunk = kConfChunkLogits;
constexpr int kConfMaxCand = kConfMaxSplits * kConfMaxTopK;   // 1024 merge candidates
constexpr int kBudgetThreads = 1024;

__device__ __forceinline__ uint32_t order_key_f(float v) {
  const uint32_t u = __float_as_uint(v == 0.0f ? 0.0f : v);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float key_value_f(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

// (m, s) <- the combination of two partial (max, sum of exp(x - max)) pairs.
__device__ __forceinline__ void lse_combine(float& m, float& s, float m2, float s2) {
  const float M = fmaxf(m, m2);
  if (M == -__builtin_inff()) return;   // both empty
  s = (m == -__builtin_inff() ? 0.0f : s * expf(m - M)) +
      (m2 == -__builtin_inff() ? 0.0f : s2 * expf(m2 - M));
  m = M;
}

// Radix select on 32-bit keys key_of(i), i < n (read from LDS): the key of rank `need`
// counted from the top (descending, need >= 1) or from the bottom (ascending), four 8-bit
// digits, most significant first.  Returns the key; *left gets how many keys equal to it
// are still needed.  nthreads threads; hist is 256 words; ctl 2 words.
template <bool kDescending, typename KeyOf>
__device__ uint32_t radix_rank(KeyOf key_of, int n, uint32_t need, uint32_t* hist,
                               uint32_t* ctl, int nthreads, uint32_t* left) {
  const int tid = threadIdx.x;
  uint32_t prefix = 0;
#pragma unroll 1
  for (int sh = 24; sh >= 0; sh -= 8) {
    for (int b = tid; b < 256; b += nthreads) hist[b] = 0;
    __syncthreads();
    for (int i = tid; i < n; i += nthreads) {
      const uint32_t dh = key_of(i) >> sh;   // this digit and the ones above it
      if ((dh >> 8) == prefix) atomicAdd(&hist[dh & 255u], 1u);
    }
    __syncthreads();
    if (tid < 64) {   // wave 0: 4 bins per lane, scanned in selection order
      uint32_t c[4], tot = 0;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int bin = kDescending ? 255 - (tid * 4 + u) : tid * 4 + u;
        c[u] = hist[bin];
        tot += c[u];
      }
      uint32_t incl = tot;
#pragma unroll
      for (int d = 1; d < 64; d <<= 1) {
        const uint32_t o = __shfl_up(incl, d, 64);
        if (tid >= d) incl += o;
      }
      uint32_t before = incl - tot;
      if (before < need && need <= incl) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          if (before < need && need <= before + c[u]) {
            ctl[0] = kDescending ? 255 - (tid * 4 + u) : tid * 4 + u;
            ctl[1] = before;
          }
          before += c[u];
        }
      }
    }
    __syncthreads();
    prefix = (prefix << 8) | ctl[0];
    need -= ctl[1];
    __syncthreads();
  }
  *left = need;
  return prefix;
}

}  // namespace

__global__ __launch_bounds__(kConfThreads) void token_conf_partial_kernel(
    const float* __restrict__ logits, int64_t vocab, int64_t row_stride, int k, int splits,
    float2* __restrict__ ms_out, float* __restrict__ top_out) {
  __shared__ uint32_t keys[kConfChunk];
  __shared__ uint32_t hist[256];
  __shared__ uint32_t ctl[4];
  __shared__ float2 wred[kConfThreads / 64];
  const int tid = threadIdx.x, split = blockIdx.x;
  const int64_t row = blockIdx.y;
  const int64_t c0 = (int64_t)split * kConfChunk;
  const int n = (int)(vocab - c0 < kConfChunk ? vocab - c0 : kConfChunk);
  const float* x = logits + row * row_stride + c0;
  const float ninf = -__builtin_inff();
  // pass 1: keys into LDS, online (max, sum)
  float m = ninf, s = 0.0f;
  for (int i = tid; i < n; i += kConfThreads) {
    const float v = x[i];
    keys[i] = order_key_f(v);
    if (v > m) {
      s = (m == ninf ? 0.0f : s * expf(m - v)) + 1.0f;
      m = v;
    } else if (v > ninf) {
      s += expf(v - m);
    }
  }
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) {
    const float m2 = __shfl_xor(m, d, 64), s2 = __shfl_xor(s, d, 64);
    lse_combine(m, s, m2, s2);
  }
  if ((tid & 63) == 0) wred[tid >> 6] = make_float2(m, s);
  __syncthreads();
  const int64_t slot = row * splits + split;
  if (tid == 0) {
    float M = wred[0].x, S = wred[0].y;
    for (int w = 1; w < kConfThreads / 64; ++w) lse_combine(M, S, wred[w].x, wred[w].y);
    ms_out[slot] = make_float2(M, S);
    ctl[2] = 0;
  }
  // the chunk's kk = min(k, n) largest logits
  const int kk = k < n ? k : n;
  float* top = top_out + slot * k;
  for (int j = kk + tid; j < k; j += kConfThreads) top[j] = ninf;   // padding
  if (kk <= 0) return;
  uint32_t left;
  const uint32_t tau = radix_rank<true>([&](int i) { return keys[i]; }, n, (uint32_t)kk, hist,
                                         ctl, kConfThreads, &left);
  // every key above tau, then `left` copies of tau (a multiset: order is irrelevant)
  for (int i = tid; i < n; i += kConfThreads)
    if (keys[i] > tau) top[atomicAdd(&ctl[2], 1u)] = key_value_f(keys[i]);
  __syncthreads();
  const int gt = (int)ctl[2];
  for (int j = tid; j < (int)left; j += kConfThreads) top[gt + j] = key_value_f(tau);
}

__global__ __launch_bounds__(kConfThreads) void token_conf_merge_kernel(
    const float2* __restrict__ ms, const float* __restrict__ top_in, int k, int splits,
    int64_t vocab, float* __restrict__ conf) {
  __shared__ float cand[kConfMaxCand];
  const int tid = threadIdx.x;
  const int64_t row = blockIdx.x;
  const int nc = splits * k;
  int p2 = 1;
  while (p2 < nc) p2 <<= 1;
  for (int i = tid; i < p2; i += kConfThreads)
    cand[i] = i < nc ? top_in[row * nc + i] : -__builtin_inff();
  __syncthreads();
  // bitonic sort, descending
  for (int size = 2; size <= p2; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = tid; i < p2 / 2; i += kConfThreads) {
        const int lo = 2 * i - (i & (stride - 1));
        const int hi = lo + stride;
        const bool desc = (lo & size) == 0;
        const float a = cand[lo], b = cand[hi];
        if (desc ? (a < b) : (a > b)) { cand[lo] = b; cand[hi] = a; }
      }
      __syncthreads();
    }
  }
  if (tid == 0) {
    float M = -__builtin_inff(), S = 0.0f;
    for (int c = 0; c < splits; ++c) lse_combine(M, S, ms[row * splits + c].x, ms[row * splits + c].y);
    const double lse = (double)M + log((double)S);
    // the k largest logits of the row are the first min(k, vocab) candidates in sorted order
    // (every chunk contributed its own min(k, chunk) largest; padding sorts last)
    const int kk = (int64_t)k < vocab ? k : (int)vocab;
    double sum = 0.0;
    for (int j = 0; j < kk; ++j) sum += (double)cand[j];
    conf[row] = (float)(lse - sum / (double)kk);
  }
}

// ---- Alg. 2 steps 2-4 -------------------------------------------------------------------
__global__ __launch_bounds__(kBudgetThreads) void budget_kernel(
    const float* __restrict__ tconf, const int64_t* __restrict__ offsets, int window,
    int stride, float bottom_pct, float scale_up, int budget_upper,
    const int32_t* __restrict__ budgets_in, int32_t* __restrict__ budgets_out,
    double* __restrict__ slopes, double* __restrict__ thresholds, int32_t* __restrict__ retained) {
#pragma clang fp contract(off)
  __shared__ float rp[kMaxBudgetWindows];       // R'_m, then the retained values in order
  __shared__ int32_t rm[kMaxBudgetWindows];     // window index of each retained value
  __shared__ uint32_t hist[256];
  __shared__ uint32_t ctl[4];
  __shared__ int64_t scan_tmp[17];
  __shared__ uint32_t mm_tmp[kBudgetThreads / 64];
  const int r = blockIdx.x, tid = threadIdx.x;
  const int64_t n = offsets[r + 1] - offsets[r];
  const float* t = tconf + offsets[r];
  double alpha = 0.0, q = __builtin_nan("");
  int kept = 0;
  if (n >= window) {
    const int M = (int)((n - window) / stride + 1);
    for (int m = tid; m < M; m += kBudgetThreads) {
      float v = t[(int64_t)m * stride];
      for (int i = 1; i < window; ++i) v = fminf(v, t[(int64_t)m * stride + i]);
      rp[m] = v;
    }
    __syncthreads();
    // percentile: order statistics lo and lo + 1 (ascending), linear interpolation
    const double pos = ((double)bottom_pct / 100.0) * (double)(M - 1);
    const int lo = (int)floor(pos);
    const double frac = pos - (double)lo;
    uint32_t left;
    auto key_of = [&](int i) { return order_key_f(rp[i]); };
    const uint32_t klo = radix_rank<false>(key_of, M, (uint32_t)lo + 1u, hist, ctl,
                                           kBudgetThreads, &left);
    const double vlo = (double)key_value_f(klo);
    double vhi = vlo;
    if (lo + 1 < M) {
      // the next order statistic: klo again if enough keys equal it, else the smallest above
      uint32_t cnt_le = 0, next = 0xFFFFFFFFu;
      for (int m = tid; m < M; m += kBudgetThreads) {
        const uint32_t km = key_of(m);
        cnt_le += km <= klo;
        if (km > klo) next = min(next, km);
      }
      int64_t tot;
      block_excl_scan_i64(cnt_le, scan_tmp, &tot);
#pragma unroll
      for (int d = 32; d >= 1; d >>= 1) next = min(next, (uint32_t)__shfl_xor((int)next, d, 64));
      if ((tid & 63) == 0) mm_tmp[tid >> 6] = next;
      __syncthreads();
      for (int w = 0; w < kBudgetThreads / 64; ++w) next = min(next, mm_tmp[w]);
      vhi = tot >= (int64_t)lo + 2 ? vlo : (double)key_value_f(next);
      q = vlo + frac * (vhi - vlo);
    } else {
      q = vlo;
    }
    // retained windows (R'_m <= Q), compacted in window order: each thread reads its
    // contiguous range first, then writes at its scanned offset (never past its range)
    const int per = (M + kBudgetThreads - 1) / kBudgetThreads;
    const int m0 = tid * per < M ? tid * per : M, m1 = m0 + per < M ? m0 + per : M;
    constexpr int kMaxPer = kMaxBudgetWindows / kBudgetThreads;
    float yv[kMaxPer];
    uint32_t cnt = 0;
#pragma unroll
    for (int u = 0; u < kMaxPer; ++u) {
      yv[u] = m0 + u < m1 ? rp[m0 + u] : 0.0f;
      cnt += (m0 + u < m1 && (double)yv[u] <= q) ? 1u : 0u;
    }
    int64_t total;
    int64_t at = block_excl_scan_i64(cnt, scan_tmp, &total);   // its barriers retire the reads
#pragma unroll
    for (int u = 0; u < kMaxPer; ++u)
      if (m0 + u < m1 && (double)yv[u] <= q) {
        rp[at] = yv[u];
        rm[at] = m0 + u;
        ++at;
      }
    __syncthreads();
    kept = (int)total;
    if (tid == 0 && kept >= 2) {   // least squares in window order
      double sx = 0.0, sy = 0.0;
      for (int i = 0; i < kept; ++i) {
        sx = sx + (double)rm[i];
        sy = sy + (double)rp[i];
      }
      const double mx = sx / (double)kept, my = sy / (double)kept;
      double num = 0.0, den = 0.0;
      for (int i = 0; i < kept; ++i) {
        const double dx = (double)rm[i] - mx, dy = (double)rp[i] - my;
        num = num + dx * dy;
        den = den + dx * dx;
      }
      alpha = num / den;
    }
  }
  if (tid == 0) {
    int32_t b = budgets_in[r];
    if (alpha < 0.0) {
      const double grown = floor((double)b * (double)scale_up);
      b = grown < (double)budget_upper ? (int32_t)grown : budget_upper;
    }
    budgets_out[r] = b;
    if (slopes) slopes[r] = alpha;
    if (thresholds) thresholds[r] = q;
    if (retained) retained[r] = kept;
  }
}

int conf_splits(int64_t vocab) { return (int)((vocab + kConfChunk - 1) / kConfChunk); }

hipError_t launch_token_confidence(const float* logits, int64_t rows, int64_t vocab,
                                   int64_t row_stride, int k, float2* ms, float* top,
                                   float* conf, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  const int splits = conf_splits(vocab);
  hipLaunchKernelGGL(token_conf_partial_kernel, dim3(splits, (unsigned)rows), dim3(kConfThreads),
                     0, s, logits, vocab, row_stride, k, splits, ms, top);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(token_conf_merge_kernel, dim3((unsigned)rows), dim3(kConfThreads), 0, s, ms,
                     top, k, splits, vocab, conf);
  return hipGetLastError();
}

hipError_t launch_budget_update(const float* tconf, const int64_t* offsets, int num_reqs,
                                int window, int stride, float bottom_pct, float scale_up,
                                int budget_upper, const int32_t* budgets_in,
                                int32_t* budgets_out, double* slopes, double* thresholds,
                                int32_t* retained, hipStream_t s) {
  if (num_reqs <= 0) return hipSuccess;
  hipLaunchKernelGGL(budget_kernel, dim3(num_reqs), dim3(kBudgetThreads), 0, s, tconf, offsets,
                     window, stride, bottom_pct, scale_up, budget_upper, budgets_in,
                     budgets_out, slopes, thresholds, retained);
  return hipGetLastError();
}

}  // namespace actkv
