// confidence.hip -- the confidence monitor and the budget rule of ActKV's adaptive budget
// allocation (Sec. 6.1; Alg. 2).
//
// Token confidence (Sec. 6.1): T = LSE(x) - (1/k) * (sum of the k largest logits of x), one
// row of logits per generated token.  Two kernels:
//   token_conf_partial_kernel  one 256-thread workgroup per (row, chunk of <= 16384 logits),
//                              64 logits per thread held in registers (all loads issued at
//                              once): the chunk's max, then sum exp(x - max) (hardware exp2,
//                              fixed order),
//                              then the chunk's k largest logits exactly: the k-th largest of
//                              the lanes' maxima in each wave bounds the answer from below,
//                              the few logits above that bound go to LDS, and a bisection on
//                              their order keys finds the k-th largest (a bisection over all
//                              64 registers of every thread when the bound keeps too many,
//                              e.g. a flat row); emitted as a multiset
//   token_conf_merge_kernel    one wave per row: the chunks' sums rescaled to the row max
//                              and added in chunk order, the k largest of the chunks' candidates by the same
//                              bound and bisection, sorted across the lanes (bitonic) and
//                              summed in fp64 in that order, T written as fp32
// Trace confidence, trend and budget (Alg. 2 steps 2-4): budget_kernel, one 1024-thread
// workgroup per request: min-pooled windows into LDS (from minima of gcd(w, s)-token blocks,
// read once and coalesced), the two order statistics of the percentile by radix select, the
// retained windows compacted in window order (in place), then one thread sums them in that
// order in fp64 with every operation rounded on its own, so the slope -- and the integer
// decision it drives -- is reproducible bit for bit.
#include "device_common.hpp"

namespace actkv {

namespace {

constexpr int kConfThreads = 256;
constexpr int kConfWaves = kConfThreads / 64;
constexpr int kConfChunk = kConfChunkLogits;
constexpr int kConfPerThread = kConfChunk / kConfThreads;       // 64 logits per thread
constexpr int kConfCandCap = 2048;                               // LDS candidates per chunk
constexpr int kConfMaxCand = kConfMaxSplits * kConfMaxTopK;      // 1024 merge candidates
constexpr int kMergePerLane = kConfMaxCand / 64;
constexpr int kBudgetThreads = 1024;

static_assert(kConfChunk % kConfThreads == 0, "whole rows of logits per thread");
static_assert(kConfMaxTopK <= 64, "the k largest fit one wave, one per lane");

__device__ __forceinline__ uint32_t order_key_f(float v) {
  const uint32_t u = __float_as_uint(v == 0.0f ? 0.0f : v);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
// The same order with -0 just below +0 (no canonicalisation): three operations.
__device__ __forceinline__ uint32_t order_key_raw(float v) {
  const uint32_t u = __float_as_uint(v);
  return u ^ ((uint32_t)((int32_t)u >> 31) | 0x80000000u);
}
__device__ __forceinline__ float key_value_f(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

__device__ __forceinline__ float wave_max_f(float v) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) v = fmaxf(v, __shfl_xor(v, d, 64));
  return v;
}
__device__ __forceinline__ float wave_sum_f(float v) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) v += __shfl_xor(v, d, 64);
  return v;
}
__device__ __forceinline__ int wave_sum_i(int v) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) v += __shfl_xor(v, d, 64);
  return v;
}
__device__ __forceinline__ uint32_t wave_max_u(uint32_t v) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) v = max(v, (uint32_t)__shfl_xor((int)v, d, 64));
  return v;
}
// Lanes below this one whose bit is set in `mask`.
__device__ __forceinline__ uint32_t lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

// The largest t with at least `need` lanes of the wave holding a key >= t, need in [1, 64]
// (0 when fewer than `need` lanes hold a key >= 1).
__device__ __forceinline__ uint32_t wave_kth_key(uint32_t key, int need) {
  uint32_t p = 0;
#pragma unroll
  for (int b = 31; b >= 0; --b) {
    const uint32_t t = p | (1u << b);
    if ((int)__popcll(__ballot(key >= t)) >= need) p = t;
  }
  return p;
}

// min(v, v of the lane kCtrl names) for a DPP row shift; lanes whose source lies outside
// their row of 16 keep v.
template <int kCtrl>
__device__ __forceinline__ uint32_t min_dpp(uint32_t v) {
  return min(v, (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, kCtrl, 0xf, 0xf, false));
}

// The minimum of v over lanes [i, i + 2^kLg) reaches every lane i that is a multiple of
// 2^kLg (kLg <= 6; other lanes get partial minima).  Within a row of 16 by DPP row shifts
// left, across rows by lane shuffles.
template <int kLg>
__device__ __forceinline__ uint32_t group_min_to_leader(uint32_t v) {
  if constexpr (kLg >= 1) v = min_dpp<0x101>(v);   // row_shl:1
  if constexpr (kLg >= 2) v = min_dpp<0x102>(v);   // row_shl:2
  if constexpr (kLg >= 3) v = min_dpp<0x104>(v);   // row_shl:4
  if constexpr (kLg >= 4) v = min_dpp<0x108>(v);   // row_shl:8
  if constexpr (kLg >= 5) v = min(v, (uint32_t)__shfl_down((int)v, 16, 64));
  if constexpr (kLg >= 6) v = min(v, (uint32_t)__shfl_down((int)v, 32, 64));
  return v;
}

// Start of a bisection for a key in [lo, hi]: *p gets the bits of hi above the highest bit
// where lo and hi differ (zeros below, so *p <= lo); returns how many low bits remain open.
__device__ __forceinline__ int open_bits(uint32_t lo, uint32_t hi, uint32_t* p) {
  if (lo == hi) {
    *p = hi;
    return 0;
  }
  const int nb = 32 - __builtin_clz(lo ^ hi);
  *p = nb == 32 ? 0u : hi & ~((1u << nb) - 1u);
  return nb;
}

// tau = the largest key t >= *tau (whose bits above `nb` are set already) with at least
// `need` of the C keys in cand (LDS) >= t, by bisection over the nb open bits; one wave.
// Keys are read into registers once (R per lane) when C <= 64 * R.
template <int R>
__device__ __forceinline__ uint32_t bisect_regs(const uint32_t* cand, int C, int nb,
                                                uint32_t tau, int need) {
  const int lane = threadIdx.x & 63;
  uint32_t c[R];
#pragma unroll
  for (int r = 0; r < R; ++r) c[r] = r * 64 + lane < C ? cand[r * 64 + lane] : 0u;
  for (int b = nb - 1; b >= 0; --b) {
    const uint32_t t = tau | (1u << b);   // >= 1: the 0 padding never counts
    int cnt = 0;
#pragma unroll
    for (int r = 0; r < R; ++r) cnt += __popcll(__ballot(c[r] >= t));
    if (cnt >= need) tau = t;
  }
  return tau;
}
__device__ __forceinline__ uint32_t bisect_lds(const uint32_t* cand, int C, int nb,
                                               uint32_t tau, int need) {
  const int lane = threadIdx.x & 63;
  if (C <= 64) return bisect_regs<1>(cand, C, nb, tau, need);
  if (C <= 128) return bisect_regs<2>(cand, C, nb, tau, need);
  if (C <= 256) return bisect_regs<4>(cand, C, nb, tau, need);
  for (int b = nb - 1; b >= 0; --b) {
    const uint32_t t = tau | (1u << b);
    int cnt = 0;
    for (int i0 = 0; i0 < C; i0 += 64) {
      const int i = i0 + lane;
      cnt += __popcll(__ballot(i < C && cand[i] >= t));
    }
    if (cnt >= need) tau = t;
  }
  return tau;
}

// The key of rank `need` (>= 1, counted from the smallest) among key_of(i), i < n (read from
// LDS), all of them in [base, base + span]: radix select on d = key - base, 8-bit digits
// from the highest one that span needs (so the first pass spreads the keys over its bins).
// Returns the key; *left gets how many keys equal to it are still needed.  nthreads
// threads; hist is 256 words; ctl 2 words.
template <typename KeyOf>
__device__ __forceinline__ uint32_t radix_rank_asc(KeyOf key_of, int n, uint32_t need,
                                                   uint32_t base, uint32_t span, uint32_t* hist,
                                                   uint32_t* ctl, int nthreads, uint32_t* left) {
  const int tid = threadIdx.x;
  const int bits = span == 0u ? 1 : 32 - __builtin_clz(span);
  uint32_t prefix = 0;
#pragma unroll 1
  for (int sh = (bits - 1) / 8 * 8; sh >= 0; sh -= 8) {
    for (int b = tid; b < 256; b += nthreads) hist[b] = 0;
    __syncthreads();
    for (int i = tid; i < n; i += nthreads) {
      const uint32_t dh = (key_of(i) - base) >> sh;   // this digit and the ones above it
      if ((dh >> 8) == prefix) atomicAdd(&hist[dh & 255u], 1u);
    }
    __syncthreads();
    if (tid < 64) {   // wave 0: 4 bins per lane, scanned from the smallest
      uint32_t c[4], tot = 0;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        c[u] = hist[tid * 4 + u];
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
            ctl[0] = tid * 4 + u;
            ctl[1] = before;
          }
          before += c[u];
        }
      }
    }
    __syncthreads();
    // the next pass clears hist and writes ctl only after its first two barriers, which
    // every thread reaches after these reads
    prefix = (prefix << 8) | ctl[0];
    need -= ctl[1];
  }
  *left = need;
  return base + prefix;
}

}  // namespace

__global__ __launch_bounds__(kConfThreads) void token_conf_partial_kernel(
    const float* __restrict__ logits, int64_t vocab, int64_t row_stride, int k, int splits,
    float2* __restrict__ ms_out, float* __restrict__ top_out) {
  __shared__ uint32_t cand[kConfCandCap];
  __shared__ float wred[kConfWaves];
  __shared__ uint32_t wkey[kConfWaves];
  __shared__ int wcnt[2][kConfWaves];
  __shared__ uint32_t ctl[2];   // candidates found; entries above the k-th largest emitted
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, split = blockIdx.x;
  const int64_t row = blockIdx.y;
  const int64_t c0 = (int64_t)split * kConfChunk;
  const int n = (int)(vocab - c0 < kConfChunk ? vocab - c0 : kConfChunk);
  const int kk = k < n ? k : n;   // >= 1: every chunk holds a logit and k >= 1
  const int64_t slot = row * splits + split;
  float* top = top_out + slot * k;
  const float ninf = -__builtin_inff();
  if (tid == 0) {
    ctl[0] = 0;
    ctl[1] = 0;
  }
  for (int j = kk + tid; j < k; j += kConfThreads) top[j] = ninf;   // padding
  // logit tid + j * 256 of the chunk in v[j]; the hardware returns 0 past the chunk
  const __amdgpu_buffer_rsrc_t rs =
      buffer_over(logits + row * row_stride + c0, n * (int)sizeof(float));
  float v[kConfPerThread];
#pragma unroll
  for (int j = 0; j < kConfPerThread; ++j)
    v[j] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                         rs, (tid + j * kConfThreads) * 4, 0, 0));
  // past a short chunk: -inf, which changes neither the max nor the sum, and among the k
  // largest stands only where -inf belongs anyway (kk <= n real logits)
  if (n < kConfChunk) {
#pragma unroll
    for (int j = 0; j < kConfPerThread; ++j)
      if (tid + j * kConfThreads >= n) v[j] = ninf;
  }
  // the chunk's max, then sum exp(x - max): each thread in j order, then a fixed tree
  float m = ninf;
#pragma unroll
  for (int j = 0; j < kConfPerThread; ++j) m = fmaxf(m, v[j]);
  m = wave_max_f(m);
  if (lane == 0) wred[wv] = m;
  __syncthreads();
  float M = wred[0];
#pragma unroll
  for (int w = 1; w < kConfWaves; ++w) M = fmaxf(M, wred[w]);
  // exp(x - M) as 2^((x - M) log2 e) on the hardware exp2 (error about 1 ulp; x = M gives
  // exactly 1); -inf adds 0
  float s = 0.0f;
  if (M != ninf) {
    constexpr float kLog2e = 1.4426950408889634f;
#pragma unroll
    for (int j = 0; j < kConfPerThread; ++j) s += fast_exp2((v[j] - M) * kLog2e);
  }
  s = wave_sum_f(s);
  // order keys (all >= 1) and the lanes' maxima
  uint32_t u[kConfPerThread];
  uint32_t lm = 0;
#pragma unroll
  for (int j = 0; j < kConfPerThread; ++j) {
    u[j] = order_key_raw(v[j]);
    lm = max(lm, u[j]);
  }
  // a lower bound of the kk-th largest key: in the wave that gives it, kk lanes hold a key
  // at least that large
  const uint32_t tw = wave_kth_key(lm, kk);
  __syncthreads();   // every thread has read the maxima
  if (lane == 0) {
    wred[wv] = s;
    wkey[wv] = tw;
  }
  __syncthreads();
  if (tid == 0) {
    float S = wred[0];
    for (int w = 1; w < kConfWaves; ++w) S += wred[w];
    ms_out[slot] = make_float2(M, S);
  }
  uint32_t lo = 1;
#pragma unroll
  for (int w = 0; w < kConfWaves; ++w) lo = max(lo, wkey[w]);
  // the keys >= lo into LDS (at least kk of them)
#pragma unroll
  for (int j = 0; j < kConfPerThread; ++j) {
    const bool p = u[j] >= lo;
    const uint64_t b = __ballot(p);
    if (b != 0ull) {
      uint32_t base = 0;
      if (lane == 0) base = atomicAdd(&ctl[0], (uint32_t)__popcll(b));
      base = (uint32_t)__shfl((int)base, 0, 64);
      const uint32_t pos = base + lanes_below(b);
      if (p && pos < (uint32_t)kConfCandCap) cand[pos] = u[j];
    }
  }
  __syncthreads();
  const int C = (int)ctl[0];
  const uint32_t hi = order_key_f(M);   // >= every key of the chunk (-0 and +0 included)
  // tau = the largest key t with at least kk keys >= t.  Counting the candidates only gives
  // the same answer for every t tested: above lo they are all the keys, at or below it there
  // are C >= kk of them.
  uint32_t tau;
  int nb = open_bits(lo, hi, &tau);
  if (C <= kConfCandCap) {
    if (wv != 0) return;
    tau = bisect_lds(cand, C, nb, tau, kk);
    // the keys above tau (fewer than kk), then kk minus that many copies of tau
    int g = 0;
    for (int i0 = 0; i0 < C; i0 += 64) {
      const int i = i0 + lane;
      const uint32_t key = i < C ? cand[i] : 0u;
      const bool above = key > tau;
      const uint64_t b = __ballot(above);
      if (above) top[g + (int)lanes_below(b)] = key_value_f(key);
      g += __popcll(b);
    }
    for (int j = g + lane; j < kk; j += 64) top[j] = key_value_f(tau);
    return;
  }
  // too many keys at the bound (a flat or heavily tied chunk): bisect over all of them
  for (int b = nb - 1; b >= 0; --b) {
    const uint32_t t = tau | (1u << b);
    int c = 0;
#pragma unroll
    for (int j = 0; j < kConfPerThread; ++j) c += u[j] >= t ? 1 : 0;
    c = wave_sum_i(c);
    if (lane == 0) wcnt[b & 1][wv] = c;
    __syncthreads();
    int tot = 0;
#pragma unroll
    for (int w = 0; w < kConfWaves; ++w) tot += wcnt[b & 1][w];
    if (tot >= kk) tau = t;
  }
#pragma unroll
  for (int j = 0; j < kConfPerThread; ++j) {
    const bool above = u[j] > tau;
    const uint64_t b = __ballot(above);
    if (b != 0ull) {
      uint32_t base = 0;
      if (lane == 0) base = atomicAdd(&ctl[1], (uint32_t)__popcll(b));
      base = (uint32_t)__shfl((int)base, 0, 64);
      if (above) top[base + lanes_below(b)] = key_value_f(u[j]);
    }
  }
  __syncthreads();
  for (int j = (int)ctl[1] + tid; j < kk; j += kConfThreads) top[j] = key_value_f(tau);
}

__global__ __launch_bounds__(64) void token_conf_merge_kernel(
    const float2* __restrict__ ms, const float* __restrict__ top_in, int k, int splits,
    int64_t vocab, float* __restrict__ conf) {
  __shared__ uint32_t cand[kConfMaxCand];
  __shared__ float best[64];
  const int lane = threadIdx.x;
  const int64_t row = blockIdx.x;
  const int nc = splits * k;   // <= kConfMaxCand
  const float* in = top_in + row * nc;
  const float ninf = -__builtin_inff();
  // the k largest logits of the row are the kk = min(k, vocab) largest candidates: every
  // chunk contributed its own min(k, chunk) largest, padded with -inf
  const int kk = (int64_t)k < vocab ? k : (int)vocab;
  const float2 msl = lane < splits ? ms[row * splits + lane] : make_float2(ninf, 0.0f);
  uint32_t u[kMergePerLane];
  uint32_t lm = 0;
#pragma unroll
  for (int s = 0; s < kMergePerLane; ++s) {
    const int i = s * 64 + lane;
    u[s] = i < nc ? order_key_f(in[i]) : 0u;
    lm = max(lm, u[s]);
  }
  const uint32_t hi = wave_max_u(lm);
  const uint32_t lo = max(wave_kth_key(lm, kk), 1u);
  int C = 0;
#pragma unroll
  for (int s = 0; s < kMergePerLane; ++s) {
    const bool p = u[s] >= lo;
    const uint64_t b = __ballot(p);
    if (p) cand[C + (int)lanes_below(b)] = u[s];
    C += __popcll(b);
  }
  __syncthreads();
  uint32_t tau;
  const int nb = open_bits(lo, hi, &tau);
  tau = bisect_lds(cand, C, nb, tau, kk);
  int g = 0;
  for (int i0 = 0; i0 < C; i0 += 64) {
    const int i = i0 + lane;
    const uint32_t key = i < C ? cand[i] : 0u;
    const bool above = key > tau;
    const uint64_t b = __ballot(above);
    if (above) best[g + (int)lanes_below(b)] = key_value_f(key);
    g += __popcll(b);
  }
  __syncthreads();
  // one of the kk largest per lane, then a bitonic sort across the lanes, descending
  float x = lane < g ? best[lane] : (lane < kk ? key_value_f(tau) : ninf);
#pragma unroll
  for (int size = 2; size <= 64; size <<= 1) {
#pragma unroll
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      const float o = __shfl_xor(x, stride, 64);
      const bool keep_max = ((lane & stride) == 0) == ((lane & size) == 0);
      x = keep_max ? fmaxf(x, o) : fminf(x, o);
    }
  }
  // the row's log-sum-exp: lane c holds chunk c's (max, sum); terms rescaled to the row max
  // and added in chunk order
  const float M = wave_max_f(msl.x);
  const float term = M == ninf || msl.x == ninf ? 0.0f : msl.y * expf(msl.x - M);
  float S = 0.0f;
  for (int c = 0; c < splits; ++c)
    S += __int_as_float(__builtin_amdgcn_readlane(__float_as_int(term), c));
  double sum = 0.0;
  for (int j = 0; j < kk; ++j)
    sum += (double)__int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), j));
  if (lane == 0) {
    const double lse = (double)M + log((double)S);
    conf[row] = (float)(lse - sum / (double)kk);
  }
}

// ---- Alg. 2 steps 2-4 -------------------------------------------------------------------
constexpr int kBudgetTokBatch = 32;   // trace tokens in flight per thread

// bkey[j] = the smallest order key of t[j g .. (j + 1) g), j < ntok / g, from one coalesced
// pass over t[0 .. ntok).  kLg >= 0: g = 2^kLg <= 64, a block sits in g consecutive lanes
// of one batch (its first token at a multiple of g), reduced across them and stored by the
// first; kLg < 0: any g, LDS atomics (bkey set to all ones beforehand).
template <int kLg>
__device__ __forceinline__ void block_minima(const float* __restrict__ t, int ntok, int g,
                                             uint32_t* bkey) {
  const int tid = threadIdx.x;
  for (int e0 = 0; e0 < ntok; e0 += kBudgetThreads * kBudgetTokBatch) {
    float v[kBudgetTokBatch];
#pragma unroll
    for (int u = 0; u < kBudgetTokBatch; ++u) {
      const int e = e0 + u * kBudgetThreads + tid;
      v[u] = e < ntok ? t[e] : 0.0f;
    }
#pragma unroll
    for (int u = 0; u < kBudgetTokBatch; ++u) {
      const int e = e0 + u * kBudgetThreads + tid;
      uint32_t kv = e < ntok ? order_key_f(v[u]) : 0xFFFFFFFFu;
      if constexpr (kLg >= 0) {
        kv = group_min_to_leader<kLg>(kv);
        if (e < ntok && (e & ((1 << kLg) - 1)) == 0) bkey[e >> kLg] = kv;
      } else {
        if (e < ntok) atomicMin(&bkey[e / g], kv);
      }
    }
  }
}

__global__ __launch_bounds__(kBudgetThreads) void budget_kernel(
    const float* __restrict__ tconf, const int64_t* __restrict__ offsets, int window,
    int stride, float bottom_pct, float scale_up, int budget_upper,
    const int32_t* __restrict__ budgets_in, int32_t* __restrict__ budgets_out,
    double* __restrict__ slopes, double* __restrict__ thresholds, int32_t* __restrict__ retained) {
#pragma clang fp contract(off)
  __shared__ float rp[kMaxBudgetWindows];       // R'_m, then the retained values in order
  __shared__ int32_t rm[kMaxBudgetWindows];     // block minima (as keys), then window indices
  __shared__ double2 pq[kBudgetThreads];        // products of the slope's sums, one batch
  __shared__ uint32_t hist[256];
  __shared__ uint32_t ctl[4];
  __shared__ int64_t scan_tmp[17];
  __shared__ uint32_t mm_tmp[2][kBudgetThreads / 64];
  __shared__ double mean_tmp[2];
  const int r = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int64_t n = offsets[r + 1] - offsets[r];
  const float* t = tconf + offsets[r];
  double alpha = 0.0, q = __builtin_nan("");
  int kept = 0;
  if (n >= window) {
    const int M = (int)((n - window) / stride + 1);
    // windows are whole blocks of g = gcd(w, s) tokens: the minima of the blocks the windows
    // cover, from one coalesced pass over those tokens, then each window's minimum over its
    // w / g blocks in LDS.  Minima are taken on order keys (-0 and +0 alike).
    int g = window, b = stride;
    while (b != 0) {
      const int r0 = g % b;
      g = b;
      b = r0;
    }
    const int64_t nbl = ((int64_t)(M - 1) * stride + window) / g;
    if (nbl <= kMaxBudgetWindows && nbl * g < (int64_t)1 << 30) {
      uint32_t* bkey = reinterpret_cast<uint32_t*>(rm);
      const int ntok = (int)nbl * g;   // <= n
      switch ((g & (g - 1)) == 0 && g <= 64 ? __builtin_ctz(g) : -1) {
        case 0: block_minima<0>(t, ntok, g, bkey); break;
        case 1: block_minima<1>(t, ntok, g, bkey); break;
        case 2: block_minima<2>(t, ntok, g, bkey); break;
        case 3: block_minima<3>(t, ntok, g, bkey); break;
        case 4: block_minima<4>(t, ntok, g, bkey); break;
        case 5: block_minima<5>(t, ntok, g, bkey); break;
        case 6: block_minima<6>(t, ntok, g, bkey); break;
        default:
          for (int j = tid; j < (int)nbl; j += kBudgetThreads) bkey[j] = 0xFFFFFFFFu;
          __syncthreads();
          block_minima<-1>(t, ntok, g, bkey);
      }
      __syncthreads();
      const int wb = window / g, sb = stride / g;
      for (int m = tid; m < M; m += kBudgetThreads) {
        uint32_t kv = bkey[m * sb];
        for (int i = 1; i < wb; ++i) kv = min(kv, bkey[m * sb + i]);
        rp[m] = key_value_f(kv);
      }
    } else {
      for (int m = tid; m < M; m += kBudgetThreads) {
        float v = t[(int64_t)m * stride];
        for (int i = 1; i < window; ++i) v = fminf(v, t[(int64_t)m * stride + i]);
        rp[m] = v;
      }
    }
    __syncthreads();
    // the range of the window keys, for the radix select
    uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
    for (int m = tid; m < M; m += kBudgetThreads) {
      const uint32_t km = order_key_f(rp[m]);
      kmin = min(kmin, km);
      kmax = max(kmax, km);
    }
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) {
      kmin = min(kmin, (uint32_t)__shfl_xor((int)kmin, d, 64));
      kmax = max(kmax, (uint32_t)__shfl_xor((int)kmax, d, 64));
    }
    if (lane == 0) {
      mm_tmp[0][wv] = kmin;
      mm_tmp[1][wv] = kmax;
    }
    __syncthreads();
    for (int w = 0; w < kBudgetThreads / 64; ++w) {
      kmin = min(kmin, mm_tmp[0][w]);
      kmax = max(kmax, mm_tmp[1][w]);
    }
    __syncthreads();   // mm_tmp is written again below
    // percentile: order statistics lo and lo + 1 (ascending), linear interpolation
    const double pos = ((double)bottom_pct / 100.0) * (double)(M - 1);
    const int lo = (int)floor(pos);
    const double frac = pos - (double)lo;
    uint32_t left;
    auto key_of = [&](int i) { return order_key_f(rp[i]); };
    const uint32_t klo = radix_rank_asc(key_of, M, (uint32_t)lo + 1u, kmin, kmax - kmin, hist,
                                        ctl, kBudgetThreads, &left);
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
      if (lane == 0) mm_tmp[0][wv] = next;
      __syncthreads();
      for (int w = 0; w < kBudgetThreads / 64; ++w) next = min(next, mm_tmp[0][w]);
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
    int64_t msum = 0;
#pragma unroll
    for (int u = 0; u < kMaxPer; ++u) {
      yv[u] = m0 + u < m1 ? rp[m0 + u] : 0.0f;
      const bool keep = m0 + u < m1 && (double)yv[u] <= q;
      cnt += keep ? 1u : 0u;
      msum += keep ? m0 + u : 0;
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
    int64_t sxi;
    block_excl_scan_i64(msum, scan_tmp, &sxi);   // its first barrier orders the writes too
    kept = (int)total;
    if (kept >= 2) {
      // least squares in window order, every operation rounded on its own.  Sum of m: an
      // integer below 2^53 at every step, so the exact integer sum is the fp64 sum in any
      // order.  Sum of R': one thread, in order.  The products of the second pass do not
      // depend on the order, so the block forms them, 1024 at a time, and one thread adds
      // them up in order.
      if (tid == 0) {
        constexpr int kB = 16;
        double sy = 0.0;
        int i0 = 0;
        for (; i0 + kB <= kept; i0 += kB) {
          float y[kB];
#pragma unroll
          for (int u = 0; u < kB; ++u) y[u] = rp[i0 + u];
#pragma unroll
          for (int u = 0; u < kB; ++u) sy = sy + (double)y[u];
        }
        for (; i0 < kept; ++i0) sy = sy + (double)rp[i0];
        mean_tmp[0] = (double)sxi / (double)kept;
        mean_tmp[1] = sy / (double)kept;
      }
      __syncthreads();
      const double mx = mean_tmp[0], my = mean_tmp[1];
      double num = 0.0, den = 0.0;
      for (int b0 = 0; b0 < kept; b0 += kBudgetThreads) {
        const int i = b0 + tid;
        if (i < kept) {
          const double dx = (double)rm[i] - mx, dy = (double)rp[i] - my;
          pq[tid] = make_double2(dx * dy, dx * dx);
        }
        __syncthreads();
        if (tid == 0) {
          const int cb = kept - b0 < kBudgetThreads ? kept - b0 : kBudgetThreads;
          constexpr int kB = 8;
          int j0 = 0;
          for (; j0 + kB <= cb; j0 += kB) {
            double2 a[kB];
#pragma unroll
            for (int u = 0; u < kB; ++u) a[u] = pq[j0 + u];
#pragma unroll
            for (int u = 0; u < kB; ++u) {
              num = num + a[u].x;
              den = den + a[u].y;
            }
          }
          for (; j0 < cb; ++j0) {
            num = num + pq[j0].x;
            den = den + pq[j0].y;
          }
        }
        __syncthreads();
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
  hipLaunchKernelGGL(token_conf_merge_kernel, dim3((unsigned)rows), dim3(64), 0, s, ms,
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
