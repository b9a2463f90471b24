// Eviction: per (request, KV head) keep the k = min(budget, L) entries with the largest
// max-pooled score, ties to the lower token index (Alg. 1 step 5, TopK), emitted in
// ascending token order; and the attention-aware LRFU variant (Sec. 5.1) that ranks by
// keep scores carried over from step to step instead.
//
// One 1024-thread workgroup per (request, KV head).  Every decision below is made on an
// unsigned key derived from the fp32 bit pattern that orders exactly like the float, so the
// result is exact and deterministic.
//   stage   the raw scores of the segment are loaded into LDS (coalesced raw buffer loads)
//   pool    max-pooled in place over the window, clipped at the ends, and copied out
//   radix   digit passes of up to 11 bits over the segment's key range (LDS histogram, most
//           significant digit first) find the key tau of the k-th largest entry and how
//           many entries equal to tau to take
//   emit    each thread owns a contiguous run of the segment; one workgroup prefix sum of
//           its (greater, equal) counts gives its output offset, so the kept indices come
//           out in ascending order
// From the pool to the emit LDS holds the order keys of the segment and every pass re-reads
// its run from there.  The passes are bound by vector ALU issue (one workgroup per segment
// leaves four waves per SIMD), so each visit of an entry is kept to a few instructions:
// keys instead of floats (no conversion per pass), batched LDS reads at immediate offsets
// (the LDS buffer is padded so a batch may read past the end of the segment), 32-bit digit
// arithmetic.
// Segments longer than the LDS capacity, up to 64,512 entries, hold their keys in registers
// instead (windows up to 7); longer ones, or wider windows, run the same steps on `pooled` in
// global memory.
#include "device_common.hpp"

namespace actkv {

namespace {

constexpr int kSelectThreads = 1024;
constexpr int kSelectLdsKeys = 38400;     // segment length kept in LDS (153,600 bytes)
static_assert(kSelectLdsKeys == kLrfuLdsLen, "LRFU segments up to this length stay in LDS");
constexpr int kMaxBins = 2048;            // largest digit: 11 bits
constexpr int kDigits = 3;                // bits 31..21, 20..10, 9..0
constexpr int kRows = (kSelectLdsKeys + kSelectThreads - 1) / kSelectThreads;   // 38
constexpr int kRowBatch = kRows / 2;      // rows of a coalesced pass in flight together
static_assert(kRows % 2 == 0, "the coalesced passes run in two batches of rows");
constexpr int kRunBatch = 8;              // run entries whose LDS reads are issued together
constexpr int kLdsPad = 16;               // LDS entries past the segment a batch may read
constexpr int kPoolHalo = 3;              // pooling windows up to 7 run in place
// Unsigned key that orders exactly like the float (negative values included; -0 == +0).
__device__ __forceinline__ uint32_t order_key(float v) {
  const uint32_t u = __float_as_uint(v == 0.0f ? 0.0f : v);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// The float whose order_key is k.
__device__ __forceinline__ float key_value(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

// -0 as +0 (the pooled score of an entry is the value its order key stands for).
__device__ __forceinline__ float canonical(float v) { return v == 0.0f ? 0.0f : v; }

// Byte offset of this lane in a coalesced pass, opaque to the compiler so that the offsets
// of two passes are not shared (and kept live) between them.
__device__ __forceinline__ int lane_byte_offset() {
  int off = (int)threadIdx.x * (int)sizeof(float);
  asm volatile("" : "+v"(off));
  return off;
}

// Among bins [0, nbins) (higher bin = larger key), find the bin b holding the need-th
// largest element: sum_{b' > b} hist[b'] < need <= sum_{b' >= b} hist[b'].  Thread t of NT
// covers max(1, nbins / NT) bins counted down from the top (nbins a power of two).  Returns b
// and the count strictly above it through LDS.
template <int NT = kSelectThreads>
__device__ __forceinline__ void find_bin(const uint32_t* hist, int nbins, uint32_t need,
                                         int64_t* scan_tmp, int* bin_out, uint32_t* above_out) {
  // nbins / NT bins per thread (at least 1); threads past the bins of a small histogram
  // hold none
  const int t = threadIdx.x, per = nbins > NT ? nbins / NT : 1;
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

// find_bin on 64-bit masses: the bin b where the mass strictly above it is below `need`
// and the mass from b up reaches it (nbins <= kSelectThreads: one bin per thread).
__device__ __forceinline__ void find_bin64(const uint64_t* hist, int nbins, uint64_t need,
                                           int64_t* scan_tmp, int* bin_out,
                                           uint64_t* above_out) {
  const int t = threadIdx.x, top = nbins - 1 - t;
  const uint64_t s = top >= 0 ? hist[top] : 0ull;
  int64_t total;
  const uint64_t ex = (uint64_t)block_excl_scan_i64((int64_t)s, scan_tmp, &total);
  if (top >= 0 && ex < need && need <= ex + s) {
    *bin_out = top;
    *above_out = ex;
  }
  __syncthreads();
}

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

// ---- building blocks of the LDS-resident selections ---------------------------------
// Thread tid owns the contiguous run [t0, t0 + n) of the segment, t0 = tid * per with per
// odd (the lanes' LDS accesses fall on distinct banks).
struct RunGeom {
  int t0, n;
};

__device__ __forceinline__ RunGeom run_geom(int L) {
  const int per = ((L + kSelectThreads - 1) / kSelectThreads) | 1;
  const int t0 = (int)threadIdx.x * per < L ? (int)threadIdx.x * per : L;
  const int t1 = t0 + per < L ? t0 + per : L;
  return RunGeom{t0, t1 - t0};
}

// Visit this thread's run in batches: every LDS read of a batch is issued before any of its
// values is used (one LDS round trip per batch).  f(i, key) receives the run position and
// the key.  The last batch may read up to kRunBatch - 1 entries past the run (inside the
// segment or its padding) and ignores them.
template <typename F>
__device__ __forceinline__ void visit_run(RunGeom g, const uint32_t* keys, F f) {
  const uint32_t* run = keys + g.t0;
  int c = 0;
#pragma unroll 1
  for (; c + kRunBatch <= g.n; c += kRunBatch) {
    uint32_t v[kRunBatch];
#pragma unroll
    for (int j = 0; j < kRunBatch; ++j) v[j] = run[c + j];
#pragma unroll
    for (int j = 0; j < kRunBatch; ++j) f(c + j, v[j]);
  }
  if (c < g.n) {
    uint32_t v[kRunBatch];
#pragma unroll
    for (int j = 0; j < kRunBatch; ++j) v[j] = run[c + j];
#pragma unroll
    for (int j = 0; j < kRunBatch; ++j)
      if (c + j < g.n) f(c + j, v[j]);
  }
}

// Coalesced load of a segment of fp32 into LDS: raw buffer loads over exactly L floats (the
// hardware returns 0 past the end), a batch of rows in flight at once.
__device__ __forceinline__ void stage_f32(int L, const float* __restrict__ in, uint32_t* vals) {
  const __amdgpu_buffer_rsrc_t rsrc = buffer_over(in, L * (int)sizeof(float));
  const int off = lane_byte_offset();
  const int rows = (L + kSelectThreads - 1) / kSelectThreads;
#pragma unroll 1
  for (int r0 = 0; r0 < rows; r0 += kRowBatch) {
    uint32_t v[kRowBatch];
#pragma unroll
    for (int j = 0; j < kRowBatch; ++j)
      v[j] = __builtin_amdgcn_raw_buffer_load_b32(rsrc, off + (r0 + j) * kSelectThreads * 4, 0,
                                                  0);
#pragma unroll
    for (int j = 0; j < kRowBatch; ++j) {
      const int t = threadIdx.x + (r0 + j) * kSelectThreads;
      if (t < L) vals[t] = v[j];
    }
  }
}

// dst[t] = xf(src[t]) for t < n, from LDS to global memory, coalesced, through raw buffer
// stores over exactly n words (the hardware drops stores at or past the end).
// n <= kSelectLdsKeys.
template <typename Xf>
__device__ __forceinline__ void copy_out_u32(int n, const uint32_t* src, void* dst, Xf xf) {
  const __amdgpu_buffer_rsrc_t rsrc = buffer_over(dst, n * (int)sizeof(uint32_t));
  const int off = lane_byte_offset(), last = n > 0 ? n - 1 : 0;
  const int rows = (n + kSelectThreads - 1) / kSelectThreads;
#pragma unroll 1
  for (int r0 = 0; r0 < rows; r0 += kRowBatch) {
    uint32_t v[kRowBatch];
#pragma unroll
    for (int j = 0; j < kRowBatch; ++j) {
      const int t = threadIdx.x + (r0 + j) * kSelectThreads;
      v[j] = src[t < last ? t : last];
    }
#pragma unroll
    for (int j = 0; j < kRowBatch; ++j)
      if (r0 + j < rows)   // uniform
        __builtin_amdgcn_raw_buffer_store_b32(xf(v[j]), rsrc,
                                              off + (r0 + j) * kSelectThreads * 4, 0, 0);
  }
}

struct AsIs {
  __device__ uint32_t operator()(uint32_t x) const { return x; }
};
struct KeyToFloatBits {   // the float an order key stands for
  __device__ uint32_t operator()(uint32_t k) const {
    return (k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k;
  }
};

// dst[j] = src[idx[j]] for j < n: indices from LDS, values gathered from global memory,
// written out coalesced.  Every idx[j] < the length of src.
__device__ __forceinline__ void gather_out_f32(int n, const int32_t* idx, const float* src,
                                               float* dst) {
  const __amdgpu_buffer_rsrc_t rsrc = buffer_over(dst, n * (int)sizeof(float));
  const int off = lane_byte_offset(), last = n > 0 ? n - 1 : 0;
  const int rows = (n + kSelectThreads - 1) / kSelectThreads;
#pragma unroll 1
  for (int r0 = 0; r0 < rows; r0 += kRowBatch) {
    float v[kRowBatch];
#pragma unroll
    for (int j = 0; j < kRowBatch; ++j) {
      const int t = threadIdx.x + (r0 + j) * kSelectThreads;
      v[j] = r0 + j < rows ? src[idx[t < last ? t : last]] : 0.0f;
    }
#pragma unroll
    for (int j = 0; j < kRowBatch; ++j)
      if (r0 + j < rows)   // uniform
        __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v[j]), rsrc,
                                              off + (r0 + j) * kSelectThreads * 4, 0, 0);
  }
}

// Max-pool in place for windows up to 2 * kPoolHalo + 1: each thread first reads the raw
// scores just outside its run (the halo), then, once every thread has done so, slides a
// window of registers along its own run, overwriting each entry with the order key of its
// pooled score (the raw scores ahead of the window are still in LDS, those behind it in
// registers).
__device__ __forceinline__ void pool_narrow_in_place(int L, int hw, RunGeom g, uint32_t* vals) {
  const float ninf = -__builtin_inff();
  const int t1 = g.t0 + g.n;
  auto raw = [&](int p) { return __uint_as_float(vals[p]); };
  float halo_l[kPoolHalo], halo_r[kPoolHalo];
#pragma unroll
  for (int j = 0; j < kPoolHalo; ++j) {
    const int pl = g.t0 - kPoolHalo + j, pr = t1 + j;   // pr <= L + 2: inside the padding
    const float vl = raw(pl < 0 ? 0 : pl), vr = raw(pr);
    halo_l[j] = (pl >= 0 && g.n > 0) ? vl : ninf;
    halo_r[j] = (pr < L && g.n > 0) ? vr : ninf;
  }
  __syncthreads();   // no thread overwrites an entry before its neighbours read their halo
  // raw score at p >= t0 that the window has not reached yet
  auto ahead = [&](float lds_value, int p) {
    const int d = p - t1;
    return d < 0 ? lds_value
                 : (d == 0 ? halo_r[0] : (d == 1 ? halo_r[1] : (d == 2 ? halo_r[2] : ninf)));
  };
  // win[x] = raw score at t - kPoolHalo + x for the entry t produced next; every LDS read
  // below is at most t1 + 2 * kPoolHalo + kRunBatch - 3 < L + kLdsPad
  float win[2 * kPoolHalo + 1];
#pragma unroll
  for (int x = 0; x < kPoolHalo; ++x) win[x] = halo_l[x];
#pragma unroll
  for (int x = 0; x <= kPoolHalo; ++x) win[kPoolHalo + x] = ahead(raw(g.t0 + x), g.t0 + x);
#pragma unroll 1
  for (int c = 0; c < g.n; c += kRunBatch) {
    float nxt[kRunBatch];   // raw scores at t0 + c + kPoolHalo + 1 + j
#pragma unroll
    for (int j = 0; j < kRunBatch; ++j) nxt[j] = raw(g.t0 + c + kPoolHalo + 1 + j);
#pragma unroll
    for (int j = 0; j < kRunBatch; ++j) nxt[j] = ahead(nxt[j], g.t0 + c + kPoolHalo + 1 + j);
#pragma unroll
    for (int j = 0; j < kRunBatch; ++j) {
      float m = win[kPoolHalo];
#pragma unroll
      for (int d = 1; d <= kPoolHalo; ++d)
        if (d <= hw) m = fmaxf(m, fmaxf(win[kPoolHalo - d], win[kPoolHalo + d]));
      if (c + j < g.n) vals[g.t0 + c + j] = order_key(m);
#pragma unroll
      for (int x = 0; x < 2 * kPoolHalo; ++x) win[x] = win[x + 1];
      win[2 * kPoolHalo] = nxt[j];
    }
  }
}

// Wider windows: every thread pools its run into registers from the raw scores, then all
// write back once every read is done (a straight loop per entry; uncommon).
__device__ __forceinline__ void pool_wide_in_place(int L, int hw, RunGeom g, uint32_t* vals) {
  constexpr int kRun = kRows + 1;   // longest run: odd >= ceil(kSelectLdsKeys / threads)
  float m[kRun];
#pragma unroll
  for (int i = 0; i < kRun; ++i) {
    const int t = g.t0 + i;
    float x = -__builtin_inff();
    if (i < g.n) {
      const int lo = t - hw < 0 ? 0 : t - hw, hi = t + hw >= L ? L - 1 : t + hw;
      for (int y = lo; y <= hi; ++y) x = fmaxf(x, __uint_as_float(vals[y]));
    }
    m[i] = x;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < kRun; ++i)
    if (i < g.n) vals[g.t0 + i] = order_key(m[i]);
}

// Pool the staged raw scores in place (LDS then holds their order keys); the pooled scores
// are also copied to `out` when given.
__device__ __forceinline__ void pool_in_lds(int L, int hw, RunGeom g, uint32_t* vals,
                                            float* out) {
  if (hw <= kPoolHalo)
    pool_narrow_in_place(L, hw, g, vals);
  else
    pool_wide_in_place(L, hw, g, vals);
  __syncthreads();
  if (out) copy_out_u32(L, vals, out, KeyToFloatBits());
}

// The steps below see the segment's keys through a visitor: visit(f) calls f(i, key) for
// every entry of this thread's run (i = position in the run), whether the keys sit in LDS
// (visit_run) or in registers (visit_regs).

// Smallest and largest key of the segment (every thread gets both).
template <typename Visit>
__device__ __forceinline__ void key_range_by(Visit visit, uint32_t* mm_tmp, uint32_t* lo,
                                             uint32_t* hi) {
  uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
  visit([&](int, uint32_t kk) {
    kmin = min(kmin, kk);
    kmax = max(kmax, kk);
  });
  block_min_max(kmin, kmax, mm_tmp, lo, hi);
}

// The same over the real keys only, for runs that carry padding keys (0, which no float's
// key is but one NaN pattern): with the padding in it the range would start at 0, and the
// first radix digit, the top bits of the keys, would put every score of a few exponents into
// a few bins, whose atomics then serialise (measured: 44 us for that pass over 64,000
// entries, against 4-5 us for the other passes).  At least one key is real.
template <typename Visit>
__device__ __forceinline__ void real_key_range_by(Visit visit, uint32_t* mm_tmp, uint32_t* lo,
                                                  uint32_t* hi) {
  uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
  visit([&](int, uint32_t kk) {
    kmin = min(kmin, kk == 0u ? 0xFFFFFFFFu : kk);
    kmax = max(kmax, kk);
  });
  block_min_max(kmin, kmax, mm_tmp, lo, hi);
}

// Radix select over the segment, keys in [lo, hi]: tau and `need` such that the kept entries
// are every key > tau and the first `need` keys equal to tau (0 < k < L): tau is the order
// key of the k-th largest, or, when a pass finds that its whole bin is kept, the key just
// below that bin (need 0).  Digits of up to 11 bits over d = key - lo, within the bit width
// of the key range, so concentrated values still spread over the whole first histogram.
template <bool kSkipBelowLo = false, typename Visit>
__device__ __forceinline__ void radix_tau_by(Visit visit, int k, uint32_t lo, uint32_t hi,
                                             uint32_t* hist, int64_t* scan_tmp, int* s_bin,
                                             uint32_t* s_above, uint32_t* tau_out,
                                             uint32_t* need_out) {
  const int tid = threadIdx.x;
  const uint32_t range = hi - lo;
  int rem = range == 0 ? 0 : 32 - __clz(range);
  uint32_t need = (uint32_t)k, prefix = 0;
#pragma unroll 1
  while (rem > 0) {
    const int bits = rem < 11 ? rem : 11, sh = rem - bits, nbins = 1 << bits;
    for (int bb = tid; bb < nbins; bb += kSelectThreads) hist[bb] = 0;
    __syncthreads();
    visit([&](int, uint32_t kk) {
      const uint32_t dh = (kk - lo) >> sh;   // this digit and the ones above it
      // keys whose higher digits match the prefix found so far (none above the range; with
      // kSkipBelowLo, padding keys below the range are left out)
      if ((!kSkipBelowLo || kk >= lo) && (dh >> bits) == prefix)
        atomicAdd(&hist[dh & (uint32_t)(nbins - 1)], 1u);
    });
    __syncthreads();
    find_bin(hist, nbins, need, scan_tmp, s_bin, s_above);
    need -= *s_above;
    prefix = (prefix << bits) | (uint32_t)*s_bin;
    rem = sh;
    // every key of the chosen bin is taken: the kept set is then every key from the bin's
    // lowest possible key up, whatever the digits below, and the passes end early.  (That
    // key is above lo: otherwise all L keys would be kept, and 0 < k < L here.)
    if (rem > 0 && hist[*s_bin] == need) {
      *tau_out = lo + (prefix << rem) - 1u;   // keys > tau: exactly those from the bin up
      *need_out = 0;
      return;
    }
  }
  *tau_out = lo + prefix;
  *need_out = need;
}

// Kept entries: every key > tau, then the first `need` keys == tau, in index order.  The
// run's greater / equal flags are kept as bit masks; one workgroup prefix sum of both counts
// places each thread's kept indices, which are staged in LDS (`idx`, kSelectLdsKeys entries
// at a time) and written out coalesced (not written when kout is null: k <= kSelectLdsKeys
// then leaves them all in idx).  When vout is given, vout[j] = vsrc[kept[j]] (vsrc in
// global memory).  Every read of the keys is done before idx is written: idx may overlay
// them.
template <typename Visit>
__device__ __forceinline__ void emit_kept_by(Visit visit, RunGeom g, uint32_t tau,
                                             uint32_t need, int k, int64_t* scan_tmp,
                                             int32_t* idx, int32_t* __restrict__ kout,
                                             const float* vsrc, float* __restrict__ vout) {
  uint64_t gtm = 0, eqm = 0;
  visit([&](int i, uint32_t kk) {
    gtm |= (uint64_t)(kk > tau) << i;
    eqm |= (uint64_t)(kk == tau) << i;
  });
  const int64_t n_gt = __popcll(gtm), n_eq = __popcll(eqm);
  // the tied entries are taken in thread order, so the threads before this one took
  // min(need, eq_before) of them (each count sum < 2^32).  The scan's barriers also retire
  // every thread's reads of the keys above.
  int64_t tot;
  const int64_t ex = block_excl_scan_i64((n_eq << 32) | n_gt, scan_tmp, &tot);
  const int64_t eq_before = ex >> 32, gt_before = ex & 0xFFFFFFFFll;
  int64_t eq_take = (int64_t)need - eq_before;
  eq_take = eq_take < 0 ? 0 : (eq_take > n_eq ? n_eq : eq_take);
  for (int64_t drop = n_eq - eq_take; drop > 0; --drop)   // keep the first eq_take ties
    eqm &= ~(1ull << (63 - __clzll(eqm)));
  const uint64_t keep = gtm | eqm;
  const int pos0 = (int)(gt_before + (eq_before < (int64_t)need ? eq_before : (int64_t)need));
#pragma unroll 1
  for (int b = 0; b < k; b += kSelectLdsKeys) {   // uniform: one chunk unless k > the LDS
    const int nc = k - b < kSelectLdsKeys ? k - b : kSelectLdsKeys;
    uint64_t m = keep;
    for (int pos = pos0; m; ++pos, m &= m - 1)
      if (pos >= b && pos < b + nc) idx[pos - b] = g.t0 + __builtin_ctzll(m);
    __syncthreads();
    if (kout) copy_out_u32(nc, reinterpret_cast<const uint32_t*>(idx), kout + b, AsIs());
    if (vout) gather_out_f32(nc, idx, vsrc, vout + b);
    __syncthreads();
  }
}

// TopK of the segment in LDS (0 <= k): indices to kout (when given; for 0 < k < L they are
// also left in LDS, over the keys) and, when vout is given, the kept values (vsrc holds the
// values the keys stand for, in global memory).
__device__ __forceinline__ void topk_lds(int L, int k, RunGeom g, uint32_t* keys, uint32_t* hist,
                                         int64_t* scan_tmp, uint32_t* mm_tmp, int* s_bin,
                                         uint32_t* s_above, int32_t* __restrict__ kout,
                                         const float* vsrc, float* __restrict__ vout) {
  if (k <= 0) return;
  if (k >= L) {
    if (kout)
      for (int t = threadIdx.x; t < L; t += kSelectThreads) kout[t] = t;
    if (vout) copy_out_u32(L, keys, vout, KeyToFloatBits());
    return;
  }
  uint32_t lo, hi, tau, need;
  auto visit = [&](auto f) { visit_run(g, keys, f); };
  key_range_by(visit, mm_tmp, &lo, &hi);
  radix_tau_by(visit, k, lo, hi, hist, scan_tmp, s_bin, s_above, &tau, &need);
  emit_kept_by(visit, g, tau, need, k, scan_tmp, reinterpret_cast<int32_t*>(keys), kout, vsrc,
               vout);
}

// Segments that fit in LDS: stage, pool, pooled scores out, radix select, emit.
__device__ __forceinline__ void select_lds(int L, int k, int hw, const float* __restrict__ in,
                                           float* pout, int32_t* __restrict__ kout, uint32_t* vals,
                                           uint32_t* hist, int64_t* scan_tmp, uint32_t* mm_tmp,
                                           int* s_bin, uint32_t* s_above) {
  stage_f32(L, in, vals);
  __syncthreads();
  const RunGeom g = run_geom(L);
  pool_in_lds(L, hw, g, vals, pout);
  topk_lds(L, k, g, vals, hist, scan_tmp, mm_tmp, s_bin, s_above, kout, nullptr, nullptr);
}

// ---- segments longer than the LDS capacity: keys in registers ---------------------------
// Thread tid owns the run [t0, t0 + n) as above (odd stride, at most kRegRun entries) and
// holds it in registers, with the pooling halo on either side.  LDS serves as the transpose
// buffer of the coalesced loads and stores, kSelectLdsKeys entries at a time, and stages the
// kept indices.  Windows up to 2 * kPoolHalo + 1.
constexpr int kRegRun = 63;                                  // odd: conflict-free LDS strides
constexpr int kSelectRegKeys = kRegRun * kSelectThreads;     // 64,512
constexpr int kRegSlots = kRegRun + 2 * kPoolHalo;
static_assert(kSelectRegKeys < 2 * kSelectLdsKeys, "a segment passes through LDS in two chunks");
static_assert(kSelectRegKeys == kLrfuMaxLen && 2 * kPoolHalo + 1 == kLrfuRegMaxWindow,
              "the LRFU selection's limits are those of the register-resident path");

// r[j] = the raw score at position t0 - kPoolHalo + j where that position lies in
// [t0 - kPoolHalo, t0 + n + kPoolHalo) and in [0, L); -inf elsewhere.
__device__ __forceinline__ void stage_regs(int L, const float* __restrict__ in, RunGeom g,
                                           uint32_t* vals, uint32_t (&r)[kRegSlots]) {
  const int q0 = g.t0 - kPoolHalo;                 // position of r[0]
  const int qlo = q0 < 0 ? 0 : q0;
  const int qhi = g.n == 0 ? qlo : (g.t0 + g.n + kPoolHalo < L ? g.t0 + g.n + kPoolHalo : L);
#pragma unroll
  for (int j = 0; j < kRegSlots; ++j) r[j] = __float_as_uint(-__builtin_inff());
#pragma unroll 1
  for (int b = 0; b < L; b += kSelectLdsKeys) {   // uniform: two chunks
    const int nc = L - b < kSelectLdsKeys ? L - b : kSelectLdsKeys;
    stage_f32(nc, in + b, vals);
    __syncthreads();
    // slots [lo, hi) of this thread fall in the chunk [b, b + nc)
    const int lo = (qlo > b ? qlo : b) - q0, hi = (qhi < b + nc ? qhi : b + nc) - q0;
#pragma unroll
    for (int j = 0; j < kRegSlots; ++j)
      if (j >= lo && j < hi) r[j] = vals[q0 + j - b];
    __syncthreads();
  }
}

// Max-pool in place: r[i] becomes the order key of the pooled score of run entry i (which
// needs r[i .. i + 2 * kPoolHalo], none of them overwritten yet), and 0 for i >= n.  Key 0
// lies below the key of every float but one NaN pattern, so these padding entries rank
// below every real entry: the visits below take all kRegRun slots with no per-entry
// condition (such conditions would be kept as one lane mask per slot in scalar registers).
__device__ __forceinline__ void pool_regs(int hw, int n, uint32_t (&r)[kRegSlots]) {
#pragma unroll
  for (int i = 0; i < kRegRun; ++i) {
    float m = __uint_as_float(r[i + kPoolHalo]);
#pragma unroll
    for (int d = 1; d <= kPoolHalo; ++d)
      if (d <= hw)
        m = fmaxf(m, fmaxf(__uint_as_float(r[i + kPoolHalo - d]),
                           __uint_as_float(r[i + kPoolHalo + d])));
    r[i] = i < n ? order_key(m) : 0u;
  }
}

// Every slot of the run, padding included (0 < k < L: the k-th largest key is a real one,
// and padding keys never exceed or equal it).  Each key passes through an empty asm
// statement, so nothing computed from the keys in one visit is kept for the next (the
// compiler would otherwise hoist per-slot values out of the radix loops, 63 of them at a
// time, and spill).
template <typename F>
__device__ __forceinline__ void visit_regs(const uint32_t (&r)[kRegSlots], F f) {
#pragma unroll
  for (int i = 0; i < kRegRun; ++i) {
    uint32_t kk = r[i];
    asm volatile("" : "+v"(kk));
    f(i, kk);
  }
}

// The pooled scores out, through LDS a chunk at a time (coalesced stores).
__device__ __forceinline__ void pooled_out_regs(int L, RunGeom g, const uint32_t (&r)[kRegSlots],
                                                uint32_t* vals, float* pout) {
#pragma unroll 1
  for (int b = 0; b < L; b += kSelectLdsKeys) {
    const int nc = L - b < kSelectLdsKeys ? L - b : kSelectLdsKeys;
    // run entries [lo, hi) lie in the chunk
    const int lo = b - g.t0 > 0 ? b - g.t0 : 0, hi = b + nc - g.t0 < g.n ? b + nc - g.t0 : g.n;
#pragma unroll
    for (int i = 0; i < kRegRun; ++i)
      if (i >= lo && i < hi) vals[g.t0 + i - b] = r[i];
    __syncthreads();
    copy_out_u32(nc, vals, pout + b, KeyToFloatBits());
    __syncthreads();
  }
}

// kSelectLdsKeys < L <= kSelectRegKeys, hw <= kPoolHalo: stage, pool, pooled scores out,
// radix select, emit -- the steps of select_lds with the keys in registers.
__device__ __forceinline__ void select_regs(int L, int k, int hw, const float* __restrict__ in,
                                            float* pout, int32_t* __restrict__ kout,
                                            uint32_t* vals, uint32_t* hist, int64_t* scan_tmp,
                                            uint32_t* mm_tmp, int* s_bin, uint32_t* s_above) {
  const RunGeom g = run_geom(L);
  uint32_t r[kRegSlots];
  stage_regs(L, in, g, vals, r);
  pool_regs(hw, g.n, r);
  if (pout) pooled_out_regs(L, g, r, vals, pout);
  if (k <= 0) return;
  if (k >= L) {
    for (int t = threadIdx.x; t < L; t += kSelectThreads) kout[t] = t;
    return;
  }
  // the key range of the real entries; the passes leave the padding (below it) out
  uint32_t lo, hi, tau, need;
  auto visit = [&](auto f) { visit_regs(r, f); };
  real_key_range_by(visit, mm_tmp, &lo, &hi);
  radix_tau_by<true>(visit, k, lo, hi, hist, scan_tmp, s_bin, s_above, &tau, &need);
  emit_kept_by(visit, g, tau, need, k, scan_tmp, reinterpret_cast<int32_t*>(vals), kout,
               nullptr, nullptr);
}

// Segments longer than the LDS capacity: the same steps on the pooled scores in global
// memory.
__device__ __forceinline__ void select_global(int L, int k, int hw, const float* __restrict__ in,
                                              float* pout, int32_t* __restrict__ kout,
                                              uint32_t* hist, int64_t* scan_tmp, int* s_bin,
                                              uint32_t* s_above) {
  const int tid = threadIdx.x;
  for (int t = tid; t < L; t += kSelectThreads) {
    const int lo = t - hw < 0 ? 0 : t - hw, hi = t + hw >= L ? L - 1 : t + hw;
    float m = in[t];
    for (int x = lo; x <= hi; ++x) m = fmaxf(m, in[x]);
    pout[t] = canonical(m);   // -0 as +0, as the other paths write it
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

// The selection of segment (r, h): pooled scores and kept indices.  Returns k.  For a
// segment held in LDS (L <= kSelectLdsKeys) either output may be null (not written).
__device__ __forceinline__ int select_segment(const DevProblem& dp, const ReqPlan& pl, int r,
                                              int h, const float* __restrict__ scores,
                                              float* pooled, int32_t* __restrict__ kout,
                                              uint32_t* lds_keys, uint32_t* hist,
                                              int64_t* scan_tmp, uint32_t* mm_tmp, int* s_bin,
                                              uint32_t* s_above) {
  const int L = pl.L;
  const int b = dp.budgets[r * dp.Hkv + h];
  const int k = b < L ? b : L;
  const float* in = scores + pl.seg_off + (int64_t)h * L;
  float* pout = pooled ? pooled + pl.seg_off + (int64_t)h * L : nullptr;
  const int hw = dp.pool_window / 2;
  if (L <= kSelectLdsKeys)
    select_lds(L, k, hw, in, pout, kout, lds_keys, hist, scan_tmp, mm_tmp, s_bin, s_above);
  else if (L <= kSelectRegKeys && hw <= kPoolHalo)
    select_regs(L, k, hw, in, pout, kout, lds_keys, hist, scan_tmp, mm_tmp, s_bin, s_above);
  else
    select_global(L, k, hw, in, pout, kout, hist, scan_tmp, s_bin, s_above);
  return k;
}

}  // namespace

__global__ __launch_bounds__(kSelectThreads) void select_kernel(DevProblem dp, int r0,
                                                                const float* __restrict__ scores,
                                                                float* pooled,
                                                                int32_t* __restrict__ kept) {
  if (!plan_ok(dp)) return;   // the workspace holds another problem's plan
  extern __shared__ uint32_t lds_keys[];
  __shared__ uint32_t hist[kMaxBins];
  __shared__ int64_t scan_tmp[17];
  __shared__ uint32_t mm_tmp[32];
  __shared__ int s_bin;
  __shared__ uint32_t s_above;

  const int h = blockIdx.x, r = r0 + (int)blockIdx.y;
  const ReqPlan pl = dp.plan[r];
  select_segment(dp, pl, r, h, scores, pooled, kept + dp.kept_off[r * dp.Hkv + h], lds_keys,
                 hist, scan_tmp, mm_tmp, &s_bin, &s_above);
}

// ---- selection and fresh-page compaction in one kernel (small problems) ------------------
//
// Two forms, with results equal to select_kernel then the fresh-page compaction, bit for bit.
// New slot j of head h is row (j % 16, h) of fresh page j / 16: the heads of a page are
// disjoint rows, so workgroups of different heads never write the same bytes.
//
// select_compact_kernel: one 1024-thread workgroup per (request, KV head) selects the
// segment as select_kernel does, then copies its own head's kept K and V rows to their fresh
// slots and writes the head's new length.  The block-table rewrite of a request must follow
// every read of its old row, so it falls to the request's last workgroup to finish: each
// workgroup counts itself in a per-request counter once its reads are done, and the one that
// completes the count rewrites the row and the freed list and sets the counter back to zero
// for the next launch (the plan kernel zeroes the counters too).  Nothing waits on another
// workgroup.
//
// select_compact_split_kernel: `splits` workgroups per (request, KV head), for batches whose
// rows are few enough that a copy by whole pages (the separate gather) does not pay for its
// extra launches.  Each part first copies the request's old block-table row and its own
// fresh page ids into LDS and counts itself at once (its last read of the row is done), then
// selects the segment (the same steps on the same scores, so the same entries: selecting it
// more than once costs nothing the otherwise idle CUs would do), and copies the slots
// [k p / splits, k (p + 1) / splits) of part p.  Part 0 writes the pooled scores, the kept
// indices and the new length; every part reads the kept indices from its own LDS, where the
// selection leaves them.  The counter's round trip and the page-id reads thus overlap the
// selection, and the copy phase touches global memory only for the rows themselves.
constexpr int kFusedRows = kSelectThreads;   // destination slots resolved per chunk
constexpr int kFusedBatch = 8;               // 16-byte loads of a thread in flight together
// LDS of the copy tables: source and destination row of every slot of a chunk.
constexpr size_t kFusedLdsBytes = 2 * sizeof(int64_t) * kFusedRows;
// The split form: segments up to this length (keys, tables and page ids share LDS), at most
// this many bytes of kept K and V rows in the whole batch, workgroups aimed for (one per
// CU), at most this many parts, at least this many slots per part.
constexpr int kSplitMaxKeys = 28672;
constexpr int64_t kSplitMaxBytes = 32ll << 20;
constexpr int kSplitTargetGroups = 256;
constexpr int kMaxSplits = 16;
constexpr int kSplitMinSlots = 128;
constexpr int kStaticSelectLds = kMaxBins * 4 + 17 * 8 + 32 * 4 + 16;   // the kernels' own LDS
static_assert(kSplitMaxKeys <= kSelectLdsKeys, "split segments are selected in LDS");

// Rows n of the chunk tables (src_off[i] -> dst_off[i], element offsets in the K plane) move
// in 16-byte pieces, K rows then V rows.  Whole batches of kFusedBatch pieces per thread
// carry no condition, so their loads are in flight together (a condition per piece made the
// compiler wait for every outstanding access before each load and store); pieces past the
// end of the last batch repeat the last piece (the same bytes to the same place).
__device__ __forceinline__ void copy_table_rows(uint16_t* kv, const int64_t* src_off,
                                                const int64_t* dst_off, int n, int CH,
                                                int64_t plane) {
  const int tid = threadIdx.x, half = n * CH, items = 2 * half;
  auto piece = [&](int it, int64_t* from, int64_t* to) {
    const bool v_plane = it >= half;
    const int i = v_plane ? it - half : it;
    const int64_t add = (v_plane ? plane : 0) + (i % CH) * 8;
    *from = src_off[i / CH] + add;
    *to = dst_off[i / CH] + add;
  };
  constexpr int kStep = kSelectThreads * kFusedBatch;
  const int full = items / kStep * kStep;
#pragma unroll 1
  for (int base = 0; base < items; base += kStep) {
    const bool whole = base < full;   // uniform
    u32x4 v[kFusedBatch];
    int64_t to[kFusedBatch];
#pragma unroll
    for (int u = 0; u < kFusedBatch; ++u) {
      const int it = base + u * kSelectThreads + tid;
      int64_t from;
      piece(whole || it < items ? it : items - 1, &from, &to[u]);
      v[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(kv + from));
    }
#pragma unroll
    for (int u = 0; u < kFusedBatch; ++u)
      __builtin_nontemporal_store(v[u], reinterpret_cast<u32x4*>(kv + to[u]));
  }
}

__global__ __launch_bounds__(kSelectThreads) void select_compact_kernel(
    DevProblem dp, const float* __restrict__ scores, float* pooled, int32_t* __restrict__ kept,
    uint16_t* kv, int32_t* bt, const int32_t* __restrict__ free_pages,
    int32_t* __restrict__ freed, int32_t* __restrict__ new_lens) {
  if (!plan_ok(dp)) return;   // the workspace holds another problem's plan
  extern __shared__ uint32_t lds_keys[];
  __shared__ uint32_t hist[kMaxBins];
  __shared__ int64_t scan_tmp[17];
  __shared__ uint32_t mm_tmp[32];
  __shared__ int s_bin;
  __shared__ uint32_t s_above;
  __shared__ int s_last;

  const int tid = threadIdx.x;
  const int h = blockIdx.x, r = blockIdx.y, Hkv = dp.Hkv, D = dp.D;
  const ReqPlan pl = dp.plan[r];
  int32_t* kout = kept + dp.kept_off[r * Hkv + h];
  const int k = select_segment(dp, pl, r, h, scores, pooled, kout, lds_keys, hist, scan_tmp,
                               mm_tmp, &s_bin, &s_above);
  if (tid == 0) new_lens[r * Hkv + h] = pl.skip ? pl.L : k;
  if (pl.skip) return;   // every head keeps everything: the request is left as it is
  __syncthreads();   // the kept indices written above are visible to the workgroup

  // ---- copies: chunks of kFusedRows new slots, resolved to (source, destination) element
  // offsets of the K plane in LDS (only the slots with both, packed in slot order; the
  // tables overlay the selection's keys)
  int64_t* src_off = reinterpret_cast<int64_t*>(lds_keys);
  int64_t* dst_off = src_off + kFusedRows;
  const int64_t plane = dp.num_pages * kPageSize * Hkv * (int64_t)D;   // K -> V, elements
  const int32_t* bt_row = bt + (int64_t)r * dp.bt_stride;
#pragma unroll 1
  for (int j0 = 0; j0 < k; j0 += kFusedRows) {
    const int nj = k - j0 < kFusedRows ? k - j0 : kFusedRows;
    int64_t src = -1, dst = -1;
    if (tid < nj) {
      const int j = j0 + tid;
      const int t = kout[j];
      if (t >= 0 && t < pl.L) {
        const int64_t page = bt_row[t / kPageSize];
        // pages outside the pool are never dereferenced (the slot is left unwritten)
        if (page >= 0 && page < dp.num_pages)
          src = ((page * kPageSize + t % kPageSize) * Hkv + h) * (int64_t)D;
      }
      const int64_t dpg = free_pages[pl.fresh_off + j / kPageSize];
      if (dpg >= 0 && dpg < dp.num_pages) dst = ((dpg * kPageSize + j % kPageSize) * Hkv + h) * (int64_t)D;
    }
    uint32_t nvalid;
    const bool valid = src >= 0 && dst >= 0;
    const uint32_t at = block_excl_count(valid, mm_tmp, &nvalid);
    if (valid) {
      src_off[at] = src;
      dst_off[at] = dst;
    }
    __syncthreads();
    copy_table_rows(kv, src_off, dst_off, (int)nvalid, D / 8, plane);
    __syncthreads();   // the tables are rewritten by the next chunk
  }

  // ---- the request's last workgroup rewrites its block-table row and freed list
  if (tid == 0) {
    __threadfence();   // this workgroup's reads of the old row are done
    s_last = atomicAdd(&dp.req_done[r], 1) == Hkv - 1;
  }
  __syncthreads();
  if (!s_last) return;
  __threadfence();
  int32_t* row = bt + (int64_t)r * dp.bt_stride;
  for (int i = tid; i < pl.Y; i += kSelectThreads) {
    const int32_t old = row[i];
    freed[pl.freed_off + i] = old;
    row[i] = i < pl.X ? free_pages[pl.fresh_off + i] : -1;
  }
  if (tid == 0) dp.req_done[r] = 0;   // ready for the next launch on this workspace
}

// LDS of the split form, in 32-bit words from the start of the dynamic LDS: the selection's
// keys (then the kept indices), the copy tables, the old block-table row, the part's fresh
// page ids.
struct SplitLds {
  int table_off, row_off, fresh_off, words;
};

__host__ __device__ constexpr SplitLds split_lds(int64_t max_L, int64_t max_k, int splits) {
  const int table_off = (int)((max_L + kLdsPad + 1) / 2 * 2);   // 8-byte aligned
  const int row_off = table_off + (int)(kFusedLdsBytes / sizeof(uint32_t));
  const int fresh_off = row_off + (int)((max_L + kPageSize - 1) / kPageSize);
  const int64_t part_slots = (max_k + splits - 1) / splits;
  return SplitLds{table_off, row_off, fresh_off,
                  fresh_off + (int)((part_slots + kPageSize - 1) / kPageSize) + 1};
}
// the largest layout (two parts of the longest segment, everything kept) fits one CU's LDS
static_assert(split_lds(kSplitMaxKeys, kSplitMaxKeys, 2).words * sizeof(uint32_t) +
                  kStaticSelectLds <= 160 * 1024,
              "the split form's LDS fits a workgroup");

__global__ __launch_bounds__(kSelectThreads) void select_compact_split_kernel(
    DevProblem dp, const float* __restrict__ scores, float* pooled, int32_t* __restrict__ kept,
    uint16_t* kv, int32_t* bt, const int32_t* __restrict__ free_pages,
    int32_t* __restrict__ freed, int32_t* __restrict__ new_lens, int splits, SplitLds lay) {
  if (!plan_ok(dp)) return;   // the workspace holds another problem's plan
  extern __shared__ uint32_t lds_keys[];
  __shared__ uint32_t hist[kMaxBins];
  __shared__ int64_t scan_tmp[17];
  __shared__ uint32_t mm_tmp[32];
  __shared__ int s_bin;
  __shared__ uint32_t s_above;
  __shared__ int s_last;

  const int tid = threadIdx.x;
  const int h = (int)blockIdx.x / splits, part = (int)blockIdx.x - h * splits;
  const int r = blockIdx.y, Hkv = dp.Hkv, D = dp.D;
  const bool lead = part == 0;
  const ReqPlan pl = dp.plan[r];
  int32_t* kout = kept + dp.kept_off[r * Hkv + h];
  if (pl.skip) {   // every head keeps everything: the request is left as it is
    if (!lead) return;
    select_segment(dp, pl, r, h, scores, pooled, kout, lds_keys, hist, scan_tmp, mm_tmp,
                   &s_bin, &s_above);
    if (tid == 0) new_lens[r * Hkv + h] = pl.L;
    return;
  }
  // this part's new slots (k as select_segment takes it)
  const int b = dp.budgets[r * Hkv + h];
  const int kk = b < pl.L ? b : pl.L;
  const int j_lo = (int)((int64_t)kk * part / splits);
  const int j_hi = (int)((int64_t)kk * (part + 1) / splits);
  const int pg_lo = j_lo / kPageSize;
  const int pg_n = j_hi > j_lo ? (j_hi - 1) / kPageSize - pg_lo + 1 : 0;

  // ---- page ids into LDS, then this workgroup counts itself: its reads of the old row are
  // done, so the request's last workgroup to count may rewrite the row at any time after
  int32_t* row_lds = reinterpret_cast<int32_t*>(lds_keys + lay.row_off);
  int32_t* fresh_lds = reinterpret_cast<int32_t*>(lds_keys + lay.fresh_off);
  const int32_t* bt_row = bt + (int64_t)r * dp.bt_stride;
  for (int i = tid; i < pl.Y; i += kSelectThreads) row_lds[i] = bt_row[i];
  for (int i = tid; i < pg_n; i += kSelectThreads) fresh_lds[i] = free_pages[pl.fresh_off + pg_lo + i];
  __syncthreads();   // every thread's row reads have returned
  int ticket = 0;    // thread 0: this workgroup's place in the request's count
  if (tid == 0) {
    __threadfence();
    ticket = atomicAdd(&dp.req_done[r], 1);
  }

  const int k = select_segment(dp, pl, r, h, scores, lead ? pooled : nullptr,
                               lead ? kout : nullptr, lds_keys, hist, scan_tmp, mm_tmp, &s_bin,
                               &s_above);
  if (lead && tid == 0) new_lens[r * Hkv + h] = k;
  __syncthreads();   // the kept indices in LDS are complete

  // ---- copies: chunks of kFusedRows new slots of this part, resolved from LDS alone
  const int32_t* kidx = reinterpret_cast<const int32_t*>(lds_keys);   // for 0 < k < L
  int64_t* src_off = reinterpret_cast<int64_t*>(lds_keys + lay.table_off);
  int64_t* dst_off = src_off + kFusedRows;
  const int64_t plane = dp.num_pages * kPageSize * Hkv * (int64_t)D;   // K -> V, elements
#pragma unroll 1
  for (int j0 = j_lo; j0 < j_hi; j0 += kFusedRows) {
    const int nj = j_hi - j0 < kFusedRows ? j_hi - j0 : kFusedRows;
    int64_t src = -1, dst = -1;
    if (tid < nj) {
      const int j = j0 + tid;
      const int t = k >= pl.L ? j : kidx[j];
      if (t >= 0 && t < pl.L) {
        const int64_t page = row_lds[t / kPageSize];
        // pages outside the pool are never dereferenced (the slot is left unwritten)
        if (page >= 0 && page < dp.num_pages)
          src = ((page * kPageSize + t % kPageSize) * Hkv + h) * (int64_t)D;
      }
      const int64_t dpg = fresh_lds[j / kPageSize - pg_lo];
      if (dpg >= 0 && dpg < dp.num_pages) dst = ((dpg * kPageSize + j % kPageSize) * Hkv + h) * (int64_t)D;
    }
    uint32_t nvalid;
    const bool valid = src >= 0 && dst >= 0;
    const uint32_t at = block_excl_count(valid, mm_tmp, &nvalid);
    if (valid) {
      src_off[at] = src;
      dst_off[at] = dst;
    }
    __syncthreads();
    copy_table_rows(kv, src_off, dst_off, (int)nvalid, D / 8, plane);
    __syncthreads();   // the tables are rewritten by the next chunk
  }

  // ---- the request's last workgroup to count rewrites its row and freed list (the old row
  // from LDS; every other workgroup read it before counting)
  if (tid == 0) s_last = ticket == Hkv * splits - 1;
  __syncthreads();
  if (!s_last) return;
  int32_t* row = bt + (int64_t)r * dp.bt_stride;
  for (int i = tid; i < pl.Y; i += kSelectThreads) {
    freed[pl.freed_off + i] = row_lds[i];
    row[i] = i < pl.X ? free_pages[pl.fresh_off + i] : -1;
  }
  if (tid == 0) dp.req_done[r] = 0;   // ready for the next launch on this workspace
}

// ---- the same selection beside a running scoring kernel ----------------------------------
//
// select_side_kernel computes exactly what select_kernel computes (the pooled scores and the
// kept indices of every (request, KV head) of a range of requests) on a small budget: 512
// threads of at most 72 registers and about 45 KB of LDS, meant to run beside other kernels
// (the pipelined step runs it on a second stream).  By the register and LDS counts two of
// its waves per SIMD fit beside a scoring wave; measured on MI355X they are not placed
// there, and the kernel starts as the scoring kernel's workgroups leave.  The segment stays
// in global memory (it was just written: the passes read it from L2), in tiles of kSideTile
// entries whose successor is always in flight:
//   pool   each tile plus the window's halo is staged in LDS (two buffers, one barrier per
//          tile), pooled, written out and counted into the first histogram (key bits 31..21)
//   radix  the second histogram (bits 20..10) counts the keys that match the first digit,
//          which are also gathered into LDS when they fit (kSideCand of them); the third
//          (bits 9..0) is then counted from LDS, else by another pass.  Result: tau, the key
//          of the k-th largest entry, and how many entries equal to tau are taken
//   emit   each thread owns kSidePer consecutive entries of a tile; a workgroup prefix sum of
//          (greater, equal) counts, carried from tile to tile, places the kept indices in
//          ascending order (ties to the lower index)
namespace {

constexpr int kSideThreads = 512;
constexpr int kSidePer = 8;                            // entries per thread and tile
constexpr int kSideTile = kSideThreads * kSidePer;     // 4096
constexpr int kSideHalo = kMaxPoolWindow / 2;          // widest pooling half-window
constexpr int kSideStage = kSideTile + 2 * kSideHalo;  // staged raw scores per tile
constexpr int kSideLoads = (kSideStage + kSideThreads - 1) / kSideThreads;   // 9
constexpr int kSideBuf = kSideLoads * kSideThreads;    // one staging buffer (floats)
constexpr int kSideCand = 2 * kSideBuf;                // candidate keys the buffers hold

// f(v, t) for every entry t < L of the segment, v = p[t], thread tid taking entries
// base + j * kSideThreads + tid of each tile: coalesced, the next tile's loads issued before
// the current tile is processed.
template <typename F>
__device__ __forceinline__ void side_pass(const float* __restrict__ p, int L, F f) {
  const int tid = threadIdx.x;
  float cur[kSidePer], nxt[kSidePer];
#pragma unroll
  for (int j = 0; j < kSidePer; ++j) {
    const int t = j * kSideThreads + tid;
    cur[j] = t < L ? p[t] : 0.0f;
  }
#pragma unroll 1
  for (int base = 0; base < L; base += kSideTile) {
    const int nb = base + kSideTile;
#pragma unroll
    for (int j = 0; j < kSidePer; ++j) {
      const int t = nb + j * kSideThreads + tid;
      nxt[j] = t < L ? p[t] : 0.0f;
    }
#pragma unroll
    for (int j = 0; j < kSidePer; ++j) {
      const int t = base + j * kSideThreads + tid;
      if (t < L) f(cur[j], t);
    }
#pragma unroll
    for (int j = 0; j < kSidePer; ++j) cur[j] = nxt[j];
  }
}

// The entries of this thread's run in tile `base` (kSidePer consecutive from
// base + tid * kSidePer), -inf past the end (never compared: masked by the caller).
__device__ __forceinline__ void side_run_load(const float* __restrict__ p, int L, int base,
                                              float (&v)[kSidePer]) {
  const int t0 = base + (int)threadIdx.x * kSidePer;
#pragma unroll
  for (int j = 0; j < kSidePer; ++j) v[j] = t0 + j < L ? p[t0 + j] : -__builtin_inff();
}

// Appends this lane's key to the LDS list when `take` (one LDS atomic per wave).
__device__ __forceinline__ void side_append(bool take, uint32_t key, uint32_t* list,
                                            uint32_t* count, int cap) {
  const uint64_t bal = __ballot(take);
  if (!bal) return;
  const int lane = threadIdx.x & 63;
  uint32_t at = 0;
  if (lane == __builtin_ctzll(bal)) at = atomicAdd(count, (uint32_t)__popcll(bal));
  at = __shfl((int)at, __builtin_ctzll(bal), 64);
  const uint32_t below = __builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32),
                                                   __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u));
  if (take && at + below < (uint32_t)cap) list[at + below] = key;
}

}  // namespace

__global__ __launch_bounds__(kSideThreads, 6) void select_side_kernel(
    DevProblem dp, int r0, const float* __restrict__ scores, float* pooled,
    int32_t* __restrict__ kept) {
  if (!plan_ok(dp)) return;   // the workspace holds another problem's plan
  __shared__ float raw[2][kSideBuf];
  __shared__ uint32_t hist[kMaxBins];
  __shared__ int64_t scan_tmp[17];
  __shared__ int s_bin;
  __shared__ uint32_t s_above, s_count, s_ncand;

  const int tid = threadIdx.x;
  const int h = blockIdx.x, r = r0 + (int)blockIdx.y, Hkv = dp.Hkv;
  const ReqPlan pl = dp.plan[r];
  const int L = pl.L;
  const int b = dp.budgets[r * Hkv + h];
  const int k = b < L ? b : L;
  const float* in = scores + pl.seg_off + (int64_t)h * L;
  float* pout = pooled + pl.seg_off + (int64_t)h * L;
  int32_t* kout = kept + dp.kept_off[r * Hkv + h];
  const int hw = dp.pool_window / 2;
  const float ninf = -__builtin_inff();

  // ---- pool (window clipped at the segment's ends) and the first digit.  Tile i is staged
  // in raw[i & 1]: that buffer was last read while pooling tile i - 2, before the barrier of
  // tile i - 1, so one barrier per tile suffices.
  for (int i = tid; i < kMaxBins; i += kSideThreads) hist[i] = 0;
  float v[kSideLoads];
#pragma unroll
  for (int u = 0; u < kSideLoads; ++u) {
    const int t = -hw + u * kSideThreads + tid;
    v[u] = (t >= 0 && t < L) ? in[t] : ninf;
  }
#pragma unroll 1
  for (int base = 0, tile = 0; base < L; base += kSideTile, ++tile) {
    float* buf = raw[tile & 1];
#pragma unroll
    for (int u = 0; u < kSideLoads; ++u) buf[u * kSideThreads + tid] = v[u];
    __syncthreads();   // the staged tile is visible (and, before tile 0, hist is zeroed)
    const int nb = base + kSideTile;
#pragma unroll
    for (int u = 0; u < kSideLoads; ++u) {   // the next tile's loads, in flight while pooling
      const int t = nb - hw + u * kSideThreads + tid;
      v[u] = (nb < L && t >= 0 && t < L) ? in[t] : ninf;
    }
#pragma unroll
    for (int j = 0; j < kSidePer; ++j) {
      const int i = j * kSideThreads + tid, t = base + i;
      if (t < L) {
        float m = buf[i + hw];
        for (int d = 1; d <= hw; ++d) m = fmaxf(m, fmaxf(buf[i + hw - d], buf[i + hw + d]));
        const uint32_t key = order_key(m);
        pout[t] = key_value(key);
        atomicAdd(&hist[key >> 21], 1u);
      }
    }
  }
  __syncthreads();   // pooled scores written (and visible to the workgroup), hist complete
  if (k <= 0) return;
  if (k >= L) {
    for (int t = tid; t < L; t += kSideThreads) kout[t] = t;
    return;
  }

  // ---- radix: tau and how many of the entries equal to it are taken
  uint32_t need = (uint32_t)k;
  find_bin<kSideThreads>(hist, kMaxBins, need, scan_tmp, &s_bin, &s_above);
  uint32_t prefix = (uint32_t)s_bin;
  need -= s_above;
  if (tid == 0) { s_count = hist[prefix]; s_ncand = 0; }
  __syncthreads();
  const bool in_lds = s_count <= (uint32_t)kSideCand;   // uniform
  uint32_t* cand = reinterpret_cast<uint32_t*>(&raw[0][0]);
  for (int i = tid; i < kMaxBins; i += kSideThreads) hist[i] = 0;
  __syncthreads();
  side_pass(pout, L, [&](float x, int) {
    const uint32_t key = order_key(x);
    const bool match = (key >> 21) == prefix;
    if (match) atomicAdd(&hist[(key >> 10) & (kMaxBins - 1)], 1u);
    if (in_lds) side_append(match, key, cand, &s_ncand, kSideCand);
  });
  __syncthreads();
  find_bin<kSideThreads>(hist, kMaxBins, need, scan_tmp, &s_bin, &s_above);
  prefix = (prefix << 11) | (uint32_t)s_bin;
  need -= s_above;
  for (int i = tid; i < kMaxBins / 2; i += kSideThreads) hist[i] = 0;
  __syncthreads();
  if (in_lds) {
    const int nc = (int)s_count;
    for (int i = tid; i < nc; i += kSideThreads) {
      const uint32_t key = cand[i];
      if ((key >> 10) == prefix) atomicAdd(&hist[key & (kMaxBins / 2 - 1)], 1u);
    }
  } else {
    side_pass(pout, L, [&](float x, int) {
      const uint32_t key = order_key(x);
      if ((key >> 10) == prefix) atomicAdd(&hist[key & (kMaxBins / 2 - 1)], 1u);
    });
  }
  __syncthreads();
  find_bin<kSideThreads>(hist, kMaxBins / 2, need, scan_tmp, &s_bin, &s_above);
  const uint32_t tau = (prefix << 10) | (uint32_t)s_bin;
  need -= s_above;

  // ---- emit: every key > tau, then the first `need` keys == tau, in index order
  int64_t gt_carry = 0, eq_carry = 0;   // uniform: counts of the tiles before
  float cur[kSidePer], nxt[kSidePer];
  side_run_load(pout, L, 0, cur);
#pragma unroll 1
  for (int base = 0; base < L; base += kSideTile) {
    side_run_load(pout, L, base + kSideTile, nxt);   // in flight during this tile
    const int t0 = base + tid * kSidePer;
    uint32_t gtm = 0, eqm = 0;
#pragma unroll
    for (int j = 0; j < kSidePer; ++j) {
      const uint32_t key = order_key(cur[j]);
      const bool in_seg = t0 + j < L;
      gtm |= (uint32_t)(in_seg && key > tau) << j;
      eqm |= (uint32_t)(in_seg && key == tau) << j;
    }
    const int64_t n_gt = __popc(gtm), n_eq = __popc(eqm);
    int64_t tot;
    const int64_t ex = block_excl_scan_i64((n_eq << 32) | n_gt, scan_tmp, &tot);
    const int64_t eq_before = eq_carry + (ex >> 32), gt_before = gt_carry + (ex & 0xFFFFFFFFll);
    int64_t eq_take = (int64_t)need - eq_before;
    eq_take = eq_take < 0 ? 0 : (eq_take > n_eq ? n_eq : eq_take);
    for (int64_t drop = n_eq - eq_take; drop > 0; --drop)   // keep the first eq_take ties
      eqm &= ~(1u << (31 - __clz(eqm)));
    int64_t pos = gt_before + (eq_before < (int64_t)need ? eq_before : (int64_t)need);
    for (uint32_t m = gtm | eqm; m; m &= m - 1, ++pos)   // pos < k by the counts above
      if (pos < k) kout[pos] = t0 + __builtin_ctz(m);
    gt_carry += tot & 0xFFFFFFFFll;
    eq_carry += tot >> 32;
#pragma unroll
    for (int j = 0; j < kSidePer; ++j) cur[j] = nxt[j];
  }
}

// ---- attention-aware LRFU keep scores (Sec. 5.1; Alg. 1 steps 2-5) -----------------------
//
// Hit mask (Alg. 1 step 3): the shortest prefix of the segment ordered by pooled score
// descending (ties: lower index first) whose running mass reaches top_p times the total.
// Masses are exact 64-bit fixed-point values (each score scaled by 2^S and truncated, S
// chosen so that the segment's total cannot overflow), so every sum is exact and
// order-independent: the same radix search as the selection, with mass histograms in place
// of counts, finds the boundary key tau and the mass still needed from entries equal to tau;
// those are then taken in index order.  Entries with a score <= 0 carry no mass.  A hit
// entry always has a positive score, so the hit decision is carried from here on by the
// contribution hit ? score : 0 that replaces the pooled score in LDS.
namespace {

// floor(v * 2^S) for the positive float whose order key is `key` (0 for v <= 0), by integer
// shifts of the significand: exact, as long as the result stays below 2^64.
__device__ __forceinline__ uint64_t fixed_mass(uint32_t key, int S) {
  if (key <= 0x80000000u) return 0ull;   // negative or zero
  const uint32_t u = key & 0x7FFFFFFFu, ex = u >> 23;
  const uint64_t sig = (u & 0x7FFFFFu) | (ex ? 0x800000u : 0u);
  const int sh = (ex ? (int)ex : 1) - 150 + S;   // v = sig * 2^((ex ? ex : 1) - 150)
  return sh >= 0 ? sig << sh : (sh > -64 ? sig >> -sh : 0ull);
}

// The top-p hit mask turned into contributions: every key of the run is replaced by the key
// of its contribution, the pooled score where it is hit, else 0.  visit(f) reads the keys as
// in the selection; rewrite(f) replaces each key kk of the run by f(kk), in index order.
template <typename Visit, typename Rewrite>
__device__ __forceinline__ void topp_contributions_by(int L, Visit visit, Rewrite rewrite,
                                                      float top_p, uint64_t* hist64,
                                                      int64_t* scan_tmp, uint32_t* mm_tmp,
                                                      int* s_bin, uint64_t* s_above) {
  constexpr uint32_t kZero = 0x80000000u;   // order_key(0.0f)
  auto keep_contributions = [&](auto keep) {
    rewrite([&](uint32_t kk) { return keep(kk) ? kk : kZero; });
  };
  const int tid = threadIdx.x;
  uint32_t lo, hi;
  // the range of the real keys (a run in registers carries padding keys, 0; they have no
  // mass, like every key at or below that of 0.0f, and never enter the histograms); its
  // barriers retire the pooled copy-out
  real_key_range_by(visit, mm_tmp, &lo, &hi);
  const float vmax = key_value(hi);
  if (!(vmax > 0.f) || !(top_p > 0.f)) {   // no positive mass to reach
    keep_contributions([](uint32_t) { return false; });
    return;
  }
  if (top_p >= 1.f) {   // the whole mass: every entry with a positive score
    keep_contributions([](uint32_t kk) { return kk > 0x80000000u; });
    return;
  }
  int e;
  frexpf(vmax, &e);   // every score < 2^e
  const int lg = 32 - __clz((uint32_t)L + 1u);   // L + 1 <= 2^lg
  const int S = 62 - e - lg;                     // total < L * 2^(e + S) < 2^62
  uint64_t mine = 0;
  // each mass passes through an empty asm statement before it is added: the sum then runs
  // slot by slot instead of all of a run's 64-bit masses being held at once
  visit([&](int, uint32_t kk) {
    uint64_t m = fixed_mass(kk, S);
    asm volatile("" : "+v"(m));
    mine += m;
  });
  int64_t total;
  block_excl_scan_i64((int64_t)mine, scan_tmp, &total);
  const double want = ceil((double)top_p * (double)total);
  uint64_t need = want > 0.0 ? (uint64_t)want : 0ull;
  if (need == 0) {
    keep_contributions([](uint32_t) { return false; });
    return;
  }
  // radix search over d = key - lo with 10-bit digits, masses as weights
  const uint32_t range = hi - lo;
  int rem = range == 0 ? 0 : 32 - __clz(range);
  uint32_t prefix = 0;
#pragma unroll 1
  while (rem > 0) {
    const int bits = rem < 10 ? rem : 10, sh = rem - bits, nbins = 1 << bits;
    for (int bb = tid; bb < nbins; bb += kSelectThreads) hist64[bb] = 0;
    if (tid == 0) { *s_bin = 0; *s_above = 0; }
    __syncthreads();
    visit([&](int, uint32_t kk) {
      const uint32_t dh = (kk - lo) >> sh;
      if ((dh >> bits) == prefix) {
        uint64_t m = fixed_mass(kk, S);
        asm volatile("" : "+v"(m));
        if (m != 0)
          atomicAdd((unsigned long long*)&hist64[dh & (uint32_t)(nbins - 1)],
                    (unsigned long long)m);
      }
    });
    __syncthreads();
    find_bin64(hist64, nbins, need, scan_tmp, s_bin, s_above);
    need -= *s_above;
    prefix = (prefix << bits) | (uint32_t)*s_bin;
    rem = sh;
    __syncthreads();
  }
  const uint32_t tau = lo + prefix;
  // entries equal to tau (each of mass m > 0: the search only descends into bins with
  // mass) are hit, in index order, while the mass before them is still short of the
  // target: the first ceil(need / m) of them
  const uint64_t m_tau = fixed_mass(tau, S);
  uint32_t n_eq = 0;
  visit([&](int, uint32_t kk) { n_eq += kk == tau; });
  int64_t eq_total;
  const int64_t eq_before = block_excl_scan_i64(n_eq, scan_tmp, &eq_total);
  const int64_t take = m_tau == 0 ? eq_total : (int64_t)((need + m_tau - 1) / m_tau);
  int64_t rank = eq_before;
  keep_contributions([&](uint32_t kk) {
    const bool eq = kk == tau;
    const bool h = kk > tau || (eq && rank < take);
    rank += eq ? 1 : 0;
    return h;
  });
}

// The same over the segment's keys in LDS.
__device__ __forceinline__ void topp_contributions(int L, RunGeom g, uint32_t* keys, float top_p,
                                                   uint64_t* hist64, int64_t* scan_tmp,
                                                   uint32_t* mm_tmp, int* s_bin,
                                                   uint64_t* s_above) {
  topp_contributions_by(
      L, [&](auto f) { visit_run(g, keys, f); },
      [&](auto f) { visit_run(g, keys, [&](int i, uint32_t kk) { keys[g.t0 + i] = f(kk); }); },
      top_p, hist64, scan_tmp, mm_tmp, s_bin, s_above);
}

// KS' = decay * KS + contribution, each operation rounded to fp32, over the whole segment
// in coalesced order; KS' goes to ks (in place) and its key replaces the contribution in LDS, the
// hit mask (contribution > 0) to hit_out when given.  Global reads and writes are raw
// buffer accesses over exactly L elements (out-of-range lanes read 0 / are dropped).
__device__ __forceinline__ void keep_score_update(int L, float decay, float* ks,
                                                  uint8_t* hit_out, uint32_t* keys) {
  const __amdgpu_buffer_rsrc_t rk = buffer_over(ks, L * (int)sizeof(float));
  const __amdgpu_buffer_rsrc_t rh = buffer_over(hit_out, hit_out ? L : 0);
  const int off = lane_byte_offset(), last = L > 0 ? L - 1 : 0;
  const int rows = (L + kSelectThreads - 1) / kSelectThreads;
#pragma unroll 1
  for (int r0 = 0; r0 < rows; r0 += kRowBatch) {
    float kv[kRowBatch], cv[kRowBatch];
#pragma unroll
    for (int j = 0; j < kRowBatch; ++j) {
      const int t = threadIdx.x + (r0 + j) * kSelectThreads;
      kv[j] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                            rk, off + (r0 + j) * kSelectThreads * 4, 0, 0));
      cv[j] = key_value(keys[t < last ? t : last]);
    }
#pragma unroll
    for (int j = 0; j < kRowBatch; ++j) {
      const int t = threadIdx.x + (r0 + j) * kSelectThreads;
      const float nk = __fadd_rn(__fmul_rn(decay, kv[j]), cv[j]);
      if (t < L) keys[t] = order_key(nk);
      __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, nk), rk,
                                            off + (r0 + j) * kSelectThreads * 4, 0, 0);
      if (hit_out)
        __builtin_amdgcn_raw_buffer_store_b8((uint8_t)(cv[j] > 0.0f ? 1 : 0), rh,
                                             (int)threadIdx.x + (r0 + j) * kSelectThreads, 0, 0);
    }
  }
}

// One (request, KV head): pool, top-p hit mask, keep-score update, TopK on the keep
// scores with the kept keep scores.
__device__ __forceinline__ void lrfu_lds(int L, int k, int hw, float top_p, float decay,
                                         const float* __restrict__ in, float* pout, float* ks,
                                         uint8_t* hit_out, int32_t* __restrict__ kout,
                                         float* __restrict__ ks_kept, uint32_t* vals,
                                         uint64_t* hist64, int64_t* scan_tmp, uint32_t* mm_tmp,
                                         int* s_bin, uint32_t* s_above32, uint64_t* s_above64) {
  stage_f32(L, in, vals);
  __syncthreads();
  const RunGeom g = run_geom(L);
  pool_in_lds(L, hw, g, vals, pout);
  topp_contributions(L, g, vals, top_p, hist64, scan_tmp, mm_tmp, s_bin, s_above64);
  __syncthreads();
  keep_score_update(L, decay, ks, hit_out, vals);
  __syncthreads();   // also makes this workgroup's writes of ks visible to its own reads
  topk_lds(L, k, g, vals, reinterpret_cast<uint32_t*>(hist64), scan_tmp, mm_tmp, s_bin,
           s_above32, kout, ks, ks_kept);
}

// keep_score_update with the run in registers (contribution keys in, KS' keys out; padding
// slots stay 0): ks passes through LDS a chunk at a time, coalesced both ways; the hit flags
// are stored from the registers.
__device__ __forceinline__ void keep_score_update_regs(int L, float decay, float* ks,
                                                       uint8_t* hit_out, RunGeom g,
                                                       uint32_t (&r)[kRegSlots], uint32_t* vals) {
#pragma unroll 1
  for (int b = 0; b < L; b += kSelectLdsKeys) {   // uniform: two chunks
    const int nc = L - b < kSelectLdsKeys ? L - b : kSelectLdsKeys;
    stage_f32(nc, ks + b, vals);
    __syncthreads();
    const int lo = b - g.t0 > 0 ? b - g.t0 : 0, hi = b + nc - g.t0 < g.n ? b + nc - g.t0 : g.n;
#pragma unroll
    for (int i = 0; i < kRegRun; ++i)
      if (i >= lo && i < hi) {
        const int p = g.t0 + i - b;
        const float c = key_value(r[i]);
        const float nk = __fadd_rn(__fmul_rn(decay, __uint_as_float(vals[p])), c);
        vals[p] = __float_as_uint(nk);
        r[i] = order_key(nk);
        if (hit_out) hit_out[g.t0 + i] = c > 0.0f ? 1 : 0;
      }
    __syncthreads();
    copy_out_u32(nc, vals, ks + b, AsIs());
    __syncthreads();   // also makes this workgroup's writes of ks visible to its own reads
  }
}

// lrfu_lds for kLrfuLdsLen < L <= kSelectRegKeys, hw <= kPoolHalo, with the keys in registers.
__device__ __forceinline__ void lrfu_regs(int L, int k, int hw, float top_p, float decay,
                                          const float* __restrict__ in, float* pout, float* ks,
                                          uint8_t* hit_out, int32_t* __restrict__ kout,
                                          float* __restrict__ ks_kept, uint32_t* vals,
                                          uint64_t* hist64, int64_t* scan_tmp, uint32_t* mm_tmp,
                                          int* s_bin, uint32_t* s_above32, uint64_t* s_above64) {
  const RunGeom g = run_geom(L);
  uint32_t r[kRegSlots];
  stage_regs(L, in, g, vals, r);
  pool_regs(hw, g.n, r);
  if (pout) pooled_out_regs(L, g, r, vals, pout);
  auto visit = [&](auto f) { visit_regs(r, f); };
  auto rewrite = [&](auto f) {
#pragma unroll
    for (int i = 0; i < kRegRun; ++i) r[i] = r[i] == 0u ? 0u : f(r[i]);   // padding stays 0
  };
  topp_contributions_by(L, visit, rewrite, top_p, hist64, scan_tmp, mm_tmp, s_bin, s_above64);
  __syncthreads();
  keep_score_update_regs(L, decay, ks, hit_out, g, r, vals);
  if (k <= 0) return;
  if (k >= L) {
    for (int t = threadIdx.x; t < L; t += kSelectThreads) {
      kout[t] = t;
      ks_kept[t] = ks[t];
    }
    return;
  }
  uint32_t lo, hi, tau, need;
  real_key_range_by(visit, mm_tmp, &lo, &hi);   // padding (0) stays out, as in select_regs
  radix_tau_by<true>(visit, k, lo, hi, reinterpret_cast<uint32_t*>(hist64), scan_tmp, s_bin,
                     s_above32, &tau, &need);
  emit_kept_by(visit, g, tau, need, k, scan_tmp, reinterpret_cast<int32_t*>(vals), kout, ks,
               ks_kept);
}

}  // namespace

// kLong = false: the segments that fit in LDS; kLong = true: the longer ones (a separate
// kernel, launched only when there are any: the register-resident path needs far more
// registers than the LDS path, which keeps its own allocation).
template <bool kLong>
__global__ __launch_bounds__(kSelectThreads) void lrfu_select_kernel(
    DevProblem dp, const float* __restrict__ scores, float top_p, float decay, float* ks,
    uint8_t* hit, float* pooled, int32_t* __restrict__ kept, float* ks_kept) {
  if (!plan_ok(dp)) return;   // the workspace holds another problem's plan
  extern __shared__ uint32_t lds_keys[];
  __shared__ uint64_t hist64[kMaxBins / 2];   // 8 KiB: 64-bit masses, or the 32-bit counts
  __shared__ int64_t scan_tmp[17];
  __shared__ uint32_t mm_tmp[32];
  __shared__ int s_bin;
  __shared__ uint32_t s_above32;
  __shared__ uint64_t s_above64;

  const int h = blockIdx.x, r = blockIdx.y, Hkv = dp.Hkv;
  const ReqPlan pl = dp.plan[r];
  const int L = pl.L;
  const int b = dp.budgets[r * Hkv + h];
  const int k = b < L ? b : L;
  const int64_t seg = pl.seg_off + (int64_t)h * L;
  const int64_t koff = dp.kept_off[r * Hkv + h];
  const int hw = dp.pool_window / 2;
  // the host rejects segments past kSelectRegKeys, and past the LDS with wider windows
  if (!kLong && L <= kSelectLdsKeys)
    lrfu_lds(L, k, hw, top_p, decay, scores + seg, pooled ? pooled + seg : nullptr, ks + seg,
             hit ? hit + seg : nullptr, kept + koff, ks_kept + koff, lds_keys, hist64, scan_tmp,
             mm_tmp, &s_bin, &s_above32, &s_above64);
  else if (kLong && L > kSelectLdsKeys && L <= kSelectRegKeys && hw <= kPoolHalo)
    lrfu_regs(L, k, hw, top_p, decay, scores + seg, pooled ? pooled + seg : nullptr, ks + seg,
              hit ? hit + seg : nullptr, kept + koff, ks_kept + koff, lds_keys, hist64,
              scan_tmp, mm_tmp, &s_bin, &s_above32, &s_above64);
}

hipError_t launch_lrfu_select(const DevProblem& dp, const HostPlan& hp, const float* scores,
                              float top_p, float decay, float* ks, uint8_t* hit, float* pooled,
                              int32_t* kept, float* ks_kept, hipStream_t s) {
  if (hp.R == 0) return hipSuccess;
  const int64_t keys = hp.max_L < kSelectLdsKeys ? hp.max_L : kSelectLdsKeys;
  const size_t lds = (size_t)(keys + kLdsPad) * sizeof(uint32_t);
  const bool any_long = hp.max_L > kSelectLdsKeys;
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void*)lrfu_select_kernel<false>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e == hipSuccess && any_long)
      e = hipFuncSetAttribute((const void*)lrfu_select_kernel<true>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(lrfu_select_kernel<false>, dim3(hp.Hkv, hp.R), dim3(kSelectThreads), lds, s,
                     dp, scores, top_p, decay, ks, hit, pooled, kept, ks_kept);
  if (any_long)
    hipLaunchKernelGGL(lrfu_select_kernel<true>, dim3(hp.Hkv, hp.R), dim3(kSelectThreads), lds,
                       s, dp, scores, top_p, decay, ks, hit, pooled, kept, ks_kept);
  return hipGetLastError();
}

hipError_t launch_select_range(const DevProblem& dp, const HostPlan& hp, int r0, int r1,
                               const float* scores, float* pooled, int32_t* kept,
                               hipStream_t s) {
  if (r0 >= r1) return hipSuccess;
  const int64_t keys = hp.max_L < kSelectLdsKeys ? hp.max_L : kSelectLdsKeys;
  const size_t lds = (size_t)(keys + kLdsPad) * sizeof(uint32_t);
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void*)select_kernel,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(select_kernel, dim3(hp.Hkv, r1 - r0), dim3(kSelectThreads), lds, s, dp, r0,
                     scores, pooled, kept);
  return hipGetLastError();
}

hipError_t launch_select(const DevProblem& dp, const HostPlan& hp, const float* scores,
                         float* pooled, int32_t* kept, hipStream_t s) {
  return launch_select_range(dp, hp, 0, hp.R, scores, pooled, kept, s);
}

int select_compact_splits(const HostPlan& hp, int head_dim) {
  const int64_t segs = (int64_t)hp.R * hp.Hkv;
  if (segs <= 0 || hp.max_L > kSplitMaxKeys || hp.num_kept * 4 * head_dim > kSplitMaxBytes)
    return 1;
  int64_t s = kSplitTargetGroups / segs;
  const int64_t by_slots = (hp.max_k + kSplitMinSlots - 1) / kSplitMinSlots;
  s = s < by_slots ? s : by_slots;
  s = s < kMaxSplits ? s : kMaxSplits;
  return s < 1 ? 1 : (int)s;
}

hipError_t launch_select_compact(const DevProblem& dp, const HostPlan& hp, const float* scores,
                                 float* pooled, int32_t* kept, void* kv, int32_t* bt,
                                 const int32_t* free_pages, int32_t* freed, int32_t* new_lens,
                                 hipStream_t s) {
  if (hp.R == 0) return hipSuccess;
  const int splits = select_compact_splits(hp, dp.D);
  if (splits > 1) {
    const SplitLds lay = split_lds(hp.max_L, hp.max_k, splits);
    const size_t lds = (size_t)lay.words * sizeof(uint32_t);
    if (lds + kStaticSelectLds > 160 * 1024) return hipErrorInvalidValue;   // by the limits above: never
    if (lds > 64 * 1024) {
      hipError_t e = hipFuncSetAttribute((const void*)select_compact_split_kernel,
                                         hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(select_compact_split_kernel, dim3(hp.Hkv * splits, hp.R),
                       dim3(kSelectThreads), lds, s, dp, scores, pooled, kept,
                       static_cast<uint16_t*>(kv), bt, free_pages, freed, new_lens, splits, lay);
    return hipGetLastError();
  }
  const int64_t keys = hp.max_L < kSelectLdsKeys ? hp.max_L : kSelectLdsKeys;
  size_t lds = (size_t)(keys + kLdsPad) * sizeof(uint32_t);
  if (lds < kFusedLdsBytes) lds = kFusedLdsBytes;
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void*)select_compact_kernel,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(select_compact_kernel, dim3(hp.Hkv, hp.R), dim3(kSelectThreads), lds, s,
                     dp, scores, pooled, kept, static_cast<uint16_t*>(kv), bt, free_pages, freed,
                     new_lens);
  return hipGetLastError();
}

hipError_t launch_select_side(const DevProblem& dp, const HostPlan& hp, int r0, int r1,
                              const float* scores, float* pooled, int32_t* kept,
                              hipStream_t s) {
  if (r0 >= r1) return hipSuccess;
  hipLaunchKernelGGL(select_side_kernel, dim3(hp.Hkv, r1 - r0), dim3(kSideThreads), 0, s, dp,
                     r0, scores, pooled, kept);
  return hipGetLastError();
}

}  // namespace actkv
