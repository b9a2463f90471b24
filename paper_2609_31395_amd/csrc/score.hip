// Recovery-based attention scoring over the paged K cache (Sec. 7.1, Alg. 3) and the
// log-sum-exp pass that supplies its normaliser when the caller has none.
//
// Shape of the work: per (request r, KV head h) the scores are column sums of
//   P = exp2(alpha * Q_h K_h^T - beta),  alpha = sm_scale * log2(e),  beta = LSE * log2(e)
// where Q_h holds the M = G * n action-query rows of the head group and K_h the L cached
// keys.  Q_h K_h^T is a real dense contraction (M x L x D) and runs on bf16 MFMA
// (v_mfma_f32_32x32x16_bf16) with fp32 accumulation; the exp2 / add epilogue runs on the
// VALU.
//
// Kernel layout (score_kernel):
//   * 512 threads = 8 waves (two per SIMD, one workgroup per CU).  A workgroup holds up to
//     512 query rows ("row chunk") of one (r, h) in registers: wave w owns row tiles w and
//     w+8 (32 rows each) as the MFMA A operand, and the beta of its rows.  Two waves per
//     SIMD let one wave's exp2 / add epilogue overlap the other's MFMAs.
//   * Keys stream through LDS in tiles of 64 (4 pages) gathered through the block table
//     with 16-byte loads (one 256-byte K row per 16 lanes), double-buffered: the global
//     loads of tile i+1 are in flight while tile i is multiplied.
//   * Each lane's accumulator column is one key, its 16 registers 16 query rows, so the
//     sum over rows is in-lane; lanes l and l+32 are combined with one exchange and the
//     eight waves through LDS in a fixed order (no atomics: deterministic, and independent
//     of where the pages physically live).
//   * The grid is persistent: the (segment, key tile) work list is cut into equal-cost
//     contiguous ranges (cost = key tiles x row tiles), one per workgroup, so ragged
//     lengths and query counts stay balanced and Q is loaded once per segment per
//     workgroup.
#include "device_common.hpp"

namespace actkv {

namespace {

// Scoring: 4 waves per workgroup, 4 row tiles (128 query rows) per wave, two workgroups per
// CU.  The two waves sharing a SIMD belong to different workgroups, so their barriers are
// independent and one wave's exp2 epilogue runs beside the other's MFMAs.
constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kTilesPerWave = kRowsPerChunk / 32 / kWaves;   // 4 row tiles of 32 rows
constexpr int kStages = 3;      // K tiles resident in LDS (two in flight)
// The LSE pass keeps 8 waves x 2 row tiles (its per-row running max/sum stay in registers).
constexpr int kLseThreads = 512;
constexpr int kLseWaves = kLseThreads / 64;
constexpr int kLseTilesPerWave = kRowsPerChunk / 32 / kLseWaves;

// Geometry of one K tile (kKeyTile keys of one KV head) in LDS.  Rows are not padded;
// instead the 16-byte chunk c of row r sits in slot c ^ (r % kChunks), which keeps both
// the direct-to-LDS loads (64 lanes write one contiguous KiB) and the MFMA operand reads
// (lanes l and l+1 read rows r, r+1 at the same logical chunk) free of bank conflicts.
template <int D, int W = kWaves>
struct TileGeom {
  static constexpr int kSteps = D / 16;                  // MFMA k-steps per row
  static constexpr int kRowBytes = D * 2;
  static constexpr int kChunks = D / 8;                  // 16-byte chunks per row
  static constexpr int kTileBytes = kKeyTile * kRowBytes;
  static constexpr int kWaveLoads = kTileBytes / 1024;   // one KiB per wave-wide load
  static constexpr int kLoadsPerWave = kWaveLoads / W;   // W waves share a tile's loads
  static constexpr int kRowsPerLoad = 1024 / kRowBytes;
  static_assert(kWaveLoads % W == 0, "tile must split evenly over the waves");
};

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}
__device__ __forceinline__ void wait_lgkmcnt0() { __builtin_amdgcn_s_waitcnt(0xC07F); }

// This wave's share of K tile `tile` (keys 64*tile ..) of request row bt_row, head h,
// fetched straight into LDS buffer `dst` with 16-byte loads.  Each wave-wide load covers
// kRowsPerLoad consecutive keys inside one page, so the page id is wave-uniform and comes
// from a scalar load (a vector load here would force a wait on the whole DMA queue).
// Keys past L read slots of the request's last page (their results are discarded); a page
// outside the pool is never dereferenced.
typedef __attribute__((address_space(3))) char lds_char;

// One wave-wide 16-byte-per-lane load from global memory straight into LDS at byte
// address lds_addr + 16 * lane (global_load_lds_dwordx4; the LDS base travels in M0, which
// is saved and restored around it).  Issued from inline assembly so that the compiler does
// not add its own wait on the whole vector-memory queue before later LDS reads: the
// pipeline below orders these loads itself (s_waitcnt vmcnt + barrier).
__device__ __forceinline__ void dma_to_lds16(const void* src, uint32_t lds_addr) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %2\n\t"
      "global_load_lds_dwordx4 %1, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(src), "s"(lds_addr)
      : "memory");
}

// Per-lane part of this wave's K-tile loads: wave-load u of wave w covers rows
// (w*kLoadsPerWave + u) * kRowsPerLoad .. of a tile, always the same slots of a page and the
// same (swizzled) 16-byte chunk, so the byte offset inside a page is fixed per segment.
template <int D, int W>
struct KLoadPlan {
  uint32_t lane_off[TileGeom<D, W>::kLoadsPerWave];   // bytes from the page base (K plane)
  int wl0;                                             // first wave-load index of this wave
};

template <int D, int W>
__device__ __forceinline__ KLoadPlan<D, W> make_k_load_plan(int h, int Hkv) {
  using Gm = TileGeom<D, W>;
  KLoadPlan<D, W> kp;
  const int lane = threadIdx.x & 63;
  kp.wl0 = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6) * Gm::kLoadsPerWave;
#pragma unroll
  for (int u = 0; u < Gm::kLoadsPerWave; ++u) {
    const int wl = kp.wl0 + u;
    const int row = wl * Gm::kRowsPerLoad + lane / Gm::kChunks;
    const int chunk = (lane % Gm::kChunks) ^ (row % Gm::kChunks);
    const int slot = (wl * Gm::kRowsPerLoad) % kPageSize + lane / Gm::kChunks;
    kp.lane_off[u] = (uint32_t)(((slot * Hkv + h) * D + chunk * 8) * 2);
  }
  return kp;
}

// Every wave-wide load of one wave within a K tile falls in the same page: the tile's keys
// 64*tile .. are split over the waves in runs of kRowsPerLoad * kLoadsPerWave = 16 keys
// (64 keys over 4 waves, or over 8 waves with two loads per page).  page_of() is the
// wave-uniform page id of that run (keys past L map to the request's last page); it is
// fetched a tile ahead so that the scalar load never stalls the DMA issue.
template <int D, int W>
__device__ __forceinline__ int64_t page_of(const int32_t* __restrict__ bt_row, int L,
                                           int64_t num_pages, const KLoadPlan<D, W>& kp,
                                           int64_t tile) {
  using Gm = TileGeom<D, W>;
  const int64_t kbase = tile * kKeyTile + kp.wl0 * Gm::kRowsPerLoad;   // wave-uniform
  int64_t page = bt_row[(kbase < L ? kbase : L - 1) / kPageSize];
  if (page < 0 || page >= num_pages) page = 0;   // never dereference outside the pool
  return page;
}

// This wave's share of a K tile whose keys live in page `page`, fetched straight into the
// LDS buffer at byte address `dst`.  Keys past L read slots of the request's last page
// (their results are discarded).
template <int D, int W>
__device__ __forceinline__ void issue_k_tile(uint32_t dst, const char* __restrict__ kv_bytes,
                                             int64_t page, int64_t page_bytes,
                                             const KLoadPlan<D, W>& kp) {
  using Gm = TileGeom<D, W>;
  static_assert(Gm::kRowsPerLoad * Gm::kLoadsPerWave <= kPageSize &&
                    kPageSize % (Gm::kRowsPerLoad * Gm::kLoadsPerWave) == 0,
                "a wave's loads of one tile must stay inside one page");
  const char* base = kv_bytes + page * page_bytes;
#pragma unroll
  for (int u = 0; u < Gm::kLoadsPerWave; ++u)
    dma_to_lds16(base + kp.lane_off[u], dst + (uint32_t)((kp.wl0 + u) * 1024));
}

// The 32x32 MFMA operand of key sub-tile `sub` (32 keys) for every k-step: lane l holds key
// sub*32 + l%32, head-dim elements 16*ks + 8*(l/32) .. +8.
template <int D>
__device__ __forceinline__ void read_k_operand(bf16x8 (&kreg)[TileGeom<D>::kSteps],
                                               const char* buf, int sub) {
  using Gm = TileGeom<D>;
  const int lane = threadIdx.x & 63;
  const int row = sub * 32 + (lane & 31);
  const char* base = buf + row * Gm::kRowBytes;
#pragma unroll
  for (int ks = 0; ks < Gm::kSteps; ++ks) {
    const int slot = (2 * ks + (lane >> 5)) ^ (row % Gm::kChunks);
    kreg[ks] = as_bf16x8(*reinterpret_cast<const u32x4*>(base + slot * 16));
  }
}

// Query rows of tile `tile` of chunk c as the MFMA A (or B) operand: lane l holds row
// l%32 with head-dim elements 16*ks + 8*(l/32) .. +8; rows past n are zero.
template <int D>
__device__ __forceinline__ void load_q_tile(bf16x8 (&qr)[TileGeom<D>::kSteps],
                                            const uint16_t* __restrict__ q, int G, int Hq,
                                            int h, int q_off, int n, int c, int tile) {
  const int lane = threadIdx.x & 63;
  int j, g;
  row_to_query(G, c, tile, lane & 31, &j, &g);
  if (j < n) {
    const uint16_t* src = q + ((int64_t)(q_off + j) * Hq + h * G + g) * D + (lane >> 5) * 8;
#pragma unroll
    for (int ks = 0; ks < TileGeom<D>::kSteps; ++ks)
      qr[ks] = as_bf16x8(*reinterpret_cast<const u32x4*>(src + ks * 16));
  } else {
#pragma unroll
    for (int ks = 0; ks < TileGeom<D>::kSteps; ++ks) qr[ks] = as_bf16x8(u32x4{0u, 0u, 0u, 0u});
  }
}

__device__ __forceinline__ void decode_segment(int64_t s, int C, int Hkv, int* r, int* c, int* h) {
  *h = (int)(s % Hkv);
  const int64_t rc = s / Hkv;
  *c = (int)(rc % C);
  *r = (int)(rc / C);
}

__device__ __forceinline__ int chunk_row_tiles(int M, int c) {
  const int rows = M - c * kRowsPerChunk;
  return rows <= 0 ? 1 : ceil_div(rows < kRowsPerChunk ? rows : kRowsPerChunk, 32);
}


}  // namespace

// Everything the key sweep of one segment needs besides the register-resident Q.
struct SweepCtx {
  const char* kv_bytes;
  const int32_t* bt_row;
  const float* beta_s;     // LDS: log2(e) * LSE of every row of the chunk (+inf = padding)
  const int32_t* pos_s;    // LDS: causal position of every row of the chunk
  float* out;              // scores (or chunk partials) of this (request, KV head)
  int64_t page_bytes, num_pages;
  int64_t i0, i1;          // key tiles of this workgroup
  int L, mask_from, G;
  float alpha, out_scale;
  uint32_t kl;             // LDS byte address of the K stages
};

// One K tile (64 keys, LDS buffer `buf`) against this wave's TPW row tiles: for each
// 32-key half, the MFMA chain of a row tile, its exp2 epilogue and its row sum, one row
// tile at a time; the per-key sums of the wave go to `rd`.
template <int D, bool kMaxMean, int TPW, bool kMask>
__device__ __forceinline__ void score_tile(const SweepCtx& cx,
                                           const bf16x8 (&qreg)[kTilesPerWave][TileGeom<D>::kSteps],
                                           const char* buf, int64_t key0, float* rd) {
  using Gm = TileGeom<D>;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, hf = lane >> 5, l32 = lane & 31;
#pragma unroll
  for (int sub = 0; sub < 2; ++sub) {
    bf16x8 kr[Gm::kSteps];
    read_k_operand<D>(kr, buf, sub);
    const int key = (int)(key0 + sub * 32 + l32);
    float a0 = 0.f, a1 = 0.f;
#pragma unroll
    for (int ti = 0; ti < TPW; ++ti) {
      f32x16 e = mfma32(qreg[ti][0], kr[0], f32x16{});
#pragma unroll
      for (int ks = 1; ks < Gm::kSteps; ++ks) e = mfma32(qreg[ti][ks], kr[ks], e);
      // beta of this lane's 16 rows: rows 8*aa + 4*hf + i of row tile w + kWaves*ti
      const float* brow = cx.beta_s + (w + kWaves * ti) * 32 + 4 * hf;
      const int32_t* prow = cx.pos_s + (w + kWaves * ti) * 32 + 4 * hf;
#pragma unroll
      for (int aa = 0; aa < 4; ++aa) {
        const float4 b4 = *reinterpret_cast<const float4*>(brow + 8 * aa);
        float x0 = __builtin_fmaf(e[4 * aa + 0], cx.alpha, -b4.x);
        float x1 = __builtin_fmaf(e[4 * aa + 1], cx.alpha, -b4.y);
        float x2 = __builtin_fmaf(e[4 * aa + 2], cx.alpha, -b4.z);
        float x3 = __builtin_fmaf(e[4 * aa + 3], cx.alpha, -b4.w);
        if (kMask) {   // exp2(-inf) = 0 for keys after the row's position
          const int4 p4 = *reinterpret_cast<const int4*>(prow + 8 * aa);
          const float ninf = -__builtin_inff();
          x0 = key > p4.x ? ninf : x0;
          x1 = key > p4.y ? ninf : x1;
          x2 = key > p4.z ? ninf : x2;
          x3 = key > p4.w ? ninf : x3;
        }
        e[4 * aa + 0] = fast_exp2(x0);
        e[4 * aa + 1] = fast_exp2(x1);
        e[4 * aa + 2] = fast_exp2(x2);
        e[4 * aa + 3] = fast_exp2(x3);
      }
      if (!kMaxMean) {
#pragma unroll
        for (int v = 0; v < 16; v += 2) { a0 += e[v]; a1 += e[v + 1]; }
      } else if (cx.G == 16) {
        // the lane's 16 rows are one query's whole group
        float mx = e[0];
#pragma unroll
        for (int v = 1; v < 16; ++v) mx = fmaxf(mx, e[v]);
        a0 += mx;
      } else if (cx.G == 8) {
        // registers 0-7 and 8-15 are two queries' groups
        float m0 = e[0], m1 = e[8];
#pragma unroll
        for (int v = 1; v < 8; ++v) { m0 = fmaxf(m0, e[v]); m1 = fmaxf(m1, e[8 + v]); }
        a0 += m0; a1 += m1;
      } else {
        // registers v0..v0+3 are four consecutive rows of the natural order
#pragma unroll
        for (int v0 = 0; v0 < 16; v0 += 4) {
          if (cx.G == 4) {
            a0 += fmaxf(fmaxf(e[v0], e[v0 + 1]), fmaxf(e[v0 + 2], e[v0 + 3]));
          } else if (cx.G == 2) {
            a0 += fmaxf(e[v0], e[v0 + 1]);
            a1 += fmaxf(e[v0 + 2], e[v0 + 3]);
          } else {
            a0 += e[v0] + e[v0 + 2];
            a1 += e[v0 + 1] + e[v0 + 3];
          }
        }
      }
      // one row tile's accumulator at a time: keeps the wave within 256 registers (the
      // other workgroup's wave on this SIMD supplies the MFMA / VALU overlap)
      __builtin_amdgcn_sched_barrier(0);
    }
    float acc = a0 + a1;
    acc += __shfl_xor(acc, 32, 64);   // lanes l and l+32 hold the same key
    if (hf == 0) rd[sub * 32 + l32] = acc;
    __builtin_amdgcn_sched_barrier(0);
  }
}

// Sweep key tiles i0 .. i1-1 of one segment with TPW row tiles (of 32 rows) per wave:
// kStages-1 tiles in flight through the direct-to-LDS pipeline and one barrier per tile.
template <int D, bool kMaxMean, int TPW>
__device__ __forceinline__ void score_sweep(const SweepCtx& cx, const KLoadPlan<D, kWaves>& kp,
                                            const bf16x8 (&qreg)[kTilesPerWave][TileGeom<D>::kSteps],
                                            char (*kbuf)[TileGeom<D>::kTileBytes],
                                            float (*red)[kWaves][kKeyTile]) {
  using Gm = TileGeom<D>;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  auto clamp_tile = [&](int64_t t) { return t < cx.i1 ? t : cx.i1 - 1; };
#pragma unroll
  for (int p = 0; p < kStages - 1; ++p)
    issue_k_tile<D, kWaves>(cx.kl + p * Gm::kTileBytes, cx.kv_bytes,
                            page_of<D, kWaves>(cx.bt_row, cx.L, cx.num_pages, kp, clamp_tile(cx.i0 + p)),
                            cx.page_bytes, kp);
  int64_t next_page = page_of<D, kWaves>(cx.bt_row, cx.L, cx.num_pages, kp,
                                         clamp_tile(cx.i0 + kStages - 1));
  for (int64_t i = cx.i0; i < cx.i1; ++i) {
    const int st = (int)((i - cx.i0) % kStages);
    // tile i has landed once at most the later tiles' loads are outstanding; the barrier
    // also retires every wave's reads of the stage the next load overwrites
    wait_vmcnt<(kStages - 2) * Gm::kLoadsPerWave>();
    __builtin_amdgcn_s_barrier();
    issue_k_tile<D, kWaves>(cx.kl + ((st + kStages - 1) % kStages) * Gm::kTileBytes, cx.kv_bytes,
                            next_page, cx.page_bytes, kp);
    next_page = page_of<D, kWaves>(cx.bt_row, cx.L, cx.num_pages, kp, clamp_tile(i + kStages));
    const int64_t key0 = i * kKeyTile;
    float* rd = red[i & 1][w];
    // tiles that reach past the first action position may hold keys hidden from some rows;
    // they take a separate, masked copy of the body so that the common body has no branch
    // (a branch per row tile would keep all of a tile's exp2 results live at once)
    if (key0 + kKeyTile - 1 > cx.mask_from)
      score_tile<D, kMaxMean, TPW, true>(cx, qreg, kbuf[st], key0, rd);
    else
      score_tile<D, kMaxMean, TPW, false>(cx, qreg, kbuf[st], key0, rd);
    wait_lgkmcnt0();
    __builtin_amdgcn_s_barrier();
    // wave w finishes keys 16w .. 16w+15 of tile i (fixed summation order over waves)
    if (lane < kKeyTile / kWaves) {
      const int kk = w * (kKeyTile / kWaves) + lane;
      const int64_t key = key0 + kk;
      if (key < cx.L) {
        float v = 0.f;
#pragma unroll
        for (int ww = 0; ww < kWaves; ++ww) v += red[i & 1][ww][kk];
        cx.out[key] = v * cx.out_scale;
      }
    }
  }
}

template <int D, bool kMaxMean>
__global__ __launch_bounds__(kThreads, 2) void score_kernel(
    DevProblem dp, const uint16_t* __restrict__ q_ptr, const uint16_t* __restrict__ kv_ptr,
    const int32_t* __restrict__ bt_ptr, const float* __restrict__ lse_ptr,
    float* __restrict__ scores_ptr, float* __restrict__ part_ptr, int64_t num_scores) {
  using Gm = TileGeom<D>;
  __shared__ __align__(1024) char kbuf[kStages][Gm::kTileBytes];
  __shared__ __align__(16) float beta_s[kRowsPerChunk];
  __shared__ __align__(16) int32_t pos_s[kRowsPerChunk];
  __shared__ float red[2][kWaves][kKeyTile];

  const int tid = threadIdx.x, w = tid >> 6;
  const int G = dp.G, Hq = dp.Hq, Hkv = dp.Hkv, C = dp.max_chunks;
  const int64_t nseg = dp.num_segments;
  const int64_t total = dp.seg_cost[nseg];
  const int64_t c0 = total * blockIdx.x / gridDim.x, c1 = total * (blockIdx.x + 1) / gridDim.x;
  if (c0 >= c1) return;

  SweepCtx cx;
  cx.kv_bytes = reinterpret_cast<const char*>(kv_ptr);
  cx.beta_s = beta_s;
  cx.pos_s = pos_s;
  cx.page_bytes = (int64_t)kPageSize * Hkv * D * 2;
  cx.num_pages = dp.num_pages;
  cx.G = G;
  cx.alpha = dp.sm_scale * kLog2e;
  cx.kl = (uint32_t)(uintptr_t)(lds_char*)&kbuf[0][0];

  // first segment: the largest s with seg_cost[s] <= c0 (it is never empty)
  int64_t lo = 0, hi = nseg;
  while (lo < hi) {
    const int64_t mid = (lo + hi + 1) / 2;
    if (dp.seg_cost[mid] <= c0) lo = mid; else hi = mid - 1;
  }
  bool first = true;
  for (int64_t s = lo; s < nseg; ++s) {
    const int64_t cs = dp.seg_cost[s], ce = dp.seg_cost[s + 1];
    if (cs >= c1) break;
    if (ce == cs) continue;
    int r, c, h;
    decode_segment(s, C, Hkv, &r, &c, &h);
    const ReqPlan pl = dp.plan[r];
    const int L = pl.L, n = pl.n, M = G * n;
    const int RT = chunk_row_tiles(M, c);
    const int64_t ntiles = ceil_div64(L, kKeyTile);
    cx.i0 = first ? (c0 - cs + RT - 1) / RT : 0;
    cx.i1 = (c1 - cs + RT - 1) / RT;
    if (cx.i1 > ntiles) cx.i1 = ntiles;
    first = false;
    if (cx.i0 >= cx.i1) continue;

    // ---- segment setup: beta / causal position of every row, Q rows into registers
    wait_vmcnt<0>();   // no load of the previous segment may still land in a K buffer
    __syncthreads();
    for (int m = tid; m < kRowsPerChunk; m += kThreads) {
      int j, g;
      row_to_query(G, c, m / 32, m % 32, &j, &g);
      beta_s[m] = j < n ? lse_ptr[(int64_t)(pl.q_off + j) * Hq + h * G + g] * kLog2e
                        : __builtin_inff();
      pos_s[m] = dp.causal ? L - n + j : L - 1;
    }
    bf16x8 qreg[kTilesPerWave][Gm::kSteps];
#pragma unroll
    for (int ti = 0; ti < kTilesPerWave; ++ti)
      load_q_tile<D>(qreg[ti], q_ptr, G, Hq, h, pl.q_off, n, c, w + kWaves * ti);
    cx.bt_row = bt_ptr + (int64_t)r * dp.bt_stride;
    cx.L = L;
    cx.mask_from = dp.causal ? L - n : L;  // keys past this may be hidden from some rows
    cx.out_scale = (kMaxMean && pl.nchunk == 1) ? (n > 0 ? 1.0f / n : 0.0f) : 1.0f;
    cx.out = (c == 0) ? scores_ptr + pl.seg_off + (int64_t)h * L
                      : part_ptr + (int64_t)(c - 1) * num_scores + pl.seg_off + (int64_t)h * L;
    const KLoadPlan<D, kWaves> kp = make_k_load_plan<D, kWaves>(h, Hkv);
    // every ordinary load of the setup has landed before the K pipeline starts, so the
    // sweep needs no compiler-inserted wait on the vector-memory queue
    wait_vmcnt<0>();
    __syncthreads();   // beta_s / pos_s visible
    // row tiles past the chunk's RT are all padding (Q = 0, beta = +inf): each wave runs
    // only as many of its row tiles as can hold real rows
    const int tpw = (RT + kWaves - 1) / kWaves;
    if (tpw >= 4) score_sweep<D, kMaxMean, 4>(cx, kp, qreg, kbuf, red);
    else if (tpw == 3) score_sweep<D, kMaxMean, 3>(cx, kp, qreg, kbuf, red);
    else if (tpw == 2) score_sweep<D, kMaxMean, 2>(cx, kp, qreg, kbuf, red);
    else score_sweep<D, kMaxMean, 1>(cx, kp, qreg, kbuf, red);
  }
  wait_vmcnt<0>();   // drain: no LDS write may be outstanding when the workgroup exits
}

// scores = (scores + sum_{c >= 1} partial_c) * scale, for requests scored in several row
// chunks (fixed order: deterministic).
__global__ __launch_bounds__(256) void chunk_reduce_kernel(DevProblem dp, float* scores,
                                                           const float* part,
                                                           int64_t num_scores) {
  const int r = blockIdx.y, h = blockIdx.z;
  const ReqPlan pl = dp.plan[r];
  if (pl.nchunk <= 1) return;
  const float scale = dp.agg == ACTKV_AGG_MAX_MEAN ? (pl.n > 0 ? 1.0f / pl.n : 0.f) : 1.f;
  const int64_t base = pl.seg_off + (int64_t)h * pl.L;
  for (int64_t t = blockIdx.x * 256 + threadIdx.x; t < pl.L; t += (int64_t)gridDim.x * 256) {
    float v = scores[base + t];
    for (int c = 1; c < pl.nchunk; ++c) v += part[(int64_t)(c - 1) * num_scores + base + t];
    scores[base + t] = v * scale;
  }
}

hipError_t launch_score(const DevProblem& dp, const HostPlan& hp, const void* q,
                        const void* kv, const int32_t* bt, const float* lse, float* scores,
                        float* score_part, hipStream_t s) {
  if (hp.num_scores == 0) return hipSuccess;
  const uint16_t* qq = static_cast<const uint16_t*>(q);
  const uint16_t* kk = static_cast<const uint16_t*>(kv);
  int dev = 0, cus = 256;
  if (hipGetDevice(&dev) == hipSuccess) {
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) cus = 256;
  }
  int64_t grid = (int64_t)cus * 2;   // two 4-wave workgroups per CU
  if (grid > hp.score_cost) grid = hp.score_cost > 0 ? hp.score_cost : 1;
  const bool mm = dp.agg == ACTKV_AGG_MAX_MEAN;
  if (dp.D == 128) {
    if (mm) hipLaunchKernelGGL((score_kernel<128, true>), dim3(grid), dim3(kThreads), 0, s, dp, qq, kk, bt, lse, scores, score_part, hp.num_scores);
    else hipLaunchKernelGGL((score_kernel<128, false>), dim3(grid), dim3(kThreads), 0, s, dp, qq, kk, bt, lse, scores, score_part, hp.num_scores);
  } else {
    if (mm) hipLaunchKernelGGL((score_kernel<64, true>), dim3(grid), dim3(kThreads), 0, s, dp, qq, kk, bt, lse, scores, score_part, hp.num_scores);
    else hipLaunchKernelGGL((score_kernel<64, false>), dim3(grid), dim3(kThreads), 0, s, dp, qq, kk, bt, lse, scores, score_part, hp.num_scores);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (hp.max_chunks > 1) {
    hipLaunchKernelGGL(chunk_reduce_kernel, dim3(64, hp.R, hp.Hkv), dim3(256), 0, s, dp, scores,
                       score_part, hp.num_scores);
    e = hipGetLastError();
  }
  return e;
}

// ---------------------------------------------------------------------------------------
// Log-sum-exp pass (online softmax).  Here K is the MFMA A operand and Q the B operand, so
// each lane's accumulator column is one query row and its 16 registers 16 keys: the
// running (max, sum) of a row stays in-lane.  One workgroup reduces kLseKeysPerBlock keys
// of one (request, row chunk, KV head) and writes a partial (max, sum) per row; a merge
// kernel combines the partials of a row in order.
// ---------------------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(kLseThreads, 1) void lse_partial_kernel(
    DevProblem dp, const uint16_t* __restrict__ q, const uint16_t* __restrict__ kv,
    const int32_t* __restrict__ bt, float2* __restrict__ part) {
  using Gm = TileGeom<D, kLseWaves>;
  __shared__ __align__(1024) char kbuf[kStages][Gm::kTileBytes];
  const uint32_t kl = (uint32_t)(uintptr_t)(lds_char*)&kbuf[0][0];
  const int kb = blockIdx.x, ch = blockIdx.y / dp.Hkv, h = blockIdx.y % dp.Hkv, r = blockIdx.z;
  const ReqPlan pl = dp.plan[r];
  if (kb >= pl.lse_blocks || ch >= pl.nchunk) return;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, hf = lane >> 5, l32 = lane & 31;
  const int G = dp.G, Hq = dp.Hq, Hkv = dp.Hkv, L = pl.L, n = pl.n, M = G * n;
  const int RT = chunk_row_tiles(M, ch);
  const float alpha = dp.sm_scale * kLog2e;
  const int32_t* bt_row = bt + (int64_t)r * dp.bt_stride;
  const char* kv_bytes = reinterpret_cast<const char*>(kv);
  const int64_t page_bytes = (int64_t)kPageSize * Hkv * D * 2;
  const KLoadPlan<D, kLseWaves> kp = make_k_load_plan<D, kLseWaves>(h, Hkv);
  const int64_t t0 = (int64_t)kb * (kLseKeysPerBlock / kKeyTile);
  int64_t t1 = t0 + kLseKeysPerBlock / kKeyTile;
  const int64_t ntiles = ceil_div64(L, kKeyTile);
  if (t1 > ntiles) t1 = ntiles;
  bf16x8 qreg[kLseTilesPerWave][Gm::kSteps];
  int pos[kLseTilesPerWave];
  float rm[kLseTilesPerWave], rs[kLseTilesPerWave];
#pragma unroll
  for (int ti = 0; ti < kLseTilesPerWave; ++ti) {
    rm[ti] = -__builtin_inff();
    rs[ti] = 0.f;
    pos[ti] = -1;
    const int tile = w + kLseWaves * ti;
    if (tile < RT) {
      load_q_tile<D>(qreg[ti], q, G, Hq, h, pl.q_off, n, ch, tile);
      int j, g;
      row_to_query(G, ch, tile, l32, &j, &g);
      pos[ti] = j < n ? (dp.causal ? L - n + j : L - 1) : -1;
    }
  }
  wait_vmcnt<0>();   // Q is in registers before the K pipeline starts
  auto clamp_tile = [&](int64_t t) { return t < t1 ? t : t1 - 1; };
#pragma unroll
  for (int p = 0; p < kStages - 1; ++p)
    issue_k_tile<D, kLseWaves>(kl + p * Gm::kTileBytes, kv_bytes,
                               page_of<D, kLseWaves>(bt_row, L, dp.num_pages, kp, clamp_tile(t0 + p)),
                               page_bytes, kp);
  int64_t next_page = page_of<D, kLseWaves>(bt_row, L, dp.num_pages, kp, clamp_tile(t0 + kStages - 1));
  for (int64_t i = t0; i < t1; ++i) {
    const int st = (int)((i - t0) % kStages);
    wait_vmcnt<(kStages - 2) * Gm::kLoadsPerWave>();
    __builtin_amdgcn_s_barrier();
    issue_k_tile<D, kLseWaves>(kl + ((st + kStages - 1) % kStages) * Gm::kTileBytes, kv_bytes,
                               next_page, page_bytes, kp);
    next_page = page_of<D, kLseWaves>(bt_row, L, dp.num_pages, kp, clamp_tile(i + kStages));
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
      bf16x8 kreg[Gm::kSteps];
      read_k_operand<D>(kreg, kbuf[st], sub);
      const int keybase = (int)(i * kKeyTile + sub * 32 + 4 * hf);
#pragma unroll
      for (int ti = 0; ti < kLseTilesPerWave; ++ti) {
        if (w + kLseWaves * ti < RT) {
          f32x16 x = {};
#pragma unroll
          for (int ks = 0; ks < Gm::kSteps; ++ks) x = mfma32(kreg[ks], qreg[ti][ks], x);
          float mx = rm[ti];
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int key = keybase + 8 * (v / 4) + (v % 4);
            x[v] = key <= pos[ti] ? x[v] * alpha : -__builtin_inff();
            mx = fmaxf(mx, x[v]);
          }
          if (mx != -__builtin_inff()) {
            float sum = rs[ti] * fast_exp2(rm[ti] - mx);
#pragma unroll
            for (int v = 0; v < 16; ++v) sum += fast_exp2(x[v] - mx);
            rs[ti] = sum;
            rm[ti] = mx;
          }
        }
      }
    }
  }
  wait_vmcnt<0>();
  // combine the two lanes that share a query row, then write one partial per row
#pragma unroll
  for (int ti = 0; ti < kLseTilesPerWave; ++ti) {
    const int tile = w + kLseWaves * ti;
    const float om = __shfl_xor(rm[ti], 32, 64), os = __shfl_xor(rs[ti], 32, 64);
    const float m = fmaxf(rm[ti], om);
    float sm = 0.f;
    if (m != -__builtin_inff()) sm = rs[ti] * fast_exp2(rm[ti] - m) + os * fast_exp2(om - m);
    if (tile < RT && hf == 0) {
      int j, g;
      row_to_query(G, ch, tile, l32, &j, &g);
      if (j < n) {
        const int64_t row = (int64_t)j * Hq + h * G + g;
        part[pl.lse_part_off + row * pl.lse_blocks + kb] = make_float2(m, sm);
      }
    }
  }
}

__global__ __launch_bounds__(256) void lse_merge_kernel(DevProblem dp, const float2* part,
                                                        float* lse) {
  const int r = blockIdx.x;
  const ReqPlan pl = dp.plan[r];
  const int rows = pl.n * dp.Hq;
  for (int row = threadIdx.x; row < rows; row += 256) {
    const float2* pp = part + pl.lse_part_off + (int64_t)row * pl.lse_blocks;
    float m = -__builtin_inff();
    for (int b = 0; b < pl.lse_blocks; ++b) m = fmaxf(m, pp[b].x);
    float s = 0.f;
    if (m != -__builtin_inff())
      for (int b = 0; b < pl.lse_blocks; ++b) s += pp[b].y * fast_exp2(pp[b].x - m);
    // natural-log LSE = (m + log2 s) * ln 2
    lse[(int64_t)pl.q_off * dp.Hq + row] =
        m == -__builtin_inff() ? -__builtin_inff() : (m + __log2f(s)) * 0.6931471805599453f;
  }
}

hipError_t launch_lse(const DevProblem& dp, const HostPlan& hp, const void* q, const void* kv,
                      const int32_t* bt, float* lse_out, float2* lse_part, hipStream_t s) {
  if (hp.sum_n == 0 || hp.R == 0) return hipSuccess;
  const int64_t max_blocks = hp.max_lse_blocks > 0 ? hp.max_lse_blocks : 1;
  dim3 grid((unsigned)max_blocks, (unsigned)(hp.max_chunks * hp.Hkv), (unsigned)hp.R);
  if (dp.D == 128)
    hipLaunchKernelGGL(lse_partial_kernel<128>, grid, dim3(kLseThreads), 0, s, dp,
                       static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(kv), bt,
                       lse_part);
  else
    hipLaunchKernelGGL(lse_partial_kernel<64>, grid, dim3(kLseThreads), 0, s, dp,
                       static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(kv), bt,
                       lse_part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(lse_merge_kernel, dim3(hp.R), dim3(256), 0, s, dp, lse_part, lse_out);
  return hipGetLastError();
}

}  // namespace actkv
