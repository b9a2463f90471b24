// Recovery-based attention scoring over the paged K cache (Sec. 7.1, Alg. 3) and the
// log-sum-exp pass that supplies its normaliser when the caller has none.
//
// Shape of the work: per (request r, KV head h) the scores are column sums of
//   P = exp2(alpha * Q_h K_h^T - beta),  alpha = sm_scale * log2(e),  beta = LSE * log2(e)
// where Q_h holds the M = G * n action-query rows of the head group and K_h the L cached
// keys.  Q_h K_h^T is a real dense contraction (M x L x D) and runs on bf16 MFMA with fp32
// accumulation; the exp2 / add epilogue runs on the VALU.
//
// Kernel layout (score_kernel):
//   * One workgroup of 8 waves per CU (two per SIMD), persistent: the list of (segment,
//     64-key tile) work, segment = (request, row chunk of up to 512 query rows, KV head), is
//     cut into equal-cost contiguous ranges, one per workgroup, so ragged lengths and query
//     counts stay balanced and Q is loaded once per segment.
//   * Each wave holds 4 row tiles of 16 query rows in registers (v_mfma_f32_16x16x32_bf16 A
//     operand) and the beta of its rows.  K tiles (64 keys, 4 pages) are gathered through
//     the block table straight into LDS (global_load_lds_dwordx4, 16 bytes per lane,
//     chunk-swizzled rows), three tiles ahead, one barrier per tile; every wave reads each
//     16-key sub-tile as its MFMA B operand.
//   * Two waves share each SIMD.  On gfx950 a wave gains little from mixing its own MFMA
//     chains and exp2 epilogue (measured with register-only probes: 68 ns per 16x16x128
//     unit and SIMD for one wave, 50 ns for two), so the overlap of the matrix core and the
//     VALU comes from the pair: while one wave waits on its chain, an exp2 or an LDS read,
//     the other issues.
//   * A lane's accumulator column is one key and 4 query rows, so the row sum is in-lane;
//     the 4 lane groups and 8 waves are combined through LDS in a fixed order (no atomics:
//     deterministic, and independent of where the pages physically live).
#include <atomic>

#include "device_common.hpp"

namespace actkv {

namespace {

constexpr int kStages = 3;   // K tiles resident in LDS for the LSE pass
// The LSE pass keeps 8 waves x 2 row tiles (its per-row running max/sum stay in registers).
constexpr int kLseThreads = 512;
constexpr int kLseWaves = kLseThreads / 64;
constexpr int kLseTilesPerWave = kRowsPerChunk / 32 / kLseWaves;
// A tile's 16 terms against a shift below the running max are summed as they come while the
// sum stays at or under this (each term then under 2^64; a 2048-key block adds at most 64
// such sums per row, far from the fp32 range).
constexpr float kLseLazyLimit = 18446744073709551616.0f;   // 2^64

// Geometry of one K tile (kKeyTile keys of one KV head) in LDS.  Rows are not padded;
// instead the 16-byte chunk c of row r sits in slot c ^ (r % kChunks), which keeps both
// the direct-to-LDS loads (64 lanes write one contiguous KiB) and the MFMA operand reads
// (lanes l and l+1 read rows r, r+1 at the same logical chunk) free of bank conflicts.
// W is the number of waves that share a tile's loads; the row geometry does not depend on it.
template <int D, int W = 8>
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
__device__ __forceinline__ int32_t page_of(const int32_t* __restrict__ bt_row, int L,
                                           const KLoadPlan<D, W>& kp, int64_t tile) {
  using Gm = TileGeom<D, W>;
  const int64_t kbase = tile * kKeyTile + kp.wl0 * Gm::kRowsPerLoad;   // wave-uniform
  return bt_row[(kbase < L ? kbase : L - 1) / kPageSize];
}

// This wave's share of a K tile whose keys live in page `page`, fetched straight into the
// LDS buffer at byte address `dst`.  Keys past L read slots of the request's last page
// (their results are discarded).
template <int D, int W>
__device__ __forceinline__ void issue_k_tile(uint32_t dst, const char* __restrict__ kv_bytes,
                                             int32_t page_entry, int64_t num_pages,
                                             int64_t page_bytes, const KLoadPlan<D, W>& kp) {
  using Gm = TileGeom<D, W>;
  static_assert(Gm::kRowsPerLoad * Gm::kLoadsPerWave <= kPageSize &&
                    kPageSize % (Gm::kRowsPerLoad * Gm::kLoadsPerWave) == 0,
                "a wave's loads of one tile must stay inside one page");
  // never dereference outside the pool (checked here, where the entry is used, so that the
  // scalar load that fetched it is not waited for a tile early)
  const int64_t page = (page_entry < 0 || page_entry >= num_pages) ? 0 : page_entry;
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

// ---- scoring: 16x16x32 MFMA units on two waves per SIMD --------------------------------
//
// A wave owns 4 row tiles of 16 query rows (the MFMA A operand, held in registers for the
// whole segment).  Each 64-key tile in LDS is cut into 4 sub-tiles of 16 keys (the B
// operand).  A "unit" is one (sub-tile, row tile) pair: kSteps dependent MFMAs into a 16x16
// accumulator -- lane l holds key l%16 and rows 4*(l/16) .. +3 -- and then its epilogue:
// exp2 of the 4 elements, summed (or max-reduced over the GQA group) into the lane's
// partial for that key.

constexpr int kRowTile = 16;
constexpr int kSubTiles = kKeyTile / 16;   // 4
static_assert(kSubTiles == 4, "unit bookkeeping below");

template <int D>
struct Geom16 {
  static constexpr int kSteps = D / 32;   // k-steps of 32 per head
};

// LDS offset of this lane's B-operand chunk for k-step ks of sub-tile 0 (sub-tile s is
// 16 rows further).  Row r = l%16 holds chunk c = 4 ks + l/16 at slot c ^ (r % kChunks):
//   r * kRowBytes + 16 ((4 ks + q) ^ x)  =  [r * kRowBytes + 16 (q ^ (x & 3))] + [(64 ks) ^ (16 (x & ~3))]
// with q = l/16, x = r % kChunks: two per-lane values give every k-step.
struct KRead16 {
  uint32_t base, xmask;
};

template <int D>
__device__ __forceinline__ KRead16 make_k_read16() {
  using Gm = TileGeom<D>;
  const int lane = threadIdx.x & 63, r = lane & 15, qd = lane >> 4, x = r % Gm::kChunks;
  KRead16 rp;
  rp.base = (uint32_t)(r * Gm::kRowBytes + 16 * (qd ^ (x & 3)));
  rp.xmask = (uint32_t)(16 * (x & ~3));
  return rp;
}

template <int D>
__device__ __forceinline__ bf16x8 lds_k16(const char* tile_buf, int sub, const KRead16& rp, int ks) {
  const uint32_t off = rp.base + ((uint32_t)(64 * ks) ^ rp.xmask);
  return as_bf16x8(*reinterpret_cast<const u32x4*>(tile_buf + sub * 16 * TileGeom<D>::kRowBytes + off));
}

__device__ __forceinline__ float dpp_xor1(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));
}
__device__ __forceinline__ float dpp_xor2(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false));
}


// The sweep.  Per tile: page ids prefetched a tile ahead (scalar), a wait for the tile's
// direct-to-LDS loads, one barrier, the loads of the tile three ahead, the finish of the
// previous tile, then 4 sub-tiles x NRT units.  A unit's exp2 epilogue runs after the next
// unit's MFMA chain (lag one), and a tile's last unit is finished before the next barrier.
// Each wave reads every K sub-tile from LDS: twice the LDS reads of four waves of 128 rows,
// which measured faster anyway (one wave per SIMD leaves the SIMD idle whenever it waits).
namespace {

constexpr int k2wThreads = 512;
constexpr int k2wWaves = k2wThreads / 64;
constexpr int k2wRowTiles = kRowsPerChunk / kRowTile / k2wWaves;   // 4
static_assert(k2wRowTiles == 4, "row-tile bookkeeping below");
static_assert(k2wWaves * kRowTile == kScoreRowStep, "the scoring cost counts rows in these steps");
constexpr int k2wStages = 4;   // K tiles in LDS (three in flight)
constexpr int k2wRedBufs = 2;  // per-key partials of a tile are read one tile later
// Per-key partials of one tile: wave w, lane group g = l/16, key k at
// red[w * k2wRedRow + g * k2wRedGrp + k]; the strides keep the writes (64 lanes) and the
// finishing reads (8 source waves x 4 keys per half-wave) on distinct banks.
constexpr int k2wRedGrp = kKeyTile + 16;          // 80 floats
constexpr int k2wRedRow = 4 * k2wRedGrp + 4;      // 324 floats
constexpr int k2wRedTile = k2wWaves * k2wRedRow;  // floats per buffer

// Query row at (row tile T = w + 8 * rt, tile row mm) of row chunk c: the natural order
// m = j * G + g, unless the group max of MAX_MEAN needs a query's G = 8 or 16 heads in one
// lane: then they sit at the same lane position of 2 or 4 consecutive row tiles of a wave.
__device__ __forceinline__ void row_query_2w(int G, bool grouped, int c, int T, int mm, int* j,
                                             int* g) {
  if (!grouped) {
    const int m = c * kRowsPerChunk + T * kRowTile + mm;
    *j = m / G;
    *g = m % G;
    return;
  }
  const int w = T % k2wWaves, rt = T / k2wWaves, a = mm >> 2, i = mm & 3;
  if (G == 8) {
    *j = c * (kRowsPerChunk / 8) + (rt >> 1) * (4 * k2wWaves) + w * 4 + a;
    *g = 4 * (rt & 1) + i;
  } else {
    *j = c * (kRowsPerChunk / 16) + w * 4 + a;
    *g = 4 * (rt & 3) + i;
  }
}

// Row tiles per wave that can hold real rows of chunk c (the same for every wave).
__device__ __forceinline__ int wave_tiles_2w(int G, bool grouped, int n, int c) {
  if (!grouped) {
    const int rows = G * n - c * kRowsPerChunk;
    if (rows <= 0) return 1;
    const int r = rows < kRowsPerChunk ? rows : kRowsPerChunk;
    return ceil_div(r, kRowTile * k2wWaves);
  }
  const int per = G / 4, qn = n - c * (kRowsPerChunk / G);
  const int groups = qn <= 0 ? 1 : ceil_div(qn, 4 * k2wWaves);
  const int t = groups * per;
  return t < k2wRowTiles ? t : k2wRowTiles;
}

// Row tile T of chunk c as the 16x16x32 A operand: lane l holds row l%16 with head-dim
// elements 32*ks + 8*(l/16) .. +8; rows past n are zero.
template <int D>
__device__ __forceinline__ void load_q16(bf16x8 (&qr)[Geom16<D>::kSteps],
                                         const uint16_t* __restrict__ q, int G, bool grouped,
                                         int Hq, int h, int q_off, int n, int c, int T) {
  const int lane = threadIdx.x & 63;
  int j, g;
  row_query_2w(G, grouped, c, T, lane & 15, &j, &g);
  if (j < n) {
    const uint16_t* src = q + ((int64_t)(q_off + j) * Hq + h * G + g) * D + (lane >> 4) * 8;
#pragma unroll
    for (int ks = 0; ks < Geom16<D>::kSteps; ++ks)
      qr[ks] = as_bf16x8(*reinterpret_cast<const u32x4*>(src + ks * 32));
  } else {
#pragma unroll
    for (int ks = 0; ks < Geom16<D>::kSteps; ++ks) qr[ks] = as_bf16x8(u32x4{0u, 0u, 0u, 0u});
  }
}

struct Ctx2w {
  const char* kv_bytes;
  const int32_t* bt_row;
  const int32_t* pos_s;    // LDS: causal position of every row of the chunk
  __amdgpu_buffer_rsrc_t out;   // scores (or chunk partials) of this (request, KV head)
  const char* kbuf;        // LDS: the K stages
  float* red;              // LDS: k2wRedBufs partial tiles
  int64_t page_bytes, num_pages;
  int i0, i1;              // key tiles of this workgroup
  int L, mask_from, G;
  float alpha, out_scale;
  uint32_t kl;             // LDS byte address of the K stages
};

// The finish of tile t: the 32 partials of every key (8 waves x 4 lane groups) summed in a
// fixed order and stored.  Wave w finishes keys 8w .. 8w+7: lane l takes key 8w + l/8 and
// the 4 partials of source wave l%8, then the 8 lanes of a key are added pairwise (xor 1,
// xor 2, then lane 4 of each group of 8 takes the other half by a row shift of 4).  Every
// lane takes part in one buffer store (lanes with nothing to write store past the end).
__device__ __forceinline__ void finish_2w(const Ctx2w& cx, int t, bool valid) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int kk = w * (kKeyTile / k2wWaves) + (lane >> 3), ww = lane & 7;
  const float* rr = cx.red + (t & (k2wRedBufs - 1)) * k2wRedTile + ww * k2wRedRow + kk;
  float v = (rr[0] + rr[k2wRedGrp]) + (rr[2 * k2wRedGrp] + rr[3 * k2wRedGrp]);
  v += dpp_xor1(v);
  v += dpp_xor2(v);
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x114, 0xF, 0xF, false));
  const int key = t * kKeyTile + kk;
  const uint32_t off = (valid && ww == 4 && key < cx.L) ? (uint32_t)key * 4u : 0x7FFFFFF0u;
  __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v * cx.out_scale), cx.out, off, 0, 0);
}

// Per-wave epilogue state.
struct Epi2w {
  float part[4];   // the lane's partials of the current sub-tile (independent add chains)
  float ex;        // SUM: the last exp2, added one element later
  float mx;        // MAX_MEAN, G = 8 / 16: running group max over the row tiles of a query
};

// Epilogue of one unit: accumulator c of row tile rt (beta bt), keys of sub-tile at `key`.
template <bool kMaxMean, bool kMask>
__device__ __forceinline__ void epilogue_2w(Epi2w& e, f32x4 c, int rt, const float (&bt)[4],
                                            const int32_t* prow, int key, float alpha, int G) {
  int pt[4] = {0, 0, 0, 0};
  if (kMask) {
    const int4 p4 = *reinterpret_cast<const int4*>(prow);
    pt[0] = p4.x; pt[1] = p4.y; pt[2] = p4.z; pt[3] = p4.w;
  }
  float p[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    float x = __builtin_fmaf(c[v], alpha, -bt[v]);
    if (kMask) x = key > pt[v] ? -__builtin_inff() : x;   // exp2(-inf) = 0
    if (!kMaxMean) {
      e.part[(v + 3) & 3] += e.ex;   // the previous exp2, off the latency path
      e.ex = fast_exp2(x);
    } else {
      p[v] = fast_exp2(x);
    }
  }
  if (kMaxMean) {
    const float m01 = fmaxf(p[0], p[1]), m23 = fmaxf(p[2], p[3]);
    if (G == 1) {
      e.part[0] += (p[0] + p[1]) + (p[2] + p[3]);
    } else if (G == 2) {
      e.part[0] += m01 + m23;
    } else if (G == 4) {
      e.part[0] += fmaxf(m01, m23);
    } else if (G == 8) {
      const float m = fmaxf(m01, m23);
      if (rt & 1) e.part[0] += fmaxf(e.mx, m); else e.mx = m;
    } else {
      const float m = fmaxf(m01, m23);
      e.mx = (rt & 3) == 0 ? m : fmaxf(e.mx, m);
      if ((rt & 3) == 3) e.part[0] += e.mx;
    }
  }
}

// The lane's partial of sub-tile s of tile t goes to LDS; the partials restart.
__device__ __forceinline__ void put_partial_2w(const Ctx2w& cx, Epi2w& e, int t, int s) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  e.part[3] += e.ex;
  e.ex = 0.f;
  cx.red[(t & (k2wRedBufs - 1)) * k2wRedTile + w * k2wRedRow + (lane >> 4) * k2wRedGrp + s * 16 +
         (lane & 15)] = (e.part[0] + e.part[1]) + (e.part[2] + e.part[3]);
  e.part[0] = e.part[1] = e.part[2] = e.part[3] = 0.f;
}

// The units of tile t (4 sub-tiles x NRT row tiles), lag-one epilogues, all finished.
template <int D, bool kMaxMean, int NRT, bool kMask>
__device__ __forceinline__ void tile_units_2w(const Ctx2w& cx, Epi2w& e, const char* tb, int t,
                                              const KRead16& rp,
                                              const bf16x8 (&qreg)[k2wRowTiles][Geom16<D>::kSteps],
                                              const float (&beta)[k2wRowTiles][4]) {
  constexpr int S = Geom16<D>::kSteps;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  f32x4 prev = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < kSubTiles; ++s) {
    bf16x8 kb[S];
#pragma unroll
    for (int ks = 0; ks < S; ++ks) kb[ks] = lds_k16<D>(tb, s, rp, ks);
#pragma unroll
    for (int rt = 0; rt < NRT; ++rt) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < S; ++ks) acc = mfma16(qreg[rt][ks], kb[ks], acc);
      // the previous unit's epilogue (sub-tile s of row tile rt - 1, or the last row tile
      // of sub-tile s - 1), independent of this chain
      if (s > 0 || rt > 0) {
        const int ps = rt > 0 ? s : s - 1, prt = rt > 0 ? rt - 1 : NRT - 1;
        epilogue_2w<kMaxMean, kMask>(e, prev, prt, beta[prt],
                                     cx.pos_s + (w + k2wWaves * prt) * kRowTile + 4 * (lane >> 4),
                                     t * kKeyTile + ps * 16 + (lane & 15), cx.alpha, cx.G);
        if (prt == NRT - 1) put_partial_2w(cx, e, t, ps);
      }
      prev = acc;
    }
  }
  epilogue_2w<kMaxMean, kMask>(e, prev, NRT - 1, beta[NRT - 1],
                               cx.pos_s + (w + k2wWaves * (NRT - 1)) * kRowTile + 4 * (lane >> 4),
                               t * kKeyTile + (kSubTiles - 1) * 16 + (lane & 15), cx.alpha, cx.G);
  put_partial_2w(cx, e, t, kSubTiles - 1);
}

// Sweep key tiles i0 .. i1-1 of one segment.  NRT == 0: a wave none of whose row tiles holds
// a real row (its partial slots stay zero; it keeps the loads, barriers and finishes).
// The vector-memory sequence of every wave is (one tile's loads, one store) per tile from
// the prologue on, so one wait count serves every tile: when tile i must have landed, the
// loads of tiles i+1 and i+2 and three stores may still be in flight.
template <int D, bool kMaxMean, int NRT>
__device__ __forceinline__ void sweep_2w(const Ctx2w& cx, const KLoadPlan<D, k2wWaves>& kp,
                                         const bf16x8 (&qreg)[k2wRowTiles][Geom16<D>::kSteps],
                                         const float (&beta)[k2wRowTiles][4]) {
  using Gm = TileGeom<D, k2wWaves>;
  constexpr int kVm = (k2wStages - 2) * (Gm::kLoadsPerWave + 1) + 1;
  auto clamp_tile = [&](int t) { return t < cx.i1 ? t : cx.i1 - 1; };
  if constexpr (NRT == 0) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
    for (int b = 0; b < k2wRedBufs; ++b)
#pragma unroll
      for (int s = 0; s < kSubTiles; ++s)
        cx.red[b * k2wRedTile + w * k2wRedRow + (lane >> 4) * k2wRedGrp + s * 16 + (lane & 15)] = 0.f;
  }
#pragma unroll
  for (int p = 0; p < k2wStages - 1; ++p) {
    issue_k_tile<D, k2wWaves>(cx.kl + p * Gm::kTileBytes, cx.kv_bytes,
                              page_of<D, k2wWaves>(cx.bt_row, cx.L, kp, clamp_tile(cx.i0 + p)),
                              cx.num_pages, cx.page_bytes, kp);
    finish_2w(cx, 0, false);   // the store slot of the tile (writes nothing)
  }
  int32_t next_page = page_of<D, k2wWaves>(cx.bt_row, cx.L, kp, clamp_tile(cx.i0 + k2wStages - 1));
  const KRead16 rp = make_k_read16<D>();
  Epi2w e;
  e.part[0] = e.part[1] = e.part[2] = e.part[3] = 0.f;
  e.ex = 0.f;
  e.mx = 0.f;
  for (int i = cx.i0; i < cx.i1; ++i) {
    const int32_t page = next_page;
    // the page of the tile after the one issued below: a scalar load, retired by the full
    // wait before the barrier (an outstanding scalar load would make every later LDS wait
    // of the tile a wait for all LDS traffic)
    next_page = page_of<D, k2wWaves>(cx.bt_row, cx.L, kp, clamp_tile(i + k2wStages));
    wait_vmcnt<kVm>();   // tile i has landed
    wait_lgkmcnt0();     // this wave's partials of tile i - 1 are written
    __builtin_amdgcn_s_barrier();
    // no wave reads tile i - 1 any more: its stage takes tile i + 3
    issue_k_tile<D, k2wWaves>(cx.kl + ((i - cx.i0 + k2wStages - 1) & (k2wStages - 1)) * Gm::kTileBytes,
                              cx.kv_bytes, page, cx.num_pages, cx.page_bytes, kp);
    finish_2w(cx, i - 1, i > cx.i0);
    if constexpr (NRT > 0) {
      const char* tb = cx.kbuf + ((i - cx.i0) & (k2wStages - 1)) * Gm::kTileBytes;
      if (i * kKeyTile + kKeyTile - 1 > cx.mask_from)
        tile_units_2w<D, kMaxMean, NRT, true>(cx, e, tb, i, rp, qreg, beta);
      else
        tile_units_2w<D, kMaxMean, NRT, false>(cx, e, tb, i, rp, qreg, beta);
    }
  }
  wait_lgkmcnt0();
  __builtin_amdgcn_s_barrier();
  finish_2w(cx, cx.i1 - 1, true);
}

}  // namespace

template <int D, bool kMaxMean>
__global__ __launch_bounds__(k2wThreads, 1) void score_kernel(
    DevProblem dp, const uint16_t* __restrict__ q_ptr, const uint16_t* __restrict__ kv_ptr,
    const int32_t* __restrict__ bt_ptr, const float* __restrict__ lse_ptr,
    float* __restrict__ scores_ptr, float* __restrict__ part_ptr, int64_t num_scores,
    int64_t seg_lo, int64_t seg_hi) {
  if (!plan_ok(dp)) return;   // the workspace holds another problem's plan
  using Gm = TileGeom<D, k2wWaves>;
  __shared__ __align__(1024) char kbuf[k2wStages][Gm::kTileBytes];
  __shared__ __align__(16) float beta_s[kRowsPerChunk];
  __shared__ __align__(16) int32_t pos_s[kRowsPerChunk];
  __shared__ __align__(16) float red[k2wRedBufs * k2wRedTile];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int G = dp.G, Hq = dp.Hq, Hkv = dp.Hkv, C = dp.max_chunks;
  const bool grouped = kMaxMean && (G == 8 || G == 16);
  const int64_t base = dp.seg_cost[seg_lo], total = dp.seg_cost[seg_hi] - base;
  const int64_t c0 = base + total * blockIdx.x / gridDim.x;
  const int64_t c1 = base + total * (blockIdx.x + 1) / gridDim.x;
  if (c0 >= c1) return;

  Ctx2w cx;
  cx.kv_bytes = reinterpret_cast<const char*>(kv_ptr);
  cx.pos_s = pos_s;
  cx.kbuf = &kbuf[0][0];
  cx.red = red;
  cx.kl = (uint32_t)(uintptr_t)(lds_char*)&kbuf[0][0];
  cx.page_bytes = (int64_t)kPageSize * Hkv * D * 2;
  cx.num_pages = dp.num_pages;
  cx.G = G;
  cx.alpha = dp.sm_scale * kLog2e;

  int64_t lo = seg_lo, hi = seg_hi;
  while (lo < hi) {
    const int64_t mid = (lo + hi + 1) / 2;
    if (dp.seg_cost[mid] <= c0) lo = mid; else hi = mid - 1;
  }
  bool first = true;
  for (int64_t s = lo; s < seg_hi; ++s) {
    const int64_t cs = dp.seg_cost[s], ce = dp.seg_cost[s + 1];
    if (cs >= c1) break;
    if (ce == cs) continue;
    int r, c, h;
    decode_segment(s, C, Hkv, &r, &c, &h);
    const ReqPlan pl = dp.plan[r];
    const int L = pl.L, n = pl.n, M = G * n;
    const int64_t TC = score_tile_cost(chunk_units(M - (int64_t)c * kRowsPerChunk));
    const int64_t ntiles = ceil_div64(L, kKeyTile);
    int64_t i1 = (c1 - cs + TC - 1) / TC;
    if (i1 > ntiles) i1 = ntiles;
    cx.i0 = first ? (int)((c0 - cs + TC - 1) / TC) : 0;
    cx.i1 = (int)i1;
    first = false;
    if (cx.i0 >= cx.i1) continue;

    wait_vmcnt<0>();   // no load of the previous segment may still land in a K buffer
    __syncthreads();
    for (int m = tid; m < kRowsPerChunk; m += k2wThreads) {
      int j, g;
      row_query_2w(G, grouped, c, m / kRowTile, m % kRowTile, &j, &g);
      beta_s[m] = j < n ? lse_ptr[(int64_t)(pl.q_off + j) * Hq + h * G + g] * kLog2e
                        : __builtin_inff();
      pos_s[m] = dp.causal ? L - n + j : L - 1;
    }
    bf16x8 qreg[k2wRowTiles][Geom16<D>::kSteps];
#pragma unroll
    for (int rt = 0; rt < k2wRowTiles; ++rt)
      load_q16<D>(qreg[rt], q_ptr, G, grouped, Hq, h, pl.q_off, n, c, w + k2wWaves * rt);
    cx.bt_row = bt_ptr + (int64_t)r * dp.bt_stride;
    cx.L = L;
    cx.mask_from = dp.causal ? L - n : L;
    cx.out_scale = (kMaxMean && pl.nchunk == 1) ? (n > 0 ? 1.0f / n : 0.0f) : 1.0f;
    cx.out = buffer_over_uniform((c == 0) ? scores_ptr + pl.seg_off + (int64_t)h * L
                                          : part_ptr + (int64_t)(c - 1) * num_scores +
                                                pl.seg_off + (int64_t)h * L,
                                 L * (int)sizeof(float));
    const KLoadPlan<D, k2wWaves> kp = make_k_load_plan<D, k2wWaves>(h, Hkv);
    wait_vmcnt<0>();
    __syncthreads();   // beta_s / pos_s visible
    float beta[k2wRowTiles][4];
#pragma unroll
    for (int rt = 0; rt < k2wRowTiles; ++rt) {
      const float4 b4 = *reinterpret_cast<const float4*>(beta_s + (w + k2wWaves * rt) * kRowTile +
                                                         4 * (lane >> 4));
      beta[rt][0] = b4.x; beta[rt][1] = b4.y; beta[rt][2] = b4.z; beta[rt][3] = b4.w;
    }
    const int nrt = wave_tiles_2w(G, grouped, n, c);
    bool real = false;
    for (int rt = 0; rt < nrt; ++rt) {
      int j, g;
      row_query_2w(G, grouped, c, w + k2wWaves * rt, lane & 15, &j, &g);
      real = real || j < n;
    }
    switch (__ballot(real) == 0ull ? 0 : nrt) {
      case 0: sweep_2w<D, kMaxMean, 0>(cx, kp, qreg, beta); break;
      case 1: sweep_2w<D, kMaxMean, 1>(cx, kp, qreg, beta); break;
      case 2: sweep_2w<D, kMaxMean, 2>(cx, kp, qreg, beta); break;
      case 3: sweep_2w<D, kMaxMean, 3>(cx, kp, qreg, beta); break;
      default: sweep_2w<D, kMaxMean, 4>(cx, kp, qreg, beta); break;
    }
  }
  wait_vmcnt<0>();   // drain: no LDS write may be outstanding when the workgroup exits
}

// scores = (scores + sum_{c >= 1} partial_c) * scale, for requests scored in several row
// chunks (fixed order: deterministic).
__global__ __launch_bounds__(256) void chunk_reduce_kernel(DevProblem dp, int r0, float* scores,
                                                           const float* part,
                                                           int64_t num_scores) {
  if (!plan_ok(dp)) return;   // the workspace holds another problem's plan
  const int r = r0 + (int)blockIdx.y, h = blockIdx.z;
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

hipError_t launch_score_range(const DevProblem& dp, const HostPlan& hp, int r0, int r1,
                              int64_t cost, const void* q, const void* kv, const int32_t* bt,
                              const float* lse, float* scores, float* score_part,
                              hipStream_t s) {
  if (hp.num_scores == 0 || r0 >= r1 || cost <= 0) return hipSuccess;
  const uint16_t* qq = static_cast<const uint16_t*>(q);
  const uint16_t* kk = static_cast<const uint16_t*>(kv);
  const int64_t spr = (int64_t)hp.max_chunks * hp.Hkv;   // a request's segments are consecutive
  const int64_t seg_lo = r0 * spr, seg_hi = r1 * spr;
  int64_t grid = device_cus();   // one workgroup per CU
  if (grid > cost) grid = cost;
  const bool mm = dp.agg == ACTKV_AGG_MAX_MEAN;
  const int64_t n = hp.num_scores;
  if (dp.D == 128) {
    if (mm) hipLaunchKernelGGL((score_kernel<128, true>), dim3(grid), dim3(k2wThreads), 0, s, dp, qq, kk, bt, lse, scores, score_part, n, seg_lo, seg_hi);
    else hipLaunchKernelGGL((score_kernel<128, false>), dim3(grid), dim3(k2wThreads), 0, s, dp, qq, kk, bt, lse, scores, score_part, n, seg_lo, seg_hi);
  } else {
    if (mm) hipLaunchKernelGGL((score_kernel<64, true>), dim3(grid), dim3(k2wThreads), 0, s, dp, qq, kk, bt, lse, scores, score_part, n, seg_lo, seg_hi);
    else hipLaunchKernelGGL((score_kernel<64, false>), dim3(grid), dim3(k2wThreads), 0, s, dp, qq, kk, bt, lse, scores, score_part, n, seg_lo, seg_hi);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (hp.max_chunks > 1) {
    hipLaunchKernelGGL(chunk_reduce_kernel, dim3(64, r1 - r0, hp.Hkv), dim3(256), 0, s, dp, r0,
                       scores, score_part, hp.num_scores);
    e = hipGetLastError();
  }
  return e;
}

hipError_t launch_score(const DevProblem& dp, const HostPlan& hp, const void* q,
                        const void* kv, const int32_t* bt, const float* lse, float* scores,
                        float* score_part, hipStream_t s) {
  return launch_score_range(dp, hp, 0, hp.R, hp.score_cost, q, kv, bt, lse, scores, score_part,
                            s);
}

// acc[i] += s[i] (streaming aggregation: the scores of one decode step added to the running
// aggregate).  Four floats per lane per step, grid-stride.
__global__ __launch_bounds__(256) void accumulate_kernel(float* acc, const float* s, int64_t n) {
  const int64_t n4 = n / 4;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += (int64_t)gridDim.x * 256) {
    float4 a = reinterpret_cast<float4*>(acc)[i];
    const float4 b = reinterpret_cast<const float4*>(s)[i];
    a.x += b.x; a.y += b.y; a.z += b.z; a.w += b.w;
    reinterpret_cast<float4*>(acc)[i] = a;
  }
  for (int64_t i = n4 * 4 + (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    acc[i] += s[i];
}

hipError_t launch_accumulate(float* acc, const float* s, int64_t n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  int64_t blocks = (n / 4 + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(accumulate_kernel, dim3((unsigned)blocks), dim3(256), 0, st, acc, s, n);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------------------
// Decode-step scoring (one action query per request: Alg. 3 as run once per generated
// token).  The G <= 16 query rows of a KV head fill one 16-row MFMA tile (rows past G are
// zero with beta = +inf).  A wave streams whole pages of its head's K (16 keys) from global
// memory straight into the MFMA B operand, kDecRing pages in flight, and keeps the pages'
// scores in LDS; every kDecFlushPages pages it adds them to the aggregate with contiguous
// 256-byte loads and stores.  (A store inside the page loop would make every later wait for
// a K load wait for the store as well.)  The waves of a workgroup are the KV heads (up to
// 8 per workgroup, head groups along y) and walk the same pages: a page's heads are
// interleaved in memory (slot-major rows), so reading them at about the same time keeps the
// DRAM accesses of a page together.  Workgroups take equal contiguous shares of the
// (request, 64-key tile) list.  Bound by reading K; no barriers.
// ---------------------------------------------------------------------------------------
constexpr int kDecMaxWaves = 8;      // KV heads per workgroup
constexpr int kDecRing = 4;          // pages of K in flight per wave
constexpr int kDecFlushPages = 64;   // pages whose scores a wave holds in LDS

template <int D, bool kMaxMean>
__global__ __launch_bounds__(kDecMaxWaves * 64) void score_decode_kernel(
    DevProblem dp, const uint16_t* __restrict__ q_ptr, const char* __restrict__ kv_bytes,
    const int32_t* __restrict__ bt_ptr, const float* __restrict__ lse_ptr,
    float* __restrict__ acc_ptr) {
  if (!plan_ok(dp)) return;   // the workspace holds another problem's plan
  constexpr int S = Geom16<D>::kSteps;
  constexpr int kFlushKeys = kDecFlushPages * kPageSize;
  __shared__ float res_s[kDecMaxWaves][kFlushKeys];
  const int lane = threadIdx.x & 63;
  const int G = dp.G, Hq = dp.Hq, Hkv = dp.Hkv, R = dp.R;
  // this wave's head, through readfirstlane: everything derived from it is then known to be
  // wave-uniform (scalar loads of the plan and block table, scalar branches)
  const int wv = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int h = (int)blockIdx.y * (int)(blockDim.x / 64) + wv;
  float* res = res_s[wv];
  // with at most one query per request every key tile costs the same,
  // score_tile_cost(chunk_units(1)), so seg_cost[r * Hkv] / (Hkv * that cost) is the number
  // of (request, key tile) pairs before request r
  auto tiles_before = [&](int rr) {
    return dp.seg_cost[(int64_t)rr * Hkv] / (Hkv * score_tile_cost(chunk_units(1)));
  };
  const int64_t total = tiles_before(R);
  const int64_t c0 = total * blockIdx.x / gridDim.x, c1 = total * (blockIdx.x + 1) / gridDim.x;
  if (c0 >= c1) return;
  const float alpha = dp.sm_scale * kLog2e;
  const int64_t page_bytes = (int64_t)kPageSize * Hkv * D * 2;
  // first request: the largest r with tiles_before(r) <= c0 (a prefix of 0 .. R, since
  // tiles_before does not decrease), 64 candidates per load and ballot
  int lo = 0;
  for (int base = 0; base <= R; base += 64) {
    const int rr = base + lane;
    const uint64_t m = __ballot(rr <= R && tiles_before(rr) <= c0);
    if (m == 0ull) break;
    lo = base + 63 - __builtin_clzll(m);
    if (m != ~0ull) break;
  }
  for (int r = lo; r < R; ++r) {
    const int64_t cs = tiles_before(r);
    if (cs >= c1) break;
    const ReqPlan pl = dp.plan[r];
    if (pl.n == 0 || pl.L == 0) continue;   // nothing to add
    const int L = pl.L;
    const int64_t ntiles = ceil_div64(L, kKeyTile);
    const int64_t t0 = c0 > cs ? c0 - cs : 0, t1 = c1 - cs < ntiles ? c1 - cs : ntiles;
    const int npages = ceil_div(L, kPageSize);
    const int p0 = (int)t0 * (kKeyTile / kPageSize);
    const int p1 = (int)t1 * (kKeyTile / kPageSize) < npages ? (int)t1 * (kKeyTile / kPageSize)
                                                              : npages;
    if (p0 >= p1) continue;
    // the query's G rows (row m = head m of the group) and beta of this lane's rows
    bf16x8 qr[S];
    load_q16<D>(qr, q_ptr, G, false, Hq, h, pl.q_off, 1, 0, 0);
    float beta[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = 4 * (lane >> 4) + i;
      beta[i] = m < G ? lse_ptr[(int64_t)pl.q_off * Hq + h * G + m] * kLog2e : __builtin_inff();
    }
    const int32_t* bt_row = bt_ptr + (int64_t)r * dp.bt_stride;
    float* out = acc_ptr + pl.seg_off + (int64_t)h * L;
    // the aggregate of this segment: reads past L return 0, writes there are dropped
    const __amdgpu_buffer_rsrc_t ars = buffer_over(out, L * (int)sizeof(float));
    const uint32_t lane_off = (uint32_t)((((lane & 15) * Hkv + h) * D) * 2 + (lane >> 4) * 16);
    for (int fb = p0; fb < p1; fb += kDecFlushPages) {
      const int pe = fb + kDecFlushPages < p1 ? fb + kDecFlushPages : p1;
      u32x4 kb[kDecRing][S];
      auto issue = [&](int slot, int p) {
        int64_t page = bt_row[p];
        if (page < 0 || page >= dp.num_pages) page = 0;   // never dereference outside the pool
        const char* base = kv_bytes + page * page_bytes + lane_off;
#pragma unroll
        for (int ks = 0; ks < S; ++ks)
          kb[slot][ks] = *reinterpret_cast<const u32x4*>(base + 64 * ks);
      };
      // Every slot is refilled after its use on every step (past the block's last page: that
      // page again) and every step computes; steps past the block keep nothing.  With no
      // conditional loads in the loop a slot keeps its registers from step to step and the
      // compiler's waits stay partial.
      const int last = pe - 1;
#pragma unroll
      for (int j = 0; j < kDecRing; ++j) issue(j, fb + j < pe ? fb + j : last);
      for (int pb = fb; pb < pe; pb += kDecRing) {
#pragma unroll
        for (int j = 0; j < kDecRing; ++j) {
          const int p = pb + j;
          f32x4 cacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int ks = 0; ks < S; ++ks) cacc = mfma16(qr[ks], as_bf16x8(kb[j][ks]), cacc);
          // this lane's 4 rows in order, then the lane groups (rows 4-7, 8-15) in order
          float v = 0.f;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float e = fast_exp2(__builtin_fmaf(cacc[i], alpha, -beta[i]));
            v = kMaxMean ? fmaxf(v, e) : v + e;
          }
          if (G > 4) {
            const float o = __shfl_xor(v, 16, 64);
            v = kMaxMean ? fmaxf(v, o) : v + o;
          }
          if (G > 8) {
            const float o = __shfl_xor(v, 32, 64);
            v = kMaxMean ? fmaxf(v, o) : v + o;
          }
          if (lane < 16 && p < pe) res[(p - fb) * kPageSize + lane] = v;
          // the slot is refilled only now, once the chain that read it has finished (an earlier
          // refill would need other registers, and the loop edge would then wait for them)
          issue(j, p + kDecRing < pe ? p + kDecRing : last);
        }
      }
      // add the block's scores to the aggregate: lane l takes keys 16 fb + 64 i + l.  All
      // loads first and no conditional ones, so the stores follow a single wait; keys past
      // the block (the next block's, or another workgroup's share) use an offset past the
      // buffer: read as 0, not written
      const int nk = (pe - fb) * kPageSize;
      float a[kFlushKeys / 64];
#pragma unroll
      for (int i = 0; i < kFlushKeys / 64; ++i) {
        const int k = i * 64 + lane;
        a[i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                             ars, k < nk ? (fb * kPageSize + k) * 4 : 0x7FFFFFF0,
                                             0, 0));
      }
#pragma unroll
      for (int i = 0; i < kFlushKeys / 64; ++i) {
        const int k = i * 64 + lane;
        const float sc = k < nk ? res[k] : 0.f;
        __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, a[i] + sc), ars,
                                              k < nk ? (fb * kPageSize + k) * 4 : 0x7FFFFFF0, 0,
                                              0);
      }
    }
  }
}

hipError_t launch_score_decode(const DevProblem& dp, const HostPlan& hp, const void* q,
                               const void* kv, const int32_t* bt, const float* lse, float* acc,
                               hipStream_t s) {
  if (hp.num_scores == 0 || hp.sum_n == 0) return hipSuccess;
  const int cus = device_cus();
  const uint16_t* qq = static_cast<const uint16_t*>(q);
  const char* kk = static_cast<const char*>(kv);
  const bool mm = dp.agg == ACTKV_AGG_MAX_MEAN;
  // waves per workgroup: the largest divisor of Hkv up to kDecMaxWaves (every wave a head)
  int waves = 1;
  for (int w = 1; w <= kDecMaxWaves; ++w)
    if (hp.Hkv % w == 0) waves = w;
  const unsigned groups = (unsigned)(hp.Hkv / waves);
  const int64_t tiles = hp.score_cost / (hp.Hkv * score_tile_cost(chunk_units(1)));   // (request, key tile) pairs
  // one resident round of workgroups (equal contiguous shares: a second round would only
  // add a tail), at most one per tile.  Residency per CU is asked once per kernel and
  // workgroup size (it depends on nothing else).
  static std::atomic<int> cached[2][2][kDecMaxWaves + 1];   // [D == 128][MAX_MEAN][waves]
  auto launch = [&](auto kernel) -> hipError_t {
    std::atomic<int>& slot = cached[dp.D == 128][mm][waves];
    int per_cu = slot.load(std::memory_order_relaxed);
    if (per_cu == 0) {
      if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, waves * 64, 0) != hipSuccess ||
          per_cu < 1)
        per_cu = 1;
      slot.store(per_cu, std::memory_order_relaxed);
    }
    int64_t blocks = (int64_t)cus * per_cu / groups;
    if (blocks > tiles) blocks = tiles;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(kernel, dim3((unsigned)blocks, groups), dim3(waves * 64), 0, s, dp, qq, kk,
                       bt, lse, acc);
    return hipGetLastError();
  };
  if (dp.D == 128)
    return mm ? launch(score_decode_kernel<128, true>) : launch(score_decode_kernel<128, false>);
  return mm ? launch(score_decode_kernel<64, true>) : launch(score_decode_kernel<64, false>);
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
  if (!plan_ok(dp)) return;   // the workspace holds another problem's plan
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
                               page_of<D, kLseWaves>(bt_row, L, kp, clamp_tile(t0 + p)),
                               dp.num_pages, page_bytes, kp);
  int32_t next_page = page_of<D, kLseWaves>(bt_row, L, kp, clamp_tile(t0 + kStages - 1));
  // keys up to the first action query's position are visible to every real row (rows past
  // n, all padding, are never written): tiles below it need no mask
  const int64_t open_to = dp.causal ? (int64_t)L - n : (int64_t)L - 1;
  for (int64_t i = t0; i < t1; ++i) {
    const int st = (int)((i - t0) % kStages);
    wait_vmcnt<(kStages - 2) * Gm::kLoadsPerWave>();
    __builtin_amdgcn_s_barrier();
    issue_k_tile<D, kLseWaves>(kl + ((st + kStages - 1) % kStages) * Gm::kTileBytes, kv_bytes,
                               next_page, dp.num_pages, page_bytes, kp);
    next_page = page_of<D, kLseWaves>(bt_row, L, kp, clamp_tile(i + kStages));
    const bool masked = i * kKeyTile + kKeyTile - 1 > open_to;
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
          if (masked) {
#pragma unroll
            for (int v = 0; v < 16; ++v) {
              const int key = keybase + 8 * (v / 4) + (v % 4);
              x[v] = key <= pos[ti] ? x[v] : -__builtin_inff();
            }
          }
          // 2^(alpha x - m) with the scale and the shift in one FMA, first against the
          // running shift m0 as it stands: while no term of the tile exceeds 2^64 the
          // (shift, sum) pair stays exact to rounding whether or not m0 is the running max,
          // so the max is taken (on the raw dot products: alpha > 0 keeps the order) only
          // for a row's first tile and when a larger value arrives
          const float m0 = rm[ti];
          float sum = 0.f;
#pragma unroll
          for (int v = 0; v < 16; ++v) sum += fast_exp2(__builtin_fmaf(x[v], alpha, -m0));
          if (sum <= kLseLazyLimit) {
            rs[ti] += sum;
          } else {   // also the first tile (m0 = -inf gives inf or NaN terms)
            float mx = -__builtin_inff();
#pragma unroll
            for (int v = 0; v < 16; ++v) mx = fmaxf(mx, x[v]);
            const float m = fmaxf(m0, mx * alpha);
            if (m != -__builtin_inff()) {
              float s2 = rs[ti] * fast_exp2(m0 - m);
#pragma unroll
              for (int v = 0; v < 16; ++v) s2 += fast_exp2(__builtin_fmaf(x[v], alpha, -m));
              rs[ti] = s2;
              rm[ti] = m;
            }
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

// One thread per (request, query row): the row's block partials in block order, eight
// loads in flight at a time.  Grid: (requests, ceil(max rows per request / 256)).
__global__ __launch_bounds__(256) void lse_merge_kernel(DevProblem dp, const float2* part,
                                                        float* lse) {
  if (!plan_ok(dp)) return;   // the workspace holds another problem's plan
  constexpr int kBatch = 8;
  const int r = blockIdx.x;
  const ReqPlan pl = dp.plan[r];
  const int rows = pl.n * dp.Hq;
  const int row = blockIdx.y * 256 + threadIdx.x;
  if (row >= rows) return;
  const float2* pp = part + pl.lse_part_off + (int64_t)row * pl.lse_blocks;
  const int nb = pl.lse_blocks;
  float m = -__builtin_inff();
  for (int b0 = 0; b0 < nb; b0 += kBatch) {
    float2 v[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) v[u] = b0 + u < nb ? pp[b0 + u] : make_float2(-__builtin_inff(), 0.f);
#pragma unroll
    for (int u = 0; u < kBatch; ++u) m = fmaxf(m, v[u].x);
  }
  float s = 0.f;
  if (m != -__builtin_inff()) {
    for (int b0 = 0; b0 < nb; b0 += kBatch) {
      float2 v[kBatch];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) v[u] = b0 + u < nb ? pp[b0 + u] : make_float2(-__builtin_inff(), 0.f);
#pragma unroll
      for (int u = 0; u < kBatch; ++u)
        if (b0 + u < nb) s += v[u].y * fast_exp2(v[u].x - m);
    }
  }
  // natural-log LSE = (m + log2 s) * ln 2
  lse[(int64_t)pl.q_off * dp.Hq + row] =
      m == -__builtin_inff() ? -__builtin_inff() : (m + __log2f(s)) * 0.6931471805599453f;
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
  const int64_t max_rows = hp.max_n * hp.Hq;
  hipLaunchKernelGGL(lse_merge_kernel, dim3((unsigned)hp.R, (unsigned)((max_rows + 255) / 256)),
                     dim3(256), 0, s, dp, lse_part, lse_out);
  return hipGetLastError();
}

}  // namespace actkv
