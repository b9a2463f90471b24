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
//   * One workgroup of 4 waves per CU (one wave per SIMD), persistent: the list of
//     (segment, 64-key tile) work, segment = (request, row chunk of up to 512 query rows,
//     KV head), is cut into equal-cost contiguous ranges, one per workgroup, so ragged
//     lengths and query counts stay balanced and Q is loaded once per segment.
//   * Each wave holds 8 row tiles of 16 query rows in registers (v_mfma_f32_16x16x32_bf16
//     A operand) and the beta of its rows.  Every wave reads each K tile from LDS once per
//     sub-tile, so the LDS read traffic per tile is (waves x tile bytes): four waves of 128
//     rows read half of what eight waves of 64 rows would.  K tiles (64 keys, 4 pages) are gathered
//     through the block table straight into LDS (global_load_lds_dwordx4, 16 bytes per
//     lane, chunk-swizzled rows), kScoreStages - 1 tiles ahead, one barrier per tile.
//   * The MFMA chains and the exp2 epilogue are software-pipelined inside each wave (see
//     the sweep below): the VALU works on one 16x16 unit while the matrix core works on
//     another.
//   * A lane's accumulator column is one key and 4 query rows, so the row sum is in-lane;
//     the 4 lane groups and 4 waves are combined through LDS in a fixed order (no
//     atomics: deterministic, and independent of where the pages physically live).
#include <atomic>

#include "device_common.hpp"

namespace actkv {

namespace {

// Scoring: 4 waves per workgroup (one per SIMD, up to 512 registers each), 128 query rows
// per wave, one workgroup per CU.  Every wave reads the whole K tile from LDS, so fewer,
// taller waves read less: LDS traffic, not arithmetic, bounded the 8-wave form.
constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kScoreStages = 4;   // K tiles resident in LDS for scoring (three in flight)
constexpr int kStages = 3;        // the same for the LSE pass
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

// ---- scoring: software-pipelined 16x16x32 MFMA units -----------------------------------
//
// A wave owns kRowTilesPerWave row tiles of 16 query rows (the MFMA A operand, held in
// registers for the whole segment).  Each 64-key tile in LDS is cut into 4 sub-tiles of 16
// keys (the B operand).  A "unit" is one (sub-tile, row tile) pair: kSteps16 dependent
// MFMAs into a 16x16 accumulator -- lane l holds key l%16 and rows 4*(l/16) .. +3 -- and
// then its epilogue: exp2 of the 4 elements, summed (or max-reduced over the GQA group)
// into the lane's partial for that key.
//
// Phase g issues the chain of unit g one MFMA per slot and, between those MFMAs, the
// epilogue of unit g - 2, whose accumulator was finished a whole phase earlier.  The two
// are independent, so the VALU works on one unit while the matrix core works on the other.
// The K operand of a sub-tile is read from LDS kOperandAhead sub-tiles before its first
// chain (rotating operand buffers), so the reads' latency is hidden behind that many
// sub-tiles of work (LDS reads queue behind the K tiles' direct-to-LDS writes).

constexpr int kRowTile = 16;
constexpr int kRowTilesPerWave = kRowsPerChunk / kRowTile / kWaves;   // 8
constexpr int kSubTiles = kKeyTile / 16;                              // 4
static_assert(kRowTilesPerWave == 8 && kSubTiles == 4, "unit bookkeeping below");
// Sub-tiles of lookahead of the operand reads, and the buffers they rotate through (sub-tile
// s of every tile uses buffer s % kOperandBufs, so the count divides the sub-tiles).
constexpr int kOperandAhead = 2;
constexpr int kOperandBufs = 4;
static_assert(kOperandAhead >= 1 && kOperandAhead <= 2 && kOperandBufs > kOperandAhead &&
                  kSubTiles % kOperandBufs == 0,
              "a chain in the next tile (units 0 and 1) reads ahead within that tile");

template <int D>
struct Geom16 {
  static constexpr int kSteps = D / 32;   // k-steps of 32 per head
};

// Query row at (row tile T = w + kWaves * rt, tile row mm) of row chunk c.  The natural
// order m = j * G + g is used unless the group max of MAX_MEAN needs a query's G = 8 or 16
// heads in one lane: then they sit at the same lane position of 2 or 4 consecutive row
// tiles of the wave (heads 4*(rt % 2) + i, resp. 4*(rt % 4) + i).
__device__ __forceinline__ void score_row_query(int G, bool grouped, int c, int T, int mm,
                                                int* j, int* g) {
  if (!grouped) {
    const int m = c * kRowsPerChunk + T * kRowTile + mm;
    *j = m / G;
    *g = m % G;
    return;
  }
  const int w = T % kWaves, rt = T / kWaves, a = mm >> 2, i = mm & 3;
  if (G == 8) {
    *j = c * (kRowsPerChunk / 8) + (rt >> 1) * (4 * kWaves) + w * 4 + a;
    *g = 4 * (rt & 1) + i;
  } else {
    *j = c * (kRowsPerChunk / 16) + (rt >> 2) * (4 * kWaves) + w * 4 + a;
    *g = 4 * (rt & 3) + i;
  }
}

// Row tiles per wave that can hold real rows of chunk c (the same for every wave).
__device__ __forceinline__ int chunk_wave_tiles(int G, bool grouped, int n, int c) {
  if (!grouped) {
    const int rows = G * n - c * kRowsPerChunk;
    if (rows <= 0) return 1;
    const int r = rows < kRowsPerChunk ? rows : kRowsPerChunk;
    return ceil_div(r, kRowTile * kWaves);
  }
  // row tiles come in groups of G / 4 (one group: 4 queries per wave)
  const int per = G / 4, qn = n - c * (kRowsPerChunk / G);
  const int groups = qn <= 0 ? 1 : ceil_div(qn, 4 * kWaves);
  const int t = groups * per;
  return t < kRowTilesPerWave ? t : kRowTilesPerWave;
}

// Row tile rt of this wave as the 16x16x32 A operand: lane l holds row l%16 with head-dim
// elements 32*ks + 8*(l/16) .. +8; rows past n are zero.
template <int D>
__device__ __forceinline__ void load_q16(bf16x8 (&qr)[Geom16<D>::kSteps],
                                         const uint16_t* __restrict__ q, int G, bool grouped,
                                         int Hq, int h, int q_off, int n, int c, int T) {
  const int lane = threadIdx.x & 63;
  int j, g;
  score_row_query(G, grouped, c, T, lane & 15, &j, &g);
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

// Per-wave state carried from phase to phase.
template <int D>
struct Pipe16 {
  f32x4 c1, c2;                       // accumulators of units g-1 and g-2
  bf16x8 kb[kOperandBufs][Geom16<D>::kSteps];   // B operands: sub-tile s reads kb[s % bufs]
  float part[4];                      // the lane's partials of the current sub-tile, one per
                                      // accumulator element (independent add chains)
  float ex;                           // SUM: the last exp2 result, added one slot later
  float mx;                           // MAX_MEAN, G = 8 / 16: running group max
};

// One phase.  kChain: chain of row tile q against operand kr.  kEpi: epilogue of st.c2 for
// row tile kRt (beta bt, causal positions at prow, key `key`).  kLoad: kl <- the operand of
// sub-tile next_sub of next_buf (read from LDS here, used a whole sub-tile later).
template <int D, bool kMaxMean, bool kMask, bool kChain, bool kEpi, bool kLoad, int kRt>
__device__ __forceinline__ void score_phase16(Pipe16<D>& st, const bf16x8 (&q)[Geom16<D>::kSteps],
                                              const bf16x8 (&kr)[Geom16<D>::kSteps],
                                              bf16x8 (&kl)[Geom16<D>::kSteps],
                                              const KRead16& rp, const char* next_buf, int next_sub,
                                              const float (&bt)[4], const int32_t* prow, int key,
                                              float alpha, int G) {
  constexpr int S = Geom16<D>::kSteps;
  constexpr int EPS = 4 / S;   // epilogue elements per MFMA slot
  f32x4 prev = st.c2;
  int pt[4] = {0, 0, 0, 0};
  if (kEpi && kMask) {
    const int4 p4 = *reinterpret_cast<const int4*>(prow);
    pt[0] = p4.x; pt[1] = p4.y; pt[2] = p4.z; pt[3] = p4.w;
  }
  if (kLoad) {
#pragma unroll
    for (int ks = 0; ks < S; ++ks) kl[ks] = lds_k16<D>(next_buf, next_sub, rp, ks);
  }
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ks = 0; ks < S; ++ks) {
    if (kChain) acc = mfma16(q[ks], kr[ks], acc);
    if (kEpi) {
#pragma unroll
      for (int v = ks * EPS; v < (ks + 1) * EPS; ++v) {
        float x = __builtin_fmaf(prev[v], alpha, -bt[v]);
        if (kMask) x = key > pt[v] ? -__builtin_inff() : x;   // exp2(-inf) = 0
        if (!kMaxMean) {
          // the previous element's exp2 is added now, off the exp2 latency path
          st.part[(v + 3) & 3] += st.ex;
          st.ex = fast_exp2(x);
        } else {
          prev[v] = fast_exp2(x);
        }
      }
    }
  }
  // one scheduling region per phase: the compiler interleaves the chain and the epilogue
  __builtin_amdgcn_sched_barrier(0);
  if (kEpi && kMaxMean) {
    const float m01 = fmaxf(prev[0], prev[1]), m23 = fmaxf(prev[2], prev[3]);
    if (G == 1) {
      st.part[0] += (prev[0] + prev[1]) + (prev[2] + prev[3]);
    } else if (G == 2) {
      st.part[0] += m01 + m23;
    } else if (G == 4) {
      st.part[0] += fmaxf(m01, m23);
    } else if (G == 8) {
      // heads 0-3 in even row tiles, 4-7 in the next one
      const float m = fmaxf(m01, m23);
      if (kRt & 1) st.part[0] += fmaxf(st.mx, m); else st.mx = m;
    } else {
      // G == 16: heads 4*(rt%4) .. +3 in row tile rt, four row tiles per query group
      const float m = fmaxf(m01, m23);
      st.mx = (kRt & 3) == 0 ? m : fmaxf(st.mx, m);
      if ((kRt & 3) == 3) st.part[0] += st.mx;
    }
    __builtin_amdgcn_sched_barrier(0);
  }
  st.c2 = st.c1;
  if (kChain) st.c1 = acc;
}

// Everything the key sweep of one segment needs besides the register-resident Q and beta.
struct SweepCtx {
  const char* kv_bytes;
  const int32_t* bt_row;
  const int32_t* pos_s;    // LDS: causal position of every row of the chunk
  __amdgpu_buffer_rsrc_t out;   // scores (or chunk partials) of this (request, KV head):
                                // exactly L floats, stores past them are dropped
  const char* kbuf;        // LDS: the K stages
  int64_t page_bytes, num_pages;
  int i0, i1;              // key tiles of this workgroup
  int L, mask_from, G;
  float alpha, out_scale;
  uint32_t kl;             // LDS byte address of the K stages
};

// Per-key partials of one tile: wave w, lane group q = l/16, key k at
// red[w][q * kRedGrp + k].  The padded strides keep both the writes (64 lanes: 4 groups x
// 16 keys) and the finishing reads (4 waves x 16 keys) on 64 distinct banks.
constexpr int kRedGrp = kKeyTile + 16;      // 80 floats: group stride = 16 banks apart
constexpr int kRedRow = 4 * kRedGrp + 16;   // 336 floats: wave stride = 16 banks apart
typedef float RedTile[kWaves][kRedRow];
constexpr int kRedBufs = 4;   // a tile's partials are read one tile later

// Sum of the 16 partials of each key of tile t in a fixed order; wave w finishes keys
// 16w .. 16w+15.  Lane l takes key 16w + l/4 and the four partials of wave l%4, then the
// four lanes of a key are summed pairwise (xor 1, then xor 2).
__device__ __forceinline__ float dpp_xor1(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));
}
__device__ __forceinline__ float dpp_xor2(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false));
}

// The finish of a tile in two halves, a phase apart, so that the LDS reads are not waited
// for at once: finish_read fetches this lane's four partials, finish_write sums them and
// the eight lanes of its key, and stores the key's score (only when `valid`).  Every lane
// takes part in the store (lanes that do not write use an offset past the buffer), so each
// wave issues exactly one vector-memory store per call whatever the keys, with no branch:
// the K pipeline's waits count on that.
__device__ __forceinline__ float4 finish_read(const RedTile& red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int kk = w * (kKeyTile / kWaves) + (lane >> 2), ww = lane & 3;
  const float* rr = red[ww] + kk;
  return make_float4(rr[0], rr[kRedGrp], rr[2 * kRedGrp], rr[3 * kRedGrp]);
}

__device__ __forceinline__ void finish_write(const SweepCtx& cx, float4 p, int t, bool valid) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int kk = w * (kKeyTile / kWaves) + (lane >> 2), ww = lane & 3;
  float v = (p.x + p.y) + (p.z + p.w);
  v += dpp_xor1(v);
  v += dpp_xor2(v);
  const int key = t * kKeyTile + kk;
  const uint32_t off = (valid && ww == 0 && key < cx.L) ? (uint32_t)key * 4u : 0x7FFFFFF0u;
  __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v * cx.out_scale), cx.out, off, 0, 0);
}

// The K pipeline's vector-memory sequence per wave is, from the first tile of a segment on,
// (loads of one K tile, one score store) repeated: the sweep's prologue issues a store that
// writes nothing after each of its tile loads, and the tile after the first one finishes
// nothing real.  So at the barrier of every tile, when the loads of tile i + 1 must have
// landed, exactly the stores and loads of the two tiles after it (and a store) may still be
// in flight: one wait count for every tile, and no branch in the loop body.
template <int D>
constexpr int kTileVmcnt = (kScoreStages - 2) * (TileGeom<D>::kLoadsPerWave + 1) + 1;

// Phases P = 2 .. U+1 of tile i, U = 4 * NRT units per tile: the chain of unit P (of tile
// i, or of tile i+1 once P >= U) and the epilogue of unit P - 2 of tile i.  The chain of
// the first unit of sub-tile s also reads the operand of sub-tile s + kOperandAhead from
// LDS.  Phase (4 - kOperandAhead) NRT is the first to read sub-tile 0 of tile i+1: the
// barrier that makes tile i+1 visible sits there, and once every wave has passed it no wave
// reads tile i's stage any more (its last sub-tile was read kOperandAhead sub-tiles
// earlier), which is then refilled.
// kMask: tile i holds keys hidden from some rows.  kLast: no tile follows.
template <int D, bool kMaxMean, int NRT, bool kMask, bool kLast, int P>
__device__ __forceinline__ void tile_phases16(const SweepCtx& cx, const KLoadPlan<D, kWaves>& kp,
                                              const KRead16& rp, Pipe16<D>& st,
                                              const bf16x8 (&qreg)[kRowTilesPerWave][Geom16<D>::kSteps],
                                              const float (&beta)[kRowTilesPerWave][4],
                                              RedTile* red, int i, int32_t& next_page,
                                              float4& fin) {
  constexpr int U = kSubTiles * NRT;
  if constexpr (P <= U + 1) {
    using Gm = TileGeom<D>;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    static_assert((kScoreStages & (kScoreStages - 1)) == 0, "stage index uses a mask");
    const int st_i = (i - cx.i0) & (kScoreStages - 1), st_n = (i + 1 - cx.i0) & (kScoreStages - 1);
    const char* buf_i = cx.kbuf + st_i * Gm::kTileBytes;
    const char* buf_n = cx.kbuf + st_n * Gm::kTileBytes;
    constexpr int kBarrier = (kSubTiles - kOperandAhead) * NRT;
    if constexpr (P == kBarrier) {
      // the page of the tile after the one refilled below: a scalar load, issued before the
      // barrier's full wait so that it is retired there (an outstanding scalar load would
      // make every later LDS wait of the tile a wait for all LDS traffic)
      const int32_t page = next_page;
      const int nt = i + kScoreStages + 1;
      next_page = page_of<D, kWaves>(cx.bt_row, cx.L, kp, nt < cx.i1 ? nt : cx.i1 - 1);
      // tile i + 1 is read from this phase on: this wave's loads of it have landed, this
      // wave's LDS traffic of tile i is retired, then the barrier
      wait_vmcnt<kTileVmcnt<D>>();
      wait_lgkmcnt0();
      __builtin_amdgcn_s_barrier();
      // no wave reads tile i any more: refill its stage with tile i + kScoreStages
      issue_k_tile<D, kWaves>(cx.kl + st_i * Gm::kTileBytes, cx.kv_bytes, page, cx.num_pages,
                              cx.page_bytes, kp);
      fin = finish_read(red[(i - 1) & (kRedBufs - 1)]);   // unused in the first tile
    }
    // epilogue: unit P - 2 of tile i
    constexpr int eu = P - 2, es = eu / NRT, er = eu % NRT;
    const int32_t* prow = cx.pos_s + (w + kWaves * er) * kRowTile + 4 * (lane >> 4);
    const int key = i * kKeyTile + es * 16 + (lane & 15);
    // chain: unit cu of tile i (P < U) or of tile i + 1
    constexpr bool kChain = P < U || !kLast;
    constexpr int cu = P < U ? P : P - U, cs = cu / NRT, cr = cu % NRT;
    // the first unit of a sub-tile reads the operand kOperandAhead sub-tiles on (in tile i+1
    // once that passes the tile's end; a chain already in tile i+1 reads within it)
    constexpr int ls = cs + kOperandAhead;
    constexpr bool kNextTile = P < U && ls >= kSubTiles;
    constexpr bool kLoad = kChain && cu % NRT == 0 && !(kNextTile && kLast);
    constexpr int lsub = ls % kSubTiles;
    score_phase16<D, kMaxMean, kMask, kChain, true, kLoad, er>(
        st, qreg[cr], st.kb[cs % kOperandBufs], st.kb[lsub % kOperandBufs], rp,
        (P < U && !kNextTile) ? buf_i : buf_n, lsub, beta[er], prow, key, cx.alpha, cx.G);
    if constexpr (er == NRT - 1) {
      // sub-tile es is complete in this lane: hand its partial to the other waves
      if (!kMaxMean) {
        st.part[3] += st.ex;   // the pending exp2 of the unit's last element
        st.ex = 0.f;
      }
      red[i & (kRedBufs - 1)][w][(lane >> 4) * kRedGrp + es * 16 + (lane & 15)] =
          (st.part[0] + st.part[1]) + (st.part[2] + st.part[3]);
      st.part[0] = st.part[1] = st.part[2] = st.part[3] = 0.f;
    }
    if constexpr (P == kBarrier + 1) {
      // the finish of tile i - 1, whose partials were read a phase ago
      finish_write(cx, fin, i - 1, i > cx.i0);
    }
    tile_phases16<D, kMaxMean, NRT, kMask, kLast, P + 1>(cx, kp, rp, st, qreg, beta, red, i,
                                                          next_page, fin);
  }
}

// Sweep key tiles i0 .. i1-1 of one segment with NRT row tiles per wave.  K tiles stream
// through kScoreStages LDS buffers (direct-to-LDS loads, kScoreStages - 1 tiles ahead),
// one barrier per tile.
template <int D, bool kMaxMean, int NRT>
__device__ __forceinline__ void score_sweep16(const SweepCtx& cx, const KLoadPlan<D, kWaves>& kp,
                                              const bf16x8 (&qreg)[kRowTilesPerWave][Geom16<D>::kSteps],
                                              const float (&beta)[kRowTilesPerWave][4],
                                              RedTile* red) {
  using Gm = TileGeom<D>;
  auto clamp_tile = [&](int t) { return t < cx.i1 ? t : cx.i1 - 1; };
  float4 fin = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int p = 0; p < kScoreStages - 1; ++p) {
    issue_k_tile<D, kWaves>(cx.kl + p * Gm::kTileBytes, cx.kv_bytes,
                            page_of<D, kWaves>(cx.bt_row, cx.L, kp, clamp_tile(cx.i0 + p)),
                            cx.num_pages, cx.page_bytes, kp);
    finish_write(cx, fin, 0, false);   // the store slot of the tile (writes nothing)
  }
  int32_t next_page = page_of<D, kWaves>(cx.bt_row, cx.L, kp,
                                         clamp_tile(cx.i0 + kScoreStages - 1));
  const KRead16 rp = make_k_read16<D>();
  Pipe16<D> st;
  st.part[0] = st.part[1] = st.part[2] = st.part[3] = 0.f;
  st.ex = 0.f;
  st.mx = 0.f;
  st.c1 = f32x4{0.f, 0.f, 0.f, 0.f};
  // prologue: tile i0 in LDS, the last stage filled, operands of the first kOperandAhead
  // sub-tiles, chains of units 0 and 1 (each reading ahead when it starts a sub-tile)
  wait_vmcnt<kTileVmcnt<D>>();
  __builtin_amdgcn_s_barrier();
  issue_k_tile<D, kWaves>(cx.kl + (kScoreStages - 1) * Gm::kTileBytes, cx.kv_bytes, next_page,
                          cx.num_pages, cx.page_bytes, kp);
  finish_write(cx, fin, 0, false);
  next_page = page_of<D, kWaves>(cx.bt_row, cx.L, kp, clamp_tile(cx.i0 + kScoreStages));
#pragma unroll
  for (int sb = 0; sb < kOperandAhead; ++sb)
#pragma unroll
    for (int ks = 0; ks < Geom16<D>::kSteps; ++ks) st.kb[sb][ks] = lds_k16<D>(cx.kbuf, sb, rp, ks);
  score_phase16<D, kMaxMean, false, true, false, true, 0>(
      st, qreg[0], st.kb[0], st.kb[kOperandAhead % kOperandBufs], rp, cx.kbuf, kOperandAhead,
      beta[0], nullptr, 0, cx.alpha, cx.G);
  constexpr int s1 = 1 / NRT;   // sub-tile of unit 1
  score_phase16<D, kMaxMean, false, true, false, NRT == 1, 0>(
      st, qreg[1 % NRT], st.kb[s1 % kOperandBufs], st.kb[(s1 + kOperandAhead) % kOperandBufs],
      rp, cx.kbuf, s1 + kOperandAhead, beta[0], nullptr, 0, cx.alpha, cx.G);
  for (int i = cx.i0; i < cx.i1; ++i) {
    const bool mask = i * kKeyTile + kKeyTile - 1 > cx.mask_from;
    if (i + 1 < cx.i1) {
      if (mask)
        tile_phases16<D, kMaxMean, NRT, true, false, 2>(cx, kp, rp, st, qreg, beta, red, i, next_page, fin);
      else
        tile_phases16<D, kMaxMean, NRT, false, false, 2>(cx, kp, rp, st, qreg, beta, red, i, next_page, fin);
    } else {
      if (mask)
        tile_phases16<D, kMaxMean, NRT, true, true, 2>(cx, kp, rp, st, qreg, beta, red, i, next_page, fin);
      else
        tile_phases16<D, kMaxMean, NRT, false, true, 2>(cx, kp, rp, st, qreg, beta, red, i, next_page, fin);
    }
  }
  // the last tile's partials
  wait_lgkmcnt0();
  __builtin_amdgcn_s_barrier();
  finish_write(cx, finish_read(red[(cx.i1 - 1) & (kRedBufs - 1)]), cx.i1 - 1, true);
}

// The sweep of a wave whose row tiles hold no real row (few query rows, e.g. one decode
// query per request): the same K loads, barriers and tile finishes as score_sweep16, but no
// MFMA and no epilogue; its partial slots stay zero.
template <int D>
__device__ __forceinline__ void score_sweep_idle(const SweepCtx& cx, const KLoadPlan<D, kWaves>& kp,
                                                 RedTile* red) {
  using Gm = TileGeom<D>;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  // this wave's partial slots of every reduction buffer: zero (no finish of the previous
  // segment reads them any more)
#pragma unroll
  for (int b = 0; b < kRedBufs; ++b)
#pragma unroll
    for (int es = 0; es < kSubTiles; ++es)
      red[b][w][(lane >> 4) * kRedGrp + es * 16 + (lane & 15)] = 0.f;
  auto clamp_tile = [&](int t) { return t < cx.i1 ? t : cx.i1 - 1; };
#pragma unroll
  for (int p = 0; p < kScoreStages - 1; ++p)
    issue_k_tile<D, kWaves>(cx.kl + p * Gm::kTileBytes, cx.kv_bytes,
                            page_of<D, kWaves>(cx.bt_row, cx.L, kp, clamp_tile(cx.i0 + p)),
                            cx.num_pages, cx.page_bytes, kp);
  int32_t next_page = page_of<D, kWaves>(cx.bt_row, cx.L, kp,
                                         clamp_tile(cx.i0 + kScoreStages - 1));
  wait_vmcnt<(kScoreStages - 2) * Gm::kLoadsPerWave>();
  wait_lgkmcnt0();
  __builtin_amdgcn_s_barrier();
  issue_k_tile<D, kWaves>(cx.kl + (kScoreStages - 1) * Gm::kTileBytes, cx.kv_bytes, next_page,
                          cx.num_pages, cx.page_bytes, kp);
  next_page = page_of<D, kWaves>(cx.bt_row, cx.L, kp, clamp_tile(cx.i0 + kScoreStages));
  for (int i = cx.i0; i < cx.i1; ++i) {
    // the barrier phase of tile i, as in tile_phases16
    const int st_i = (i - cx.i0) & (kScoreStages - 1);
    wait_vmcnt<(kScoreStages - 2) * Gm::kLoadsPerWave>();
    wait_lgkmcnt0();
    __builtin_amdgcn_s_barrier();
    issue_k_tile<D, kWaves>(cx.kl + st_i * Gm::kTileBytes, cx.kv_bytes, next_page, cx.num_pages,
                            cx.page_bytes, kp);
    const int nt = i + kScoreStages + 1;
    next_page = page_of<D, kWaves>(cx.bt_row, cx.L, kp, nt < cx.i1 ? nt : cx.i1 - 1);
    finish_write(cx, finish_read(red[(i - 1) & (kRedBufs - 1)]), i - 1, i > cx.i0);
  }
  wait_lgkmcnt0();
  __builtin_amdgcn_s_barrier();
  finish_write(cx, finish_read(red[(cx.i1 - 1) & (kRedBufs - 1)]), cx.i1 - 1, true);
}

template <int D, bool kMaxMean>
__global__ __launch_bounds__(kThreads, 1) void score_kernel(
    DevProblem dp, const uint16_t* __restrict__ q_ptr, const uint16_t* __restrict__ kv_ptr,
    const int32_t* __restrict__ bt_ptr, const float* __restrict__ lse_ptr,
    float* __restrict__ scores_ptr, float* __restrict__ part_ptr, int64_t num_scores,
    int64_t seg_lo, int64_t seg_hi) {
  if (!plan_ok(dp)) return;   // the workspace holds another problem's plan
  using Gm = TileGeom<D>;
  __shared__ __align__(1024) char kbuf[kScoreStages][Gm::kTileBytes];
  __shared__ __align__(16) float beta_s[kRowsPerChunk];
  __shared__ __align__(16) int32_t pos_s[kRowsPerChunk];
  __shared__ RedTile red[kRedBufs];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int G = dp.G, Hq = dp.Hq, Hkv = dp.Hkv, C = dp.max_chunks;
  const bool grouped = kMaxMean && (G == 8 || G == 16);
  // this launch scores segments [seg_lo, seg_hi) (whole requests: a request's segments are
  // consecutive); workgroup b takes the b-th equal share of their cost
  const int64_t base = dp.seg_cost[seg_lo], total = dp.seg_cost[seg_hi] - base;
  const int64_t c0 = base + total * blockIdx.x / gridDim.x;
  const int64_t c1 = base + total * (blockIdx.x + 1) / gridDim.x;
  if (c0 >= c1) return;

  SweepCtx cx;
  cx.kv_bytes = reinterpret_cast<const char*>(kv_ptr);
  cx.pos_s = pos_s;
  cx.kbuf = &kbuf[0][0];
  cx.kl = (uint32_t)(uintptr_t)(lds_char*)&kbuf[0][0];
  cx.page_bytes = (int64_t)kPageSize * Hkv * D * 2;
  cx.num_pages = dp.num_pages;
  cx.G = G;
  cx.alpha = dp.sm_scale * kLog2e;

  // first segment: the largest s with seg_cost[s] <= c0 (it is never empty)
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
    // cost of each of the segment's key tiles (the unit of the split over workgroups)
    const int64_t TC = score_tile_cost(chunk_row_tiles(M, c));
    const int64_t ntiles = ceil_div64(L, kKeyTile);
    int64_t i1 = (c1 - cs + TC - 1) / TC;
    if (i1 > ntiles) i1 = ntiles;
    cx.i0 = first ? (int)((c0 - cs + TC - 1) / TC) : 0;   // c0 < ce: below ntiles
    cx.i1 = (int)i1;
    first = false;
    if (cx.i0 >= cx.i1) continue;

    // ---- segment setup: beta / causal position of every row, Q rows into registers
    wait_vmcnt<0>();   // no load of the previous segment may still land in a K buffer
    __syncthreads();
    for (int m = tid; m < kRowsPerChunk; m += kThreads) {
      int j, g;
      score_row_query(G, grouped, c, m / kRowTile, m % kRowTile, &j, &g);
      beta_s[m] = j < n ? lse_ptr[(int64_t)(pl.q_off + j) * Hq + h * G + g] * kLog2e
                        : __builtin_inff();
      pos_s[m] = dp.causal ? L - n + j : L - 1;
    }
    bf16x8 qreg[kRowTilesPerWave][Geom16<D>::kSteps];
#pragma unroll
    for (int rt = 0; rt < kRowTilesPerWave; ++rt)
      load_q16<D>(qreg[rt], q_ptr, G, grouped, Hq, h, pl.q_off, n, c, w + kWaves * rt);
    cx.bt_row = bt_ptr + (int64_t)r * dp.bt_stride;
    cx.L = L;
    cx.mask_from = dp.causal ? L - n : L;  // keys past this may be hidden from some rows
    cx.out_scale = (kMaxMean && pl.nchunk == 1) ? (n > 0 ? 1.0f / n : 0.0f) : 1.0f;
    cx.out = buffer_over_uniform((c == 0) ? scores_ptr + pl.seg_off + (int64_t)h * L
                                          : part_ptr + (int64_t)(c - 1) * num_scores +
                                                pl.seg_off + (int64_t)h * L,
                                 L * (int)sizeof(float));
    const KLoadPlan<D, kWaves> kp = make_k_load_plan<D, kWaves>(h, Hkv);
    // every ordinary load of the setup has landed before the K pipeline starts, so the
    // sweep needs no compiler-inserted wait on the vector-memory queue
    wait_vmcnt<0>();
    __syncthreads();   // beta_s / pos_s visible
    // beta of this lane's rows (4*(l/16) + i of each row tile): fixed for the sweep
    float beta[kRowTilesPerWave][4];
#pragma unroll
    for (int rt = 0; rt < kRowTilesPerWave; ++rt) {
      const float4 b4 = *reinterpret_cast<const float4*>(beta_s + (w + kWaves * rt) * kRowTile +
                                                         4 * (lane >> 4));
      beta[rt][0] = b4.x; beta[rt][1] = b4.y; beta[rt][2] = b4.z; beta[rt][3] = b4.w;
    }
    // row tiles past the chunk's real rows are all padding (Q = 0, beta = +inf): every
    // wave runs only as many row tiles as can hold real rows
    const int nrt = chunk_wave_tiles(G, grouped, n, c);
    // a wave none of whose row tiles holds a real row keeps the schedule but does no work
    bool real = false;
    for (int rt = 0; rt < (nrt < kRowTilesPerWave ? nrt : kRowTilesPerWave); ++rt) {
      int j, g;
      score_row_query(G, grouped, c, w + kWaves * rt, lane & 15, &j, &g);
      real = real || j < n;
    }
    if (__ballot(real) == 0ull) {
      score_sweep_idle<D>(cx, kp, red);
    } else {
      switch (nrt < kRowTilesPerWave ? nrt : kRowTilesPerWave) {
        case 1: score_sweep16<D, kMaxMean, 1>(cx, kp, qreg, beta, red); break;
        case 2: score_sweep16<D, kMaxMean, 2>(cx, kp, qreg, beta, red); break;
        case 3: score_sweep16<D, kMaxMean, 3>(cx, kp, qreg, beta, red); break;
        case 4: score_sweep16<D, kMaxMean, 4>(cx, kp, qreg, beta, red); break;
        case 5: score_sweep16<D, kMaxMean, 5>(cx, kp, qreg, beta, red); break;
        case 6: score_sweep16<D, kMaxMean, 6>(cx, kp, qreg, beta, red); break;
        case 7: score_sweep16<D, kMaxMean, 7>(cx, kp, qreg, beta, red); break;
        default: score_sweep16<D, kMaxMean, 8>(cx, kp, qreg, beta, red); break;
      }
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
    if (mm) hipLaunchKernelGGL((score_kernel<128, true>), dim3(grid), dim3(kThreads), 0, s, dp, qq, kk, bt, lse, scores, score_part, n, seg_lo, seg_hi);
    else hipLaunchKernelGGL((score_kernel<128, false>), dim3(grid), dim3(kThreads), 0, s, dp, qq, kk, bt, lse, scores, score_part, n, seg_lo, seg_hi);
  } else {
    if (mm) hipLaunchKernelGGL((score_kernel<64, true>), dim3(grid), dim3(kThreads), 0, s, dp, qq, kk, bt, lse, scores, score_part, n, seg_lo, seg_hi);
    else hipLaunchKernelGGL((score_kernel<64, false>), dim3(grid), dim3(kThreads), 0, s, dp, qq, kk, bt, lse, scores, score_part, n, seg_lo, seg_hi);
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
  // with at most one query a request's cost is Hkv x its 64-key tiles (one row tile), so
  // one query per request: every tile costs score_tile_cost(1), so
  // seg_cost[r * Hkv] / (Hkv * score_tile_cost(1)) is the number of tiles before request r
  auto tiles_before = [&](int rr) {
    return dp.seg_cost[(int64_t)rr * Hkv] / (Hkv * score_tile_cost(1));
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
  const int64_t tiles = hp.score_cost / (hp.Hkv * score_tile_cost(1));   // (request, key tile) pairs
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
          // the running max on the raw dot products (alpha > 0 keeps the order), then
          // 2^(alpha x - m) with the scale and the shift in one FMA
          float mx = -__builtin_inff();
          if (masked) {
#pragma unroll
            for (int v = 0; v < 16; ++v) {
              const int key = keybase + 8 * (v / 4) + (v % 4);
              x[v] = key <= pos[ti] ? x[v] : -__builtin_inff();
              mx = fmaxf(mx, x[v]);
            }
          } else {
#pragma unroll
            for (int v = 0; v < 16; ++v) mx = fmaxf(mx, x[v]);
          }
          const float m = fmaxf(rm[ti], mx * alpha);
          if (m != -__builtin_inff()) {
            float sum = rs[ti] * fast_exp2(rm[ti] - m);
#pragma unroll
            for (int v = 0; v < 16; ++v) sum += fast_exp2(__builtin_fmaf(x[v], alpha, -m));
            rs[ti] = sum;
            rm[ti] = m;
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
