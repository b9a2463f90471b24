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

constexpr int kThreads = 512;   // 8 waves: two per SIMD at one workgroup per CU
constexpr int kWaves = kThreads / 64;
constexpr int kTilesPerWave = kRowsPerChunk / 32 / kWaves;   // 2 row tiles of 32 rows

template <int D>
struct TileGeom {
  static constexpr int kSteps = D / 16;                 // MFMA k-steps per row
  static constexpr int kChunksPerRow = D / 8;           // 16-byte chunks per K row
  static constexpr int kLoadsPerThread = kKeyTile * kChunksPerRow / kThreads;
  static constexpr int kStride = D * 2 + 16;            // padded LDS row (bytes)
  static constexpr int kTileBytes = kKeyTile * kStride;
};

// Global loads of K tile `tile` (keys 64*tile ..) of request r, head h into registers.
template <int D>
__device__ __forceinline__ void load_k_tile(u32x4 (&pre)[TileGeom<D>::kLoadsPerThread],
                                            const uint16_t* __restrict__ kv,
                                            const int32_t* __restrict__ bt_row, int L, int h,
                                            int Hkv, int64_t num_pages, int64_t tile) {
  using Gm = TileGeom<D>;
#pragma unroll
  for (int u = 0; u < Gm::kLoadsPerThread; ++u) {
    const int q = threadIdx.x + kThreads * u;
    const int row = q / Gm::kChunksPerRow, ch = q % Gm::kChunksPerRow;
    const int64_t key = tile * kKeyTile + row;
    const int64_t page = key < L ? (int64_t)bt_row[key / kPageSize] : -1;
    // a page outside the pool is never dereferenced (its keys read as zero)
    if (page >= 0 && page < num_pages) {
      const uint16_t* src =
          kv + ((page * kPageSize + key % kPageSize) * Hkv + h) * (int64_t)D + ch * 8;
      pre[u] = *reinterpret_cast<const u32x4*>(src);
    } else {
      pre[u] = u32x4{0u, 0u, 0u, 0u};
    }
  }
}

template <int D>
__device__ __forceinline__ void store_k_tile(const u32x4 (&pre)[TileGeom<D>::kLoadsPerThread],
                                             char* buf) {
  using Gm = TileGeom<D>;
#pragma unroll
  for (int u = 0; u < Gm::kLoadsPerThread; ++u) {
    const int q = threadIdx.x + kThreads * u;
    const int row = q / Gm::kChunksPerRow, ch = q % Gm::kChunksPerRow;
    *reinterpret_cast<u32x4*>(buf + row * Gm::kStride + ch * 16) = pre[u];
  }
}

// The 32x32 MFMA operand of key sub-tile `sub` (32 keys) for every k-step: lane l holds key
// sub*32 + l%32, head-dim elements 16*ks + 8*(l/32) .. +8.
template <int D>
__device__ __forceinline__ void read_k_operand(bf16x8 (&kreg)[TileGeom<D>::kSteps],
                                               const char* buf, int sub) {
  using Gm = TileGeom<D>;
  const int lane = threadIdx.x & 63;
  const char* row = buf + (sub * 32 + (lane & 31)) * Gm::kStride + (lane >> 5) * 16;
#pragma unroll
  for (int ks = 0; ks < Gm::kSteps; ++ks)
    kreg[ks] = as_bf16x8(*reinterpret_cast<const u32x4*>(row + ks * 32));
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

struct ScoreArgs {
  DevProblem dp;
  const uint16_t* q;
  const uint16_t* kv;
  const int32_t* bt;
  const float* lse;
  float* scores;
  float* score_part;
  int64_t num_scores;
};

}  // namespace

template <int D, bool kMaxMean>
__global__ __launch_bounds__(kThreads, 1) void score_kernel(ScoreArgs a) {
  using Gm = TileGeom<D>;
  __shared__ __align__(16) char kbuf[2][Gm::kTileBytes];
  __shared__ __align__(16) float beta_s[kRowsPerChunk];
  __shared__ __align__(16) int32_t pos_s[kRowsPerChunk];
  __shared__ float red[2][kWaves][kKeyTile];

  const DevProblem& dp = a.dp;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, hf = lane >> 5, l32 = lane & 31;
  const int G = dp.G, Hq = dp.Hq, Hkv = dp.Hkv, C = dp.max_chunks;
  const float alpha = dp.sm_scale * kLog2e;
  const int64_t nseg = dp.num_segments;
  const int64_t total = dp.seg_cost[nseg];
  const int64_t c0 = total * blockIdx.x / gridDim.x, c1 = total * (blockIdx.x + 1) / gridDim.x;
  if (c0 >= c1) return;

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
    const int64_t i0 = first ? (c0 - cs + RT - 1) / RT : 0;
    int64_t i1 = (c1 - cs + RT - 1) / RT;
    if (i1 > ntiles) i1 = ntiles;
    first = false;
    if (i0 >= i1) continue;

    // ---- segment setup: beta / causal position of every row, Q rows into registers
    __syncthreads();  // LDS of the previous segment no longer in use
    for (int m = tid; m < kRowsPerChunk; m += kThreads) {
      int j, g;
      row_to_query(G, c, m / 32, m % 32, &j, &g);
      beta_s[m] = j < n ? a.lse[(int64_t)(pl.q_off + j) * Hq + h * G + g] * kLog2e
                        : __builtin_inff();
      pos_s[m] = dp.causal ? L - n + j : L - 1;
    }
    bf16x8 qreg[kTilesPerWave][Gm::kSteps];
#pragma unroll
    for (int ti = 0; ti < kTilesPerWave; ++ti)
      if (w + kWaves * ti < RT) load_q_tile<D>(qreg[ti], a.q, G, Hq, h, pl.q_off, n, c, w + kWaves * ti);
    const int32_t* bt_row = a.bt + (int64_t)r * dp.bt_stride;
    const float out_scale = (kMaxMean && pl.nchunk == 1) ? (n > 0 ? 1.0f / n : 0.0f) : 1.0f;
    float* out = (c == 0) ? a.scores + pl.seg_off + (int64_t)h * L
                          : a.score_part + (int64_t)(c - 1) * a.num_scores + pl.seg_off +
                                (int64_t)h * L;
    const int mask_from = dp.causal ? L - n : L;  // keys past this may be hidden from rows

    u32x4 pre[Gm::kLoadsPerThread];
    load_k_tile<D>(pre, a.kv, bt_row, L, h, Hkv, dp.num_pages, i0);
    store_k_tile<D>(pre, kbuf[0]);
    __syncthreads();
    // beta of this lane's 16 rows per row tile: rows 8*aa + 4*hf + i
    float beta[kTilesPerWave][16];
#pragma unroll
    for (int ti = 0; ti < kTilesPerWave; ++ti) {
      const float* brow = beta_s + (w + kWaves * ti) * 32 + 4 * hf;
#pragma unroll
      for (int aa = 0; aa < 4; ++aa) {
        const float4 b4 = (w + kWaves * ti < RT) ? *reinterpret_cast<const float4*>(brow + 8 * aa)
                                                 : make_float4(0.f, 0.f, 0.f, 0.f);
        beta[ti][4 * aa + 0] = b4.x; beta[ti][4 * aa + 1] = b4.y;
        beta[ti][4 * aa + 2] = b4.z; beta[ti][4 * aa + 3] = b4.w;
      }
    }

    // ---- pipelined sweep over key tiles i0 .. i1-1
    int buf = 0;
    for (int64_t i = i0; i < i1; ++i) {
      const bool has_next = i + 1 < i1;
      if (has_next) load_k_tile<D>(pre, a.kv, bt_row, L, h, Hkv, dp.num_pages, i + 1);
      const int64_t key0 = i * kKeyTile;
      const bool needs_mask = key0 + kKeyTile - 1 > mask_from;
#pragma unroll
      for (int sub = 0; sub < 2; ++sub) {
        bf16x8 kreg[Gm::kSteps];
        read_k_operand<D>(kreg, kbuf[buf], sub);
        const int key = (int)(key0 + sub * 32 + l32);
        float sacc0 = 0.f, sacc1 = 0.f;
#pragma unroll
        for (int ti = 0; ti < kTilesPerWave; ++ti) {
          const int tile = w + kWaves * ti;
          if (tile < RT) {
            f32x16 p = {};
#pragma unroll
            for (int ks = 0; ks < Gm::kSteps; ++ks) p = mfma32(qreg[ti][ks], kreg[ks], p);
#pragma unroll
            for (int v = 0; v < 16; ++v) p[v] = fast_exp2(__builtin_fmaf(p[v], alpha, -beta[ti][v]));
            if (needs_mask) {
              const int32_t* prow = pos_s + tile * 32 + 4 * hf;
#pragma unroll
              for (int v = 0; v < 16; ++v)
                if (key > prow[8 * (v / 4) + (v % 4)]) p[v] = 0.f;
            }
            if (!kMaxMean) {
#pragma unroll
              for (int v = 0; v < 16; v += 2) { sacc0 += p[v]; sacc1 += p[v + 1]; }
            } else if (G == 16) {
              // the lane's 16 rows are one query's whole group
              float mx = p[0];
#pragma unroll
              for (int v = 1; v < 16; ++v) mx = fmaxf(mx, p[v]);
              sacc0 += mx;
            } else if (G == 8) {
              // registers 0-7 and 8-15 are two queries' groups
              float m0 = p[0], m1 = p[8];
#pragma unroll
              for (int v = 1; v < 8; ++v) { m0 = fmaxf(m0, p[v]); m1 = fmaxf(m1, p[8 + v]); }
              sacc0 += m0; sacc1 += m1;
            } else {
              // registers v0..v0+3 are four consecutive rows of the natural order
#pragma unroll
              for (int v0 = 0; v0 < 16; v0 += 4) {
                if (G == 4) {
                  sacc0 += fmaxf(fmaxf(p[v0], p[v0 + 1]), fmaxf(p[v0 + 2], p[v0 + 3]));
                } else if (G == 2) {
                  sacc0 += fmaxf(p[v0], p[v0 + 1]);
                  sacc1 += fmaxf(p[v0 + 2], p[v0 + 3]);
                } else {
                  sacc0 += p[v0] + p[v0 + 2];
                  sacc1 += p[v0 + 1] + p[v0 + 3];
                }
              }
            }
          }
        }
        float acc = sacc0 + sacc1;
        acc += __shfl_xor(acc, 32, 64);   // lanes l and l+32 hold the same key
        if (hf == 0) red[buf][w][sub * 32 + l32] = acc;
      }
      if (has_next) store_k_tile<D>(pre, kbuf[buf ^ 1]);
      __syncthreads();
      if (tid < kKeyTile) {
        const int64_t key = key0 + tid;
        if (key < L) {
          float v = 0.f;
#pragma unroll
          for (int ww = 0; ww < kWaves; ++ww) v += red[buf][ww][tid];
          out[key] = v * out_scale;
        }
      }
      buf ^= 1;
    }
  }
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
  ScoreArgs a{dp, static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(kv), bt, lse,
              scores, score_part, hp.num_scores};
  int dev = 0, cus = 256;
  if (hipGetDevice(&dev) == hipSuccess) {
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) cus = 256;
  }
  int64_t grid = (int64_t)cus;   // one 8-wave workgroup per CU
  if (grid > hp.score_cost) grid = hp.score_cost > 0 ? hp.score_cost : 1;
  const bool mm = dp.agg == ACTKV_AGG_MAX_MEAN;
  if (dp.D == 128) {
    if (mm) hipLaunchKernelGGL((score_kernel<128, true>), dim3(grid), dim3(kThreads), 0, s, a);
    else hipLaunchKernelGGL((score_kernel<128, false>), dim3(grid), dim3(kThreads), 0, s, a);
  } else {
    if (mm) hipLaunchKernelGGL((score_kernel<64, true>), dim3(grid), dim3(kThreads), 0, s, a);
    else hipLaunchKernelGGL((score_kernel<64, false>), dim3(grid), dim3(kThreads), 0, s, a);
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
__global__ __launch_bounds__(kThreads, 1) void lse_partial_kernel(DevProblem dp, const uint16_t* q,
                                                                  const uint16_t* kv,
                                                                  const int32_t* bt, float2* part) {
  using Gm = TileGeom<D>;
  __shared__ __align__(16) char kbuf[2][Gm::kTileBytes];
  const int kb = blockIdx.x, ch = blockIdx.y / dp.Hkv, h = blockIdx.y % dp.Hkv, r = blockIdx.z;
  const ReqPlan pl = dp.plan[r];
  if (kb >= pl.lse_blocks || ch >= pl.nchunk) return;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, hf = lane >> 5, l32 = lane & 31;
  const int G = dp.G, Hq = dp.Hq, Hkv = dp.Hkv, L = pl.L, n = pl.n, M = G * n;
  const int RT = chunk_row_tiles(M, ch);
  const float alpha = dp.sm_scale * kLog2e;

  bf16x8 qreg[kTilesPerWave][Gm::kSteps];
  int pos[kTilesPerWave];
  float rm[kTilesPerWave], rs[kTilesPerWave];
#pragma unroll
  for (int ti = 0; ti < kTilesPerWave; ++ti) {
    rm[ti] = -__builtin_inff();
    rs[ti] = 0.f;
    pos[ti] = -1;
    const int tile = w + kWaves * ti;
    if (tile < RT) {
      load_q_tile<D>(qreg[ti], q, G, Hq, h, pl.q_off, n, ch, tile);
      int j, g;
      row_to_query(G, ch, tile, l32, &j, &g);
      pos[ti] = j < n ? (dp.causal ? L - n + j : L - 1) : -1;
    }
  }
  const int32_t* bt_row = bt + (int64_t)r * dp.bt_stride;
  const int64_t t0 = (int64_t)kb * (kLseKeysPerBlock / kKeyTile);
  int64_t t1 = t0 + kLseKeysPerBlock / kKeyTile;
  const int64_t ntiles = ceil_div64(L, kKeyTile);
  if (t1 > ntiles) t1 = ntiles;

  u32x4 pre[Gm::kLoadsPerThread];
  load_k_tile<D>(pre, kv, bt_row, L, h, Hkv, dp.num_pages, t0);
  store_k_tile<D>(pre, kbuf[0]);
  __syncthreads();
  int buf = 0;
  for (int64_t i = t0; i < t1; ++i) {
    const bool has_next = i + 1 < t1;
    if (has_next) load_k_tile<D>(pre, kv, bt_row, L, h, Hkv, dp.num_pages, i + 1);
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
      bf16x8 kreg[Gm::kSteps];
      read_k_operand<D>(kreg, kbuf[buf], sub);
      const int keybase = (int)(i * kKeyTile + sub * 32 + 4 * hf);
#pragma unroll
      for (int ti = 0; ti < kTilesPerWave; ++ti) {
        if (w + kWaves * ti < RT) {
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
    if (has_next) store_k_tile<D>(pre, kbuf[buf ^ 1]);
    __syncthreads();
    buf ^= 1;
  }
  // combine the two lanes that share a query row, then write one partial per row
#pragma unroll
  for (int ti = 0; ti < kTilesPerWave; ++ti) {
    const int tile = w + kWaves * ti;
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
    hipLaunchKernelGGL(lse_partial_kernel<128>, grid, dim3(kThreads), 0, s, dp,
                       static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(kv), bt,
                       lse_part);
  else
    hipLaunchKernelGGL(lse_partial_kernel<64>, grid, dim3(kThreads), 0, s, dp,
                       static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(kv), bt,
                       lse_part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(lse_merge_kernel, dim3(hp.R), dim3(256), 0, s, dp, lse_part, lse_out);
  return hipGetLastError();
}

}  // namespace actkv
