// Per-request planning on the device (integer only): offsets of every ragged array,
// the untouched-request rule, fresh / freed page counts (Alg. 4 steps 1-5 count the same
// quantities per request) and the scoring cost prefix used to balance the scoring grid.
#include "device_common.hpp"

namespace actkv {

namespace {

// Exclusive prefix sums of N values at once over the block (blockDim.x a multiple of 64,
// <= 1024): wave scans, then every thread adds up the totals of the waves before its own
// (broadcast LDS reads).  v is replaced by its exclusive prefix, tot gets the block sums.
template <int N>
__device__ __forceinline__ void block_excl_scan_n(int64_t (&v)[N], int64_t (*tmp)[N],
                                                  int64_t (&tot)[N]) {
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x / kWave;
  const int nw = blockDim.x / kWave;
  int64_t inc[N];
#pragma unroll
  for (int i = 0; i < N; ++i) inc[i] = wave_incl_scan_i64(v[i]);
  if (lane == kWave - 1) {
#pragma unroll
    for (int i = 0; i < N; ++i) tmp[w][i] = inc[i];
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < N; ++i) {
    int64_t before = 0, all = 0;
    for (int u = 0; u < nw; ++u) {
      const int64_t t = tmp[u][i];
      before += u < w ? t : 0;
      all += t;
    }
    tot[i] = all;
    v[i] = before + inc[i] - v[i];
  }
  __syncthreads();   // tmp is written again by the next call
}

}  // namespace

__global__ __launch_bounds__(1024) void plan_kernel(DevProblem dp) {
  constexpr int kScans = 8;
  __shared__ int64_t tmp[1024 / kWave][kScans];
  const int R = dp.R, Hkv = dp.Hkv, G = dp.G, C = dp.max_chunks;
  int64_t carry_n = 0, carry_L = 0, carry_X = 0, carry_Y = 0, carry_k = 0, carry_cost = 0,
          carry_lse = 0, carry_ip = 0;
  for (int base = 0; base < R; base += blockDim.x) {
    const int r = base + threadIdx.x;
    const bool ok = r < R;
    int32_t L = 0, n = 0, X = 0, Y = 0, skip = 1, nchunk = 1, lse_blocks = 0;
    int64_t ksum = 0, cost = 0;
    if (ok) {
      L = dp.seq_lens[r];
      n = dp.q_lens[r];
      int32_t kmax = 0, bmin = INT32_MAX;
      // budgets 8 at a time, every load of a batch issued before any is used
      for (int h0 = 0; h0 < Hkv; h0 += 8) {
        int32_t bb[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) bb[u] = h0 + u < Hkv ? dp.budgets[r * Hkv + h0 + u] : INT32_MAX;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          if (h0 + u >= Hkv) break;
          const int32_t b = bb[u];
          const int32_t k = b < L ? b : L;
          ksum += k;
          kmax = k > kmax ? k : kmax;
          bmin = b < bmin ? b : bmin;
        }
      }
      skip = bmin >= L;
      X = skip ? 0 : ceil_div(kmax, kPageSize);
      Y = skip ? 0 : ceil_div(L, kPageSize);
      const int M = G * n;
      nchunk = M > 0 ? ceil_div(M, kRowsPerChunk) : 1;
      const int64_t ntiles = ceil_div64(L, kKeyTile);
      for (int c = 0; c < nchunk; ++c) {
        const int rows = M - c * kRowsPerChunk;
        const int rt = (int)chunk_units(rows);
        cost += ntiles * score_tile_cost(rt) * Hkv;
      }
      lse_blocks = (int32_t)ceil_div64(L, kLseKeysPerBlock);
    }
    int64_t sv[kScans] = {n, (int64_t)L * Hkv, X, Y, ksum, cost, (int64_t)n * dp.Hq * lse_blocks,
                          Y - X};
    int64_t tot[kScans];
    block_excl_scan_n<kScans>(sv, tmp, tot);
    const int64_t q_off = carry_n + sv[0], seg_off = carry_L + sv[1], x_off = carry_X + sv[2],
                  y_off = carry_Y + sv[3], k_off = carry_k + sv[4], c_off = carry_cost + sv[5],
                  l_off = carry_lse + sv[6], f_off = carry_ip + sv[7];
    carry_n += tot[0]; carry_L += tot[1]; carry_X += tot[2]; carry_Y += tot[3];
    carry_k += tot[4]; carry_cost += tot[5]; carry_lse += tot[6]; carry_ip += tot[7];
    if (ok) {
      ReqPlan p;
      p.L = L; p.n = n; p.X = X; p.Y = Y; p.skip = skip; p.nchunk = nchunk;
      p.q_off = (int32_t)q_off; p.fresh_off = (int32_t)x_off; p.freed_off = (int32_t)y_off;
      p.lse_blocks = lse_blocks; p.seg_off = seg_off; p.lse_part_off = l_off;
      p.ip_freed_off = (int32_t)f_off;
      dp.plan[r] = p;
      dp.req_done[r] = 0;
      // kept offsets per (r, h)
      int64_t ko = k_off;
      for (int h0 = 0; h0 < Hkv; h0 += 8) {
        int32_t bb[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) bb[u] = h0 + u < Hkv ? dp.budgets[r * Hkv + h0 + u] : 0;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          if (h0 + u >= Hkv) break;
          dp.kept_off[r * Hkv + h0 + u] = ko;
          ko += bb[u] < L ? bb[u] : L;
        }
      }
      // scoring cost prefix per segment (r, c, h), c < max_chunks
      const int M = G * n;
      const int64_t ntiles = ceil_div64(L, kKeyTile);
      int64_t co = c_off;
      for (int c = 0; c < C; ++c) {
        for (int h = 0; h < Hkv; ++h) {
          dp.seg_cost[((int64_t)r * C + c) * Hkv + h] = co;
          if (c < nchunk) {
            const int rows = M - c * kRowsPerChunk;
            const int rt = (int)chunk_units(rows);
            co += ntiles * score_tile_cost(rt);
          }
        }
      }
    }
  }
  if (threadIdx.x == 0) {
    dp.kept_off[(int64_t)R * Hkv] = carry_k;
    dp.seg_cost[dp.num_segments] = carry_cost;
    *dp.plan_sig = dp.sig;   // the plan now belongs to this problem
  }
}

hipError_t launch_plan(const DevProblem& dp, hipStream_t s) {
  // one workgroup; as many waves as the requests need (a scan step per 1024 requests)
  int threads = (dp.R + kWave - 1) / kWave * kWave;
  threads = threads < kWave ? kWave : (threads > 1024 ? 1024 : threads);
  hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(threads), 0, s, dp);
  return hipGetLastError();
}

}  // namespace actkv
