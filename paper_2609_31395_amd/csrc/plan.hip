// Per-request planning on the device (integer only): offsets of every ragged array,
// the untouched-request rule, fresh / freed page counts (Alg. 4 steps 1-5 count the same
// quantities per request) and the scoring cost prefix used to balance the scoring grid.
#include "device_common.hpp"

namespace actkv {

__global__ __launch_bounds__(1024) void plan_kernel(DevProblem dp) {
  __shared__ int64_t tmp[17];
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
      for (int h = 0; h < Hkv; ++h) {
        const int32_t b = dp.budgets[r * Hkv + h];
        const int32_t k = b < L ? b : L;
        ksum += k;
        kmax = k > kmax ? k : kmax;
        bmin = b < bmin ? b : bmin;
      }
      skip = bmin >= L;
      X = skip ? 0 : ceil_div(kmax, kPageSize);
      Y = skip ? 0 : ceil_div(L, kPageSize);
      const int M = G * n;
      nchunk = M > 0 ? ceil_div(M, kRowsPerChunk) : 1;
      const int64_t ntiles = ceil_div64(L, kKeyTile);
      for (int c = 0; c < nchunk; ++c) {
        const int rows = M - c * kRowsPerChunk;
        const int rt = rows <= 0 ? 1 : ceil_div(rows < kRowsPerChunk ? rows : kRowsPerChunk, 32);
        cost += ntiles * rt * Hkv;
      }
      lse_blocks = (int32_t)ceil_div64(L, kLseKeysPerBlock);
    }
    int64_t tot;
    const int64_t q_off = carry_n + block_excl_scan_i64(n, tmp, &tot); carry_n += tot;
    const int64_t seg_off = carry_L + block_excl_scan_i64((int64_t)L * Hkv, tmp, &tot); carry_L += tot;
    const int64_t x_off = carry_X + block_excl_scan_i64(X, tmp, &tot); carry_X += tot;
    const int64_t y_off = carry_Y + block_excl_scan_i64(Y, tmp, &tot); carry_Y += tot;
    const int64_t k_off = carry_k + block_excl_scan_i64(ksum, tmp, &tot); carry_k += tot;
    const int64_t c_off = carry_cost + block_excl_scan_i64(cost, tmp, &tot); carry_cost += tot;
    const int64_t l_off = carry_lse + block_excl_scan_i64((int64_t)n * dp.Hq * lse_blocks, tmp, &tot);
    carry_lse += tot;
    const int64_t f_off = carry_ip + block_excl_scan_i64(Y - X, tmp, &tot);
    carry_ip += tot;
    if (ok) {
      ReqPlan p;
      p.L = L; p.n = n; p.X = X; p.Y = Y; p.skip = skip; p.nchunk = nchunk;
      p.q_off = (int32_t)q_off; p.fresh_off = (int32_t)x_off; p.freed_off = (int32_t)y_off;
      p.lse_blocks = lse_blocks; p.seg_off = seg_off; p.lse_part_off = l_off;
      p.ip_freed_off = (int32_t)f_off;
      dp.plan[r] = p;
      // kept offsets per (r, h)
      int64_t ko = k_off;
      for (int h = 0; h < Hkv; ++h) {
        dp.kept_off[r * Hkv + h] = ko;
        const int32_t b = dp.budgets[r * Hkv + h];
        ko += b < L ? b : L;
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
            const int rt = rows <= 0 ? 1 : ceil_div(rows < kRowsPerChunk ? rows : kRowsPerChunk, 32);
            co += ntiles * rt;
          }
        }
      }
    }
  }
  if (threadIdx.x == 0) {
    dp.kept_off[(int64_t)R * Hkv] = carry_k;
    dp.seg_cost[dp.num_segments] = carry_cost;
  }
}

hipError_t launch_plan(const DevProblem& dp, hipStream_t s) {
  hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(1024), 0, s, dp);
  return hipGetLastError();
}

}  // namespace actkv
