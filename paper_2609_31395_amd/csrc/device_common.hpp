// Device helpers for the libactkv kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "actkv_internal.h"

namespace actkv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr float kLog2e = 1.4426950408889634f;

__device__ __forceinline__ int64_t ceil_div64(int64_t a, int64_t b) { return (a + b - 1) / b; }
__device__ __forceinline__ int ceil_div(int a, int b) { return (a + b - 1) / b; }

// C += A(32x16) * B(16x32), bf16 inputs, fp32 accumulate.  Lane l holds A row l%32 and
// B column l%32, each with k = 8*(l/32) .. +8; C column l%32, rows 8*(v/4)+4*(l/32)+v%4.
__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// C += A(16x32) * B(32x16), bf16 inputs, fp32 accumulate.  Lane l holds A row l%16 and
// B column l%16, each with k = 8*(l/16) .. +8; C column l%16, rows 4*(l/16) + v.
__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// True when the workspace holds this problem's plan.  Every kernel that reads the plan
// checks this first and returns at once (the whole workgroup) when it does not hold: a
// caller that claims a plan it does not have gets no output, never an access outside its
// buffers.
__device__ __forceinline__ bool plan_ok(const DevProblem& dp) {
  return __builtin_amdgcn_readfirstlane((uint32_t)(*dp.plan_sig == dp.sig)) != 0u;
}

// Word 3 of a raw (stride 0) buffer resource on CDNA: 32-bit data format; reads at byte
// offsets at or past num_records return 0 and writes there are dropped.
constexpr int kBufferRsrcWord3 = 0x00020000;

// A raw buffer resource over `bytes` bytes at p.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_over(const void* p, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, bytes,
                                           kBufferRsrcWord3);
}

// The same for a pointer and size that every lane of the wave holds, taken from the first
// lane: the compiler then keeps the resource in scalar registers (a resource it cannot
// prove uniform is applied lane group by lane group, in a loop).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_over_uniform(const void* p, int bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
  return buffer_over(reinterpret_cast<const void*>(((uint64_t)hi << 32) | lo),
                     __builtin_amdgcn_readfirstlane(bytes));
}

// One DPP step on a 64-bit value (both halves moved by the same lane pattern); lanes with
// no source, and lanes of rows outside kRowMask, read 0.
template <int kCtrl, int kRowMask>
__device__ __forceinline__ int64_t dpp_i64(int64_t v) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)v, kCtrl, kRowMask,
                                                            0xf, false);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(
      0, (int)(uint32_t)((uint64_t)v >> 32), kCtrl, kRowMask, 0xf, false);
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// The 64-bit value of lane `lane` (wave-uniform) for every lane.
__device__ __forceinline__ int64_t readlane_i64(int64_t v, int lane) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, lane);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)v >> 32), lane);
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// Inclusive prefix sum over one wave (64 lanes) of a 64-bit value: shifts by 1, 2, 4 and 8
// lanes within each row of 16, then the last lane of row 0 (row 2) is added into row 1
// (row 3), and the last lane of row 1 into rows 2 and 3.
__device__ __forceinline__ int64_t wave_incl_scan_i64(int64_t v) {
  v += dpp_i64<0x111, 0xf>(v);   // row_shr:1
  v += dpp_i64<0x112, 0xf>(v);   // row_shr:2
  v += dpp_i64<0x114, 0xf>(v);   // row_shr:4
  v += dpp_i64<0x118, 0xf>(v);   // row_shr:8
  v += dpp_i64<0x142, 0xa>(v);   // row_bcast:15 into rows 1 and 3
  v += dpp_i64<0x143, 0xc>(v);   // row_bcast:31 into rows 2 and 3
  return v;
}

// Exclusive prefix sum over the whole block (blockDim.x a multiple of 64, <= 1024).
// `tmp` is __shared__ int64_t[16 + 1].  Returns the exclusive prefix; *total the sum.  Every
// thread adds up the wave totals itself (broadcast LDS reads), so there is no serial step.
__device__ __forceinline__ int64_t block_excl_scan_i64(int64_t v, int64_t* tmp, int64_t* total) {
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x / kWave;
  const int nw = blockDim.x / kWave;
  const int64_t inc = wave_incl_scan_i64(v);
  if (lane == kWave - 1) tmp[w] = inc;
  __syncthreads();
  // lanes 0..nw-1 of every wave pick up the wave totals and scan them within the first row
  int64_t t = lane < nw ? tmp[lane] : 0;
  t += dpp_i64<0x111, 0xf>(t);
  t += dpp_i64<0x112, 0xf>(t);
  t += dpp_i64<0x114, 0xf>(t);
  t += dpp_i64<0x118, 0xf>(t);
  const int64_t all = readlane_i64(t, nw - 1);
  const int64_t before = w > 0 ? readlane_i64(t, w > 0 ? w - 1 : 0) : 0;
  __syncthreads();   // tmp may be written again right after
  *total = all;
  return before + inc - v;
}

// Exclusive prefix count of a per-thread flag across the block, in thread order.
// `tmp` is __shared__ uint32_t[16 + 1].
__device__ __forceinline__ uint32_t block_excl_count(bool flag, uint32_t* tmp, uint32_t* total) {
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x / kWave;
  const int nw = blockDim.x / kWave;
  const uint64_t bal = __ballot(flag);
  const uint32_t below = __popcll(bal & ((lane == 0) ? 0ull : (~0ull >> (kWave - lane))));
  if (lane == 0) tmp[w] = (uint32_t)__popcll(bal);
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t acc = 0;
    for (int i = 0; i < nw; ++i) { uint32_t t = tmp[i]; tmp[i] = acc; acc += t; }
    tmp[16] = acc;
  }
  __syncthreads();
  uint32_t ex = tmp[w] + below;
  *total = tmp[16];
  __syncthreads();
  return ex;
}

// Map a query row of chunk `chunk`, tile `tile`, tile-local row `mm` (0..31) to its action
// query j and head-in-group g.  For G in {8, 16} the rows of one query are placed so that
// a single lane of the 32x32 MFMA accumulator holds all G of them (needed by MAX_MEAN);
// otherwise row m = j * G + g.
__device__ __forceinline__ void row_to_query(int G, int chunk, int tile, int mm, int* j, int* g) {
  const int m = chunk * kRowsPerChunk + tile * 32 + mm;
  if (G == 8 || G == 16) {
    const int a = mm >> 3, hf = (mm >> 2) & 1, i = mm & 3;
    const int qbase = (chunk * kRowsPerChunk + tile * 32) / G;
    if (G == 8) { *j = qbase + 2 * hf + (a >> 1); *g = 4 * (a & 1) + i; }
    else { *j = qbase + hf; *g = 4 * a + i; }
  } else {
    *j = m / G;
    *g = m % G;
  }
}

}  // namespace actkv
