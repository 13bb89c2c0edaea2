// Small device helpers shared by the SparsePR HIP translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sparsepr_internal.hpp"

namespace sparsepr {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t u) {
  return __uint_as_float(((uint32_t)u) << 16);
}

// Element offset of K/V head bh = b*Hkv + h in the [B, Hkv, N, d] K and V.
__device__ __forceinline__ int64_t kv_base(const Geom& g, int bh) {
  const int b = bh / g.Hkv, h = bh - b * g.Hkv;
  return (int64_t)b * g.kvsb + (int64_t)h * g.kvsh;
}

// Element offset, in the [B, H, N, d] Q and output, of query head j < G of
// K/V head bh: query heads h*G .. h*G + G - 1 share K/V head h.
__device__ __forceinline__ int64_t q_base(const Geom& g, int bh, int j) {
  const int b = bh / g.Hkv, h = bh - b * g.Hkv;
  return (int64_t)b * g.sb + (int64_t)(h * g.G + j) * g.sh;
}

// Load element `idx` of a bf16 or fp32 tensor as float.
__device__ __forceinline__ float load_x(const void* p, int bf16, int64_t idx) {
  if (bf16) return bf16_bits_to_f32(((const uint16_t*)p)[idx]);
  return ((const float*)p)[idx];
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__device__ __forceinline__ int wave_sum_i(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Exclusive prefix sum over `n` ints in LDS array `a` (in place) by the whole
// block; returns the total.  `tmp` needs blockDim.x/64 + 1 ints of LDS.
__device__ inline int block_exclusive_scan(int* a, int n, int* tmp) {
  const int tid = threadIdx.x, nt = blockDim.x;
  const int per = (n + nt - 1) / nt;
  const int lo = min(n, tid * per), hi = min(n, lo + per);
  int s = 0;
  for (int i = lo; i < hi; ++i) s += a[i];
  // inclusive scan of the per-thread sums across the block
  const int lane = tid & 63, wid = tid >> 6, nw = (nt + 63) >> 6;
  int x = s;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) tmp[wid] = x;
  __syncthreads();
  if (tid == 0) {
    int run = 0;
    for (int w = 0; w < nw; ++w) {
      const int t = tmp[w];
      tmp[w] = run;
      run += t;
    }
    tmp[nw] = run;
  }
  __syncthreads();
  int run = tmp[wid] + x - s;  // exclusive start of this thread's segment
  for (int i = lo; i < hi; ++i) {
    const int t = a[i];
    a[i] = run;
    run += t;
  }
  const int total = tmp[nw];
  __syncthreads();
  return total;
}

// Monotone map of a float onto uint32 (larger float -> larger integer).
__device__ __forceinline__ uint32_t float_order_bits(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

}  // namespace sparsepr
