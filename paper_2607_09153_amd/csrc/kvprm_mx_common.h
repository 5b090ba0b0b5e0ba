// Device helpers shared by the matrix-core kernels of libkvprm (projections in kvprm_mfma.hip,
// attention in kvprm_attn.hip): vector types, the streaming load, the MFMA wrapper, bf16 hi/lo
// splitting of fp32 operands, the operand-buffer store and wave/block reductions.
#pragma once

#include "kvprm_internal.h"

namespace kvprm {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// 16-byte load of data that a call reads exactly once (cache pages of the private ranges, weight
// tiles): non-temporal, so the stream does not allocate in the caches and displace lines that
// are reused. Measured on the paged K/V read pattern: 6.5 TB/s instead of 5.6 with plain loads.
__device__ __forceinline__ uint4 ld_stream(const uint4 *p) {
  const u32x4 v = __builtin_nontemporal_load((const u32x4 *)p);
  return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ floatx4 mfma16(const uint4 &a, const uint4 &b, const floatx4 &c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// round-to-nearest-even fp32 -> bf16 bits (finite inputs)
__device__ __forceinline__ uint32_t bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

__device__ __forceinline__ void split_hi_lo(float x, uint32_t &hi, uint32_t &lo) {
  hi = bf16_rne(x);
  lo = bf16_rne(x - __uint_as_float(hi << 16));
}

__device__ __forceinline__ uint32_t pack2(uint32_t a, uint32_t b) { return a | (b << 16); }

// Two fp32 values -> packed bf16 pairs hi (RNE) and lo = RNE(x - hi) (the hardware pack-convert,
// one instruction per pair): hi + lo carries 16 significant bits of each value.
__device__ __forceinline__ void split2(float x0, float x1, uint32_t &hi, uint32_t &lo) {
  typedef __bf16 bf16x2v __attribute__((ext_vector_type(2)));
  typedef float f32x2v __attribute__((ext_vector_type(2)));
  const f32x2v xv = {x0, x1};
  hi = __builtin_bit_cast(uint32_t, __builtin_convertvector(xv, bf16x2v));
  const f32x2v rv = {x0 - __uint_as_float(hi << 16), x1 - __uint_as_float(hi & 0xFFFF0000u)};
  lo = __builtin_bit_cast(uint32_t, __builtin_convertvector(rv, bf16x2v));
}

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ float ld_w(const void *p, size_t i, int wdt) {
  return wdt ? __uint_as_float((uint32_t)((const uint16_t *)p)[i] << 16) : ((const float *)p)[i];
}

// Store v for input k of candidate cand into an operand buffer (hi and lo halves).
__device__ __forceinline__ void store_operand(uint16_t *op, int NT, int Bp, int k, int cand,
                                              float v) {
  uint32_t hi, lo;
  split_hi_lo(v, hi, lo);
  const int kb = k >> 5, c = (k >> 3) & 3, i = k & 7;
  int col = cand;
  op[((size_t)((kb * NT + (col >> 4)) * 64 + c * 16 + (col & 15))) * 8 + i] = (uint16_t)hi;
  col = cand + Bp;
  op[((size_t)((kb * NT + (col >> 4)) * 64 + c * 16 + (col & 15))) * 8 + i] = (uint16_t)lo;
}

__device__ __forceinline__ float wsum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__device__ __forceinline__ float wmax(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
  return v;
}

// Deterministic 256-thread block reductions; every thread receives the result.
__device__ __forceinline__ float bsum(float v, float *red) {
  v = wsum(v);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  return (red[0] + red[1]) + (red[2] + red[3]);
}

__device__ __forceinline__ float ld_bf16(const void *p, size_t i) {
  return __uint_as_float((uint32_t)((const uint16_t *)p)[i] << 16);
}

}  // namespace kvprm
