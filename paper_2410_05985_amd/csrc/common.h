// Shared device helpers of the LayUp HIP library (gfx950 only).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef uint16_t bf16_t;  // bfloat16 bit pattern
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// float -> bfloat16, round to nearest even (NaN stays NaN): the gfx950
// conversion instruction v_cvt_pk_bf16_f32, two values per instruction and no
// branches.
__device__ __forceinline__ bf16_t f2bf(float f) { return __builtin_bit_cast(bf16_t, (__bf16)f); }

__device__ __forceinline__ float bf2f(bf16_t h) {
  return __builtin_bit_cast(float, ((uint32_t)h) << 16);
}

// two floats -> packed bf16 pair (lo in bits 0..15)
__device__ __forceinline__ uint32_t pack_bf2(float lo, float hi) {
  const bf16x2 v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

// e^d to about an ulp with the hardware base-2 exponential (|d| < 87): the
// argument d*log2(e) is split into an integer n and a remainder f in
// [-1/2, 1/2] that carries the product's low bits (log2(e) as a two-float
// sum), so exp2 sees an argument whose rounding error is ~2^-25 absolute.
__device__ __forceinline__ float exp_acc(float d) {
  const float L2E_HI = 1.44269502162933349609375f;       // float nearest log2(e)
  const float L2E_LO = 1.925963033500011079e-08f;        // log2(e) - L2E_HI
  const float n = __builtin_rintf(d * L2E_HI);
  float f = fmaf(d, L2E_HI, -n);
  f = fmaf(d, L2E_LO, f);
  return __builtin_ldexpf(__builtin_amdgcn_exp2f(f), (int)n);
}

__device__ __forceinline__ float warp_sum(float v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ float warp_max(float v) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Block-wide sum for blockDim.x a multiple of 64 and <= 1024.  Every thread
// receives the total.  Fixed order: deterministic for a fixed block size.
__device__ __forceinline__ float block_sum(float v, float* red /* >= 16 floats of LDS */) {
  v = warp_sum(v);
  const int w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float t = 0.f;
  for (int i = 0; i < nw; ++i) t += red[i];
  return t;
}

__device__ __forceinline__ float block_max(float v, float* red) {
  v = warp_max(v);
  const int w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float t = -INFINITY;
  for (int i = 0; i < nw; ++i) t = fmaxf(t, red[i]);
  return t;
}

static inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
