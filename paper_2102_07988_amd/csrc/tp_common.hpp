// Shared device/host helpers of the stage engine: storage types, bf16
// rounding, wave/block reductions, launch-error plumbing.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/terapipe.h"

namespace tp {

// bf16 is carried as raw 16-bit storage; arithmetic is always fp32.
struct bf16 {
  uint16_t v;
};

__host__ __device__ inline float to_f32(float x) { return x; }
__host__ __device__ inline float to_f32(bf16 x) {
  union {
    uint32_t u;
    float f;
  } c;
  c.u = (uint32_t)x.v << 16;
  return c.f;
}

// Round to nearest, ties to even (the rounding the stage uses for every bf16
// store); NaN stays NaN.
__host__ __device__ inline uint16_t f32_to_bf16_bits(float f) {
  union {
    uint32_t u;
    float f;
  } c;
  c.f = f;
  uint32_t u = c.u;
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// fp16 carried as raw 16-bit storage too (the stage's mixed-precision path
// keeps the operands of the query/key/value product and of the attention
// scores in fp16); conversions round to nearest even.
struct f16s {
  uint16_t v;
};
__host__ __device__ inline uint16_t f32_to_f16_bits(float f) {
  return __builtin_bit_cast(uint16_t, (_Float16)f);
}
__host__ __device__ inline float f16_bits_to_f32(uint16_t b) {
  return (float)__builtin_bit_cast(_Float16, b);
}
__host__ __device__ inline float to_f32(f16s x) { return f16_bits_to_f32(x.v); }

template <typename T>
__host__ __device__ inline T from_f32(float x);
template <>
__host__ __device__ inline float from_f32<float>(float x) {
  return x;
}
template <>
__host__ __device__ inline bf16 from_f32<bf16>(float x) {
  bf16 b;
  b.v = f32_to_bf16_bits(x);
  return b;
}

template <>
__host__ __device__ inline f16s from_f32<f16s>(float x) {
  f16s h;
  h.v = f32_to_f16_bits(x);
  return h;
}

template <typename T>
__device__ inline float ld(const T* p) {
  return to_f32(*p);
}
template <typename T>
__device__ inline void st(T* p, float v) {
  *p = from_f32<T>(v);
}

// GELU, tanh form: 0.5 z (1 + tanh(sqrt(2/pi) (z + 0.044715 z^3))).
__device__ inline float gelu_tanh(float z) {
  const float c = 0.7978845608028654f, a = 0.044715f;
  return 0.5f * z * (1.0f + tanhf(c * (z + a * z * z * z)));
}
__device__ inline float gelu_tanh_grad(float z) {
  const float c = 0.7978845608028654f, a = 0.044715f;
  const float th = tanhf(c * (z + a * z * z * z));
  return 0.5f * (1.0f + th) + 0.5f * z * (1.0f - th * th) * c * (1.0f + 3.0f * a * z * z);
}

__device__ inline float wave_sum(float v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ inline float wave_max(float v) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Block-wide sum for blockDim.x a multiple of 64 (<= 1024).  `red` is LDS of
// >= 16 floats.  Every thread gets the result.
__device__ inline float block_sum(float v, float* red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  v = wave_sum(v);
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float s = 0.f;
  for (int i = 0; i < nw; ++i) s += red[i];
  return s;
}
__device__ inline float block_max(float v, float* red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  v = wave_max(v);
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float s = -INFINITY;
  for (int i = 0; i < nw; ++i) s = fmaxf(s, red[i]);
  return s;
}

// 8 consecutive bf16 values <-> fp32 (16-byte accesses; p 16-byte aligned)
__device__ inline void ld8(const bf16* p, float* x) {
  const uint4 u = *(const uint4*)p;
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[2 * i] = __uint_as_float(w[i] << 16);
    x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
__device__ inline void st8(bf16* p, const float* x) {
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
    w[i] = (uint32_t)f32_to_bf16_bits(x[2 * i]) | ((uint32_t)f32_to_bf16_bits(x[2 * i + 1]) << 16);
  *(uint4*)p = make_uint4(w[0], w[1], w[2], w[3]);
}
__device__ inline void st8(f16s* p, const float* x) {
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
    w[i] = (uint32_t)f32_to_f16_bits(x[2 * i]) | ((uint32_t)f32_to_f16_bits(x[2 * i + 1]) << 16);
  *(uint4*)p = make_uint4(w[0], w[1], w[2], w[3]);
}
__device__ inline void ld8(const float* p, float* x) {
  const float4 a = ((const float4*)p)[0], b = ((const float4*)p)[1];
  x[0] = a.x, x[1] = a.y, x[2] = a.z, x[3] = a.w, x[4] = b.x, x[5] = b.y, x[6] = b.z, x[7] = b.w;
}
__device__ inline void st8(float* p, const float* x) {
  ((float4*)p)[0] = make_float4(x[0], x[1], x[2], x[3]);
  ((float4*)p)[1] = make_float4(x[4], x[5], x[6], x[7]);
}

__host__ __device__ inline int cdiv(long a, long b) { return (int)((a + b - 1) / b); }

// A launch reports its status through hipGetLastError(), which also returns an
// error left behind by any earlier runtime call of the thread (a failed event
// query, say) that nobody read.  Every launcher calls this before its first
// launch, so the status it returns belongs to its own launches.
inline void clear_stale_error() { (void)hipGetLastError(); }

}  // namespace tp
