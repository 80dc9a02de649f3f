// Device helpers of the step kernels: 16-bit conversions, MFMA wrappers and
// the target-margin formulas.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "pfc_internal.h"

namespace pfc {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// Storage tags of the 16-bit operand types.
struct Bf16Tag {};
struct F16Tag {};

__device__ __forceinline__ float bf16_to_float(uint16_t h) {
  return __uint_as_float(((uint32_t)h) << 16);
}

// Round-to-nearest-even float -> bfloat16 (finite inputs).
__device__ __forceinline__ uint16_t float_to_bf16(float f) {
  const uint32_t u = __float_as_uint(f);
  const uint32_t bias = 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)((u + bias) >> 16);
}

__device__ __forceinline__ float f16_to_float(uint16_t h) {
  _Float16 v;
  __builtin_memcpy(&v, &h, 2);
  return (float)v;
}

__device__ __forceinline__ uint16_t float_to_f16(float f) {
  const _Float16 v = (_Float16)f;  // hardware conversion, round to nearest even
  uint16_t h;
  __builtin_memcpy(&h, &v, 2);
  return h;
}

template <typename Tag>
__device__ __forceinline__ float to_float(uint16_t h);
template <>
__device__ __forceinline__ float to_float<Bf16Tag>(uint16_t h) { return bf16_to_float(h); }
template <>
__device__ __forceinline__ float to_float<F16Tag>(uint16_t h) { return f16_to_float(h); }

template <typename Tag>
__device__ __forceinline__ uint16_t from_float(float f);
template <>
__device__ __forceinline__ uint16_t from_float<Bf16Tag>(float f) { return float_to_bf16(f); }
template <>
__device__ __forceinline__ uint16_t from_float<F16Tag>(float f) { return float_to_f16(f); }

// Two floats to a packed pair of fp16 values, round to nearest even.
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_f16x2(float a, float b) {
  const f16x2_t v = {(_Float16)a, (_Float16)b};
  return __builtin_bit_cast(uint32_t, v);
}
__device__ __forceinline__ float f16_lo(uint32_t v) {
  return (float)__builtin_bit_cast(f16x2_t, v).x;
}
__device__ __forceinline__ float f16_hi(uint32_t v) {
  return (float)__builtin_bit_cast(f16x2_t, v).y;
}

// D(32x32, fp32) += A(32x16) * B(16x32).  Lane l supplies A[l%32][8(l/32)..+7]
// and B[8(l/32)..+7][l%32]; accumulator register r of lane l is
// D[8(r/4) + 4(l/32) + r%4][l%32].
__device__ __forceinline__ f32x16_t mfma_32x32x16(const uint4& a, const uint4& b, f32x16_t c,
                                                  Bf16Tag) {
  bf16x8_t av, bv;
  __builtin_memcpy(&av, &a, 16);
  __builtin_memcpy(&bv, &b, 16);
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bv, c, 0, 0, 0);
}
__device__ __forceinline__ f32x16_t mfma_32x32x16(const uint4& a, const uint4& b, f32x16_t c,
                                                  F16Tag) {
  f16x8_t av, bv;
  __builtin_memcpy(&av, &a, 16);
  __builtin_memcpy(&bv, &b, 16);
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(av, bv, c, 0, 0, 0);
}

// Target logit and its slope d f / d cos (divided by s).  CosFace:
// s (c - m), slope 1.  ArcFace: s cos(acos(c) + m) = s (c cos m - sin(theta) sin m),
// slope sin(theta + m) / sin(theta) = cos m + c sin m / sin(theta), with
// sin(theta) = sqrt(max(1 - c^2, 1e-12)).
struct Margin {
  float s, m, cos_m, sin_m;
  int kind;  // pfc_margin
};

__device__ __forceinline__ float target_logit(const Margin& mg, float c) {
  if (mg.kind == 0) return mg.s * (c - mg.m);
  const float sin_t = sqrtf(fmaxf(1.0f - c * c, 0.0f));
  return mg.s * (c * mg.cos_m - sin_t * mg.sin_m);
}

__device__ __forceinline__ float target_slope(const Margin& mg, float c) {
  if (mg.kind == 0) return 1.0f;
  const float sin_t = sqrtf(fmaxf(1.0f - c * c, 1e-12f));
  return mg.cos_m + c * mg.sin_m / sin_t;
}

// Softmax-gradient coefficient of one logit, without the s/B factor:
// (p - [j == y]) * slope, p = exp(f - lse).  A logit the PFC* filter dropped
// (stored cosine -inf) has p = 0, also in a row whose denominator it leaves
// empty (lse = -inf).
__device__ __forceinline__ float grad_coef(const Margin& mg, float c, bool is_target, float lse) {
  if (is_target) {
    const float p = __expf(target_logit(mg, c) - lse);
    return (p - 1.0f) * target_slope(mg, c);
  }
  return c == -INFINITY ? 0.0f : __expf(mg.s * c - lse);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// Lane move within rows of 16 lanes (DPP; CTRL: quad_perm 0x00-0xFF, row_mirror
// 0x140, row_half_mirror 0x141).
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, true));
}

// Sum over the wave's 64 lanes, returned as a wave-uniform value: butterfly
// within each 16-lane row by lane moves (no LDS), then the four row sums in a
// fixed order.
__device__ __forceinline__ float wave_total(float v) {
  v += dpp_mov<0xB1>(v);    // quad_perm [1,0,3,2]: pairs
  v += dpp_mov<0x4E>(v);    // quad_perm [2,3,0,1]: quads
  v += dpp_mov<0x141>(v);   // row_half_mirror: the other quad of the 8-lane half
  v += dpp_mov<0x140>(v);   // row_mirror: the other half of the row
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  return (r0 + r1) + (r2 + r3);
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
  return v;
}

// Merge two (max, sum 2^(. - max)) pairs (base-2 log-sum-exp).
__device__ __forceinline__ float2 lse_merge2(float2 a, float2 b) {
  const float mx = fmaxf(a.x, b.x);
  if (mx == -INFINITY) return make_float2(-INFINITY, 0.0f);
  return make_float2(mx, a.y * exp2f(a.x - mx) + b.y * exp2f(b.x - mx));
}

// Merge two (max, sum exp(. - max)) pairs.
__device__ __forceinline__ float2 lse_merge(float2 a, float2 b) {
  const float mx = fmaxf(a.x, b.x);
  if (mx == -INFINITY) return make_float2(-INFINITY, 0.0f);
  return make_float2(mx, a.y * __expf(a.x - mx) + b.y * __expf(b.x - mx));
}

}  // namespace pfc
