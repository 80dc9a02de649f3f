// Stage 3: inverse row norms of the batch and of the gathered active class
// centres (normalised cosine logits, Partial FC Sec. 3.1; the sampled
// classifier W[S], Sec. 3.3.2).
//
// The normalised rows are never materialised: the contractions use the raw
// 16-bit rows (exact products in fp32) and apply 1/||x_n|| and 1/||w_j|| as
// row / column scales.  These kernels read each row once with 16-byte
// loads, one wavefront per row (a 512-wide 16-bit row is exactly 64 x 16 B).
#include "pfc_device.h"

namespace pfc {
namespace {

constexpr float kEpsNorm = 1e-12f;

template <typename Tag>
__device__ __forceinline__ float sumsq8(const uint4& v) {
  const uint16_t* h = reinterpret_cast<const uint16_t*>(&v);
  float acc = 0.0f;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float f = to_float<Tag>(h[e]);
    acc = fmaf(f, f, acc);
  }
  return acc;
}

// inv_x[n] and the transposed bf16 copy xT[i * ldb + n] (zero for n >= B),
// the K-contiguous operand of the class-gradient contraction.
template <typename Tag>
__global__ void __launch_bounds__(256) k_prep_x16(const uint16_t* __restrict__ X, int B, int d,
                                                  int ldb, float* __restrict__ inv_x,
                                                  uint16_t* __restrict__ xT) {
  const int lane = threadIdx.x & 63;
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (n >= ldb) return;
  if (n >= B) {
    for (int i = lane; i < d; i += 64) xT[(int64_t)i * ldb + n] = 0;
    return;
  }
  const uint16_t* row = X + (int64_t)n * d;
  float ss = 0.0f;
  for (int c = lane; c < d / 8; c += 64) {
    const uint4 v = *reinterpret_cast<const uint4*>(row + 8 * c);
    ss += sumsq8<Tag>(v);
    const uint16_t* h = reinterpret_cast<const uint16_t*>(&v);
#pragma unroll
    for (int e = 0; e < 8; ++e)
      xT[(int64_t)(8 * c + e) * ldb + n] = float_to_bf16(to_float<Tag>(h[e]));
  }
  ss = wave_sum(ss);
  if (lane == 0) inv_x[n] = 1.0f / fmaxf(sqrtf(ss), kEpsNorm);
}

template <typename Tag>
__global__ void __launch_bounds__(256) k_norm_w16(const uint16_t* __restrict__ W, int d,
                                                  const int32_t* __restrict__ active,
                                                  const int32_t* __restrict__ n_active,
                                                  int64_t cap, float* __restrict__ inv_w) {
  const int lane = threadIdx.x & 63;
  const int64_t j = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (j >= cap || j >= *n_active) return;
  const uint16_t* row = W + (int64_t)active[j] * d;
  float ss = 0.0f;
  for (int c = lane; c < d / 8; c += 64)
    ss += sumsq8<Tag>(*reinterpret_cast<const uint4*>(row + 8 * c));
  ss = wave_sum(ss);
  if (lane == 0) inv_w[j] = 1.0f / fmaxf(sqrtf(ss), kEpsNorm);
}

__global__ void __launch_bounds__(256) k_prep_x32(const float* __restrict__ X, int B, int d,
                                                  float* __restrict__ inv_x) {
  const int lane = threadIdx.x & 63;
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (n >= B) return;
  const float* row = X + (int64_t)n * d;
  float ss = 0.0f;
  for (int i = lane; i < d; i += 64) ss = fmaf(row[i], row[i], ss);
  ss = wave_sum(ss);
  if (lane == 0) inv_x[n] = 1.0f / fmaxf(sqrtf(ss), kEpsNorm);
}

__global__ void __launch_bounds__(256) k_norm_w32(const float* __restrict__ W, int d,
                                                  const int32_t* __restrict__ active,
                                                  const int32_t* __restrict__ n_active,
                                                  int64_t cap, float* __restrict__ inv_w) {
  const int lane = threadIdx.x & 63;
  const int64_t j = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (j >= cap || j >= *n_active) return;
  const float* row = W + (int64_t)active[j] * d;
  float ss = 0.0f;
  for (int c = lane; c < d / 4; c += 64) {
    const float4 v = *reinterpret_cast<const float4*>(row + 4 * c);
    ss = fmaf(v.x, v.x, fmaf(v.y, v.y, fmaf(v.z, v.z, fmaf(v.w, v.w, ss))));
  }
  for (int i = (d / 4) * 4 + lane; i < d; i += 64) ss = fmaf(row[i], row[i], ss);
  ss = wave_sum(ss);
  if (lane == 0) inv_w[j] = 1.0f / fmaxf(sqrtf(ss), kEpsNorm);
}

}  // namespace

hipError_t launch_prep(const StepArgs& a, const StepWs& w, hipStream_t stream) {
  const int B = (int)a.B, d = (int)a.d;
  const unsigned wblocks = (unsigned)ceil_div(a.cap, 4);
  timing_start(1, stream);
  if (a.dtype == 0) {
    hipLaunchKernelGGL(k_prep_x32, dim3((unsigned)ceil_div(B, 4)), dim3(256), 0, stream,
                       (const float*)a.X, B, d, w.inv_x);
    hipLaunchKernelGGL(k_norm_w32, dim3(wblocks), dim3(256), 0, stream, (const float*)a.W, d,
                       a.active, a.n_active, a.cap, w.inv_w);
  } else if (a.dtype == 1) {
    hipLaunchKernelGGL(k_prep_x16<Bf16Tag>, dim3((unsigned)ceil_div(w.ldb, 4)), dim3(256), 0,
                       stream, (const uint16_t*)a.X, B, d, w.ldb, w.inv_x, (uint16_t*)w.xT);
    hipLaunchKernelGGL(k_norm_w16<Bf16Tag>, dim3(wblocks), dim3(256), 0, stream,
                       (const uint16_t*)a.W, d, a.active, a.n_active, a.cap, w.inv_w);
  } else {
    hipLaunchKernelGGL(k_prep_x16<F16Tag>, dim3((unsigned)ceil_div(w.ldb, 4)), dim3(256), 0,
                       stream, (const uint16_t*)a.X, B, d, w.ldb, w.inv_x, (uint16_t*)w.xT);
    hipLaunchKernelGGL(k_norm_w16<F16Tag>, dim3(wblocks), dim3(256), 0, stream,
                       (const uint16_t*)a.W, d, a.active, a.n_active, a.cap, w.inv_w);
  }
  timing_stop(1, stream);
  return hipGetLastError();
}

}  // namespace pfc
