// Stage 3: inverse row norms of the batch and of the gathered active class
// centres (normalised cosine logits, Partial FC Sec. 3.1; the sampled
// classifier W[S], Sec. 3.3.2).
//
// The normalised rows are never materialised: the contractions use the raw
// 16-bit rows (exact products in fp32) and apply 1/||x_n|| and 1/||w_j|| as
// row / column scales.  On the 16-bit paths the class-row norms come out of
// the forward contraction kernel, which streams every active row through
// LDS anyway; this file holds the batch side (norms, the transposed bf16
// copy used by the class-gradient contraction) and the fp32 path.
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

// inv_x[n]; a transposed bf16 copy of the normalised batch x_hat in blocks
// of 32 rows (block c = [d][32]: entry (i, r) = x_hat[32 c + r][i]), the
// K-major operand of the class-gradient contraction, which a workgroup
// transposes through LDS; and the raw rows in 32-wide column blocks (block k
// = [ld_xt][32]: entry (n, e) = X[n][32 k + e]), the forward's operand, whose
// k-th chunk of a run of rows is then contiguous.  Rows n in [B, ld_xt) are
// zero in both.  Also clears the running max of 1/||w_j||.
// Workgroups past the first ld_xt / 32 write the padded copy of the active
// row ids that the contraction kernels read a chunk or tile at a time, with
// no wait on |S|: act_pad[j] = active[min(j, |S| - 1)] (0 if S is empty).
constexpr int kPrepRows = 32;
constexpr int kPadPerBlock = 4 * 256;   // act_pad entries per workgroup
template <typename Tag>
__global__ void __launch_bounds__(256) k_prep_x16(const uint16_t* __restrict__ X, int B, int d,
                                                  int64_t ld_xt, float* __restrict__ inv_x,
                                                  uint16_t* __restrict__ xbT,
                                                  uint16_t* __restrict__ xblk,
                                                  float* __restrict__ inv_w_max,
                                                  const int32_t* __restrict__ active,
                                                  const int32_t* __restrict__ n_active_p,
                                                  int32_t* __restrict__ act_pad, int64_t n_pad) {
  __shared__ uint16_t tile[kPrepRows][512 + 8];
  const int64_t n_row_blocks = ld_xt / kPrepRows;
  if (blockIdx.x >= n_row_blocks) {
    // Four consecutive entries per thread (n_pad is a multiple of 4).
    const int64_t i = (blockIdx.x - n_row_blocks) * kPadPerBlock + 4 * threadIdx.x;
    if (i >= n_pad) return;
    const int64_t K = *n_active_p;
    int o[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] = K > 0 ? active[i + e < K ? i + e : K - 1] : 0;
    *reinterpret_cast<int4*>(act_pad + i) = make_int4(o[0], o[1], o[2], o[3]);
    return;
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n0 = blockIdx.x * kPrepRows;
  if (blockIdx.x == 0 && threadIdx.x == 0) *inv_w_max = 0.0f;
  // Each wave's eight rows: all loads first (one memory round trip, not eight).
  const bool c_ok = lane < d / 8;   // d <= 512: one 16-byte piece per lane
  uint4 rows[kPrepRows / 4];
#pragma unroll
  for (int k = 0; k < kPrepRows / 4; ++k) {
    const int n = n0 + wave + 4 * k;
    rows[k] = make_uint4(0, 0, 0, 0);
    if (n < B && c_ok) rows[k] = *reinterpret_cast<const uint4*>(X + (int64_t)n * d + 8 * lane);
  }
#pragma unroll
  for (int k = 0; k < kPrepRows / 4; ++k) {
    const int r = wave + 4 * k;
    const int n = n0 + r;
    const uint4 v = rows[k];
    const float ss = wave_sum(sumsq8<Tag>(v));
    const float ix = 1.0f / fmaxf(sqrtf(ss), kEpsNorm);
    if (lane == 0 && n < B) inv_x[n] = ix;
    if (c_ok) {
      *reinterpret_cast<uint4*>(xblk + ((int64_t)(lane >> 2) * ld_xt + n) * 32 + 8 * (lane & 3)) = v;
      const uint16_t* h = reinterpret_cast<const uint16_t*>(&v);
      uint16_t o[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = float_to_bf16(to_float<Tag>(h[e]) * ix);
      uint4 ov;
      __builtin_memcpy(&ov, o, 16);
      *reinterpret_cast<uint4*>(&tile[r][8 * lane]) = ov;
    }
  }
  __syncthreads();
  // Column i of the tile (32 rows) -> block blockIdx.x of xbT, row i: four
  // 16-byte pieces (the block is contiguous: [d][32]).
  uint16_t* blk = xbT + (int64_t)blockIdx.x * d * kPrepRows;
  for (int q = threadIdx.x; q < d * 4; q += 256) {
    const int i = q >> 2, r0 = (q & 3) * 8;
    uint16_t o[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = tile[r0 + e][i];
    uint4 ov;
    __builtin_memcpy(&ov, o, 16);
    *reinterpret_cast<uint4*>(blk + i * kPrepRows + r0) = ov;
  }
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
  } else {
    const unsigned grid = (unsigned)(w.ld_xt / kPrepRows + ceil_div(w.n_act_pad, kPadPerBlock));
    if (a.dtype == 1)
      hipLaunchKernelGGL(k_prep_x16<Bf16Tag>, dim3(grid), dim3(256), 0, stream,
                         (const uint16_t*)a.X, B, d, w.ld_xt, w.inv_x, (uint16_t*)w.xbT,
                         (uint16_t*)w.xblk, w.inv_w_max, a.active, a.n_active, w.act_pad,
                         w.n_act_pad);
    else
      hipLaunchKernelGGL(k_prep_x16<F16Tag>, dim3(grid), dim3(256), 0, stream,
                         (const uint16_t*)a.X, B, d, w.ld_xt, w.inv_x, (uint16_t*)w.xbT,
                         (uint16_t*)w.xblk, w.inv_w_max, a.active, a.n_active, w.act_pad,
                         w.n_act_pad);
  }
  timing_stop(1, stream);
  return hipGetLastError();
}

}  // namespace pfc
