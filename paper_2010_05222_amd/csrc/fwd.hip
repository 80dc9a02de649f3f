// Stages 4-5 (the parts outside the fused contraction kernel of fwdx.hip):
// the row-wise log-sum-exp and the batch loss (Partial FC Sec. 3.1,
// Eq. sampled_probability; the max / sum decomposition of Sec. 3.2.1), and
// the fp32 path of the cosine contraction for small problems.
//
// On the 16-bit paths the fused kernel leaves one (m, sum 2^(f - m)) pair per
// row and class slice; k_lse16 merges a row's pairs into lse_n and its loss
// term, and k_loss takes the deterministic batch mean.
#include "pfc_gemm.h"

namespace pfc {
namespace {

// Merge the per-slice (m, sum) pairs of a row: lse_n, and the row's loss
// term.  One workgroup per row: the row maximum M over the slices, then
// sum_s sum_s * 2^(m_s - M), each a fixed-order reduction.  A row with no
// live logit (every pair (-inf, 0)) gets lse = -inf.
__global__ void __launch_bounds__(256) k_lse16(const float2* __restrict__ stats, int n_split,
                                               const int32_t* __restrict__ yhat,
                                               const float* __restrict__ tgt, int B,
                                               float* __restrict__ row_lse,
                                               float* __restrict__ loss_part) {
  __shared__ float red[4];
  const int n = blockIdx.x;
  const int t = threadIdx.x, lane = t & 63;
  const int64_t nct = n_split;
  const float2* row = stats + (int64_t)n * n_split;
  float mx = -INFINITY;
  for (int64_t c = t; c < nct; c += 256) mx = fmaxf(mx, row[c].x);
  mx = wave_max(mx);
  if (lane == 0) red[t >> 6] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  __syncthreads();
  float sm = 0.0f;
  if (mx != -INFINITY)
    for (int64_t c = t; c < nct; c += 256) {
      const float2 v = row[c];
      sm += v.y * exp2f(v.x - mx);
    }
  sm = wave_sum(sm);
  if (lane == 0) red[t >> 6] = sm;
  __syncthreads();
  if (t == 0) {
    sm = (red[0] + red[1]) + (red[2] + red[3]);
    const float lse = (mx + log2f(sm)) * 0.6931471805599453f;
    row_lse[n] = lse;
    loss_part[n] = yhat[n] >= 0 ? lse - tgt[n] : 0.0f;
  }
}

// fp32 path (small problems): one thread per (row, class) dot product.
// With tau < 1, a negative whose cosine exceeds tau is stored as -inf (PFC*,
// Eq. noise_filtering): its logit and its coefficient in the backward are 0.
__global__ void __launch_bounds__(256) k_fwd32(const float* __restrict__ X,
                                               const float* __restrict__ W,
                                               const int32_t* __restrict__ active,
                                               const int32_t* __restrict__ n_active_p,
                                               const int32_t* __restrict__ yhat,
                                               const float* __restrict__ inv_x,
                                               const float* __restrict__ inv_w, int B, int d,
                                               int64_t cap, int64_t ld_cos, float tau,
                                               float* __restrict__ cos32) {
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int n = blockIdx.y;
  if (j >= cap || j >= *n_active_p || n >= B) return;
  const float* x = X + (int64_t)n * d;
  const float* w = W + (int64_t)active[j] * d;
  float acc = 0.0f;
  for (int i = 0; i < d; ++i) acc = fmaf(x[i], w[i], acc);
  const float c = acc * inv_x[n] * inv_w[j];
  cos32[(int64_t)n * ld_cos + j] = (tau < 1.0f && j != yhat[n] && c > tau) ? -INFINITY : c;
}

__global__ void __launch_bounds__(256) k_lse32(const float* __restrict__ cos32, int64_t ld_cos,
                                               const int32_t* __restrict__ n_active_p,
                                               const int32_t* __restrict__ yhat, int B, Margin mg,
                                               float* __restrict__ row_lse,
                                               float* __restrict__ loss_part) {
  const int lane = threadIdx.x & 63;
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (n >= B) return;
  const int K = *n_active_p;
  const int yh = yhat[n];
  float2 acc = make_float2(-INFINITY, 0.0f);
  float ft = 0.0f;
  for (int j = lane; j < K; j += 64) {
    const float c = cos32[(int64_t)n * ld_cos + j];
    const float f = j == yh ? target_logit(mg, c) : mg.s * c;
    if (j == yh) ft = f;
    acc = lse_merge(acc, make_float2(f, 1.0f));
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    float2 o;
    o.x = __shfl_xor(acc.x, off, 64);
    o.y = __shfl_xor(acc.y, off, 64);
    acc = lse_merge(acc, o);
    ft += __shfl_xor(ft, off, 64);
  }
  if (lane == 0) {
    const float lse = acc.x + __logf(acc.y);
    row_lse[n] = lse;
    loss_part[n] = yh >= 0 ? lse - ft : 0.0f;
  }
}

// Deterministic batch mean of the row loss terms (one workgroup).
__global__ void __launch_bounds__(1024) k_loss(const float* __restrict__ loss_part, int B,
                                               float* __restrict__ loss) {
  __shared__ double part[16];
  double acc = 0.0;
  for (int n = threadIdx.x; n < B; n += blockDim.x) acc += (double)loss_part[n];
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 64);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    double s = 0.0;
    for (int w = 0; w < (int)(blockDim.x >> 6); ++w) s += part[w];
    *loss = (float)(s / (double)B);
  }
}

}  // namespace

hipError_t launch_forward(const StepArgs& a, const StepWs& w, hipStream_t stream) {
  hipError_t e = launch_prep(a, w, stream);
  if (e != hipSuccess) return e;
  const int B = (int)a.B, d = (int)a.d;
  Margin mg{a.s, a.m, cosf(a.m), sinf(a.m), a.margin};
  if (a.dtype == 0) {
    dim3 grid((unsigned)ceil_div(a.cap, 256), (unsigned)B);
    timing_start(2, stream);
    hipLaunchKernelGGL(k_fwd32, grid, dim3(256), 0, stream, (const float*)a.X,
                       (const float*)a.W, a.active, a.n_active, a.labels_mapped, w.inv_x,
                       w.inv_w, B, d, a.cap, w.ld_cos, a.tau, (float*)w.lbuf);
    timing_stop(2, stream);
    timing_start(3, stream);
    hipLaunchKernelGGL(k_lse32, dim3((unsigned)ceil_div(B, 4)), dim3(256), 0, stream,
                       (const float*)w.lbuf, w.ld_cos, a.n_active, a.labels_mapped, B, mg,
                       a.row_lse_out, w.loss_part);
  } else {
    timing_start(2, stream);
    launch_fwdx16(a, w, mg, stream);
    timing_stop(2, stream);
    timing_start(3, stream);
    hipLaunchKernelGGL(k_lse16, dim3((unsigned)B), dim3(256), 0, stream, w.stats, w.n_split,
                       a.labels_mapped, w.tgt, B, a.row_lse_out, w.loss_part);
  }
  hipLaunchKernelGGL(k_loss, dim3(1), dim3(1024), 0, stream, w.loss_part, B, a.loss);
  timing_stop(3, stream);
  return hipGetLastError();
}

}  // namespace pfc
