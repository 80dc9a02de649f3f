// Stage 6: backward through the sampled margin softmax and both
// normalisations, and lazy momentum SGD on the active rows
// (Partial FC Eq. proxy_update, Eq. pfc_center_update, Sec. 3.2.1 matrix form:
// G = (P - Y)/B, dW = X^T G, dX = G W^T, restricted to the active set S).
//
// The softmax gradient is rebuilt on the fly from the forward's quantised
// cosines and lse_n; its coefficient without the s/B factor is
//   g'_{nj} = (p_{nj} - [j = y_n]) * slope_{nj}.
//
// dX (k_dx16): split-K MFMA GEMM, dX_hat^T[i][n] = sum_j W[S_j][i] *
//   (g'_{nj} / ||w_j||).  A workgroup owns 64 batch rows x all of d and a slice
//   of the classes; the gathered W rows are transposed into LDS so both MFMA
//   operands are contiguous along the class axis.  Split partials are summed
//   in a fixed order by k_dx_final, which also applies the normalisation
//   backward of x.
// dW + update (k_dw16): a workgroup owns 64 active classes x all of d and
//   reduces over the whole batch (dW_hat_j = sum_n g'_{nj} x_hat_n), so its
//   epilogue has complete rows: tangent projection, momentum, weight step
//   and the scatter back into the persistent W / momentum rows (unique rows,
//   no atomics).  Runs after k_dx16, which still reads the old W.
#include "pfc_device.h"

namespace pfc {
namespace {

constexpr int kDMax = 512;      // widest d of the 16-bit kernels
constexpr int kDxNT = 64;       // batch rows per dX tile
constexpr int kDxJK = 32;       // classes per reduction chunk
constexpr int kDxLds = kDxJK + 8;
constexpr int kDwJT = 64;       // classes per dW tile
constexpr int kDwNK = 32;       // batch rows per reduction chunk
constexpr int kDwLds = kDwNK + 8;

template <typename Tag>
__device__ __forceinline__ uint16_t to_bf16_bits(uint16_t h);
template <>
__device__ __forceinline__ uint16_t to_bf16_bits<Bf16Tag>(uint16_t h) { return h; }
template <>
__device__ __forceinline__ uint16_t to_bf16_bits<F16Tag>(uint16_t h) {
  return float_to_bf16(f16_to_float(h));
}

__device__ __forceinline__ uint16_t u16_at(const uint4& v, int e) {
  return reinterpret_cast<const uint16_t*>(&v)[e];
}

template <typename Tag>
__global__ void __launch_bounds__(256) k_dx16(
    const uint16_t* __restrict__ W, const int32_t* __restrict__ active,
    const int32_t* __restrict__ n_active_p, const int32_t* __restrict__ yhat,
    const float* __restrict__ row_lse, const float* __restrict__ inv_w,
    const int16_t* __restrict__ cosq, int64_t ld_cos, int B, int d, int n_rt, int n_split,
    int64_t n_tiles, int64_t per_xcd, Margin mg, float* __restrict__ dx_part) {
  // The batch-row tiles of one split share its class range: keep them on one XCD.
  const int64_t t = (int64_t)(blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  if (t >= n_tiles) return;
  const int split = (int)(t / n_rt);
  const int rt = (int)(t % n_rt);
  const int n0 = rt * kDxNT;
  const int K = *n_active_p;
  const int64_t n_chunks = ceil_div((int64_t)K, (int64_t)kDxJK);
  const int64_t per = ceil_div(n_chunks, (int64_t)n_split);
  const int64_t c_begin = split * per;
  const int64_t c_end = c_begin + per < n_chunks ? c_begin + per : n_chunks;

  __shared__ __attribute__((aligned(16))) uint16_t Wt[kDMax * kDxLds];   // [i][j]
  __shared__ __attribute__((aligned(16))) uint16_t A1[kDxNT * kDxLds];   // [n][j]

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, l32 = lane & 31;
  // W-load role: 8 columns of d, two groups of 4 consecutive classes.
  const int colchunk = tid & 63;
  const bool col_ok = colchunk * 8 < d;
  const int quad0 = tid >> 6;
  // Coefficient role: one batch row, 8 consecutive classes.
  const int rl = tid >> 2;
  const int jc = (tid & 3) * 8;
  const int rn = n0 + rl;
  const bool rvalid = rn < B;
  const float lse_n = rvalid ? row_lse[rn] : 0.0f;
  const int yh = rvalid ? yhat[rn] : -1;

  const uint4 zero = make_uint4(0, 0, 0, 0);
  uint4 wv[2][4];
  uint4 cq;
  float4 iw0, iw1;
  auto gload = [&](int64_t c) {
    const int64_t jb = c * kDxJK;
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int64_t jj = jb + 4 * (quad0 + 4 * u) + e;
        wv[u][e] = (jj < K && col_ok)
                       ? *reinterpret_cast<const uint4*>(W + (int64_t)active[jj] * d + 8 * colchunk)
                       : zero;
      }
    const bool cvalid = rvalid && jb + jc < K;
    cq = cvalid ? *reinterpret_cast<const uint4*>(cosq + (int64_t)rn * ld_cos + jb + jc) : zero;
    iw0 = *reinterpret_cast<const float4*>(inv_w + jb + jc);
    iw1 = *reinterpret_cast<const float4*>(inv_w + jb + jc + 4);
  };
  auto swrite = [&](int64_t c) {
    const int64_t jb = c * kDxJK;
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int e8 = 0; e8 < 8; ++e8) {
        uint2 p;
        p.x = (uint32_t)to_bf16_bits<Tag>(u16_at(wv[u][0], e8)) |
              ((uint32_t)to_bf16_bits<Tag>(u16_at(wv[u][1], e8)) << 16);
        p.y = (uint32_t)to_bf16_bits<Tag>(u16_at(wv[u][2], e8)) |
              ((uint32_t)to_bf16_bits<Tag>(u16_at(wv[u][3], e8)) << 16);
        *reinterpret_cast<uint2*>(&Wt[(8 * colchunk + e8) * kDxLds + 4 * (quad0 + 4 * u)]) = p;
      }
    const float iwv[8] = {iw0.x, iw0.y, iw0.z, iw0.w, iw1.x, iw1.y, iw1.z, iw1.w};
    uint16_t o[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int64_t j = jb + jc + k;
      float coef = 0.0f;
      if (rvalid && j < K) {
        const float cd = dequantise_cos((int16_t)u16_at(cq, k));
        coef = grad_coef(mg, cd, j == yh, lse_n) * iwv[k];
      }
      o[k] = float_to_bf16(coef);
    }
    uint4 ov;
    __builtin_memcpy(&ov, o, 16);
    *reinterpret_cast<uint4*>(&A1[rl * kDxLds + jc]) = ov;
  };

  f32x16_t acc[4][2];
#pragma unroll
  for (int mb = 0; mb < 4; ++mb)
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mb][nb][r] = 0.0f;
  const int i_base = wave * 128;

  if (c_begin < c_end) gload(c_begin);
  for (int64_t c = c_begin; c < c_end; ++c) {
    swrite(c);
    __syncthreads();
    if (c + 1 < c_end) gload(c + 1);
    if (i_base < d) {
#pragma unroll
      for (int kk = 0; kk < kDxJK / 16; ++kk) {
        uint4 af[4], bf[2];
#pragma unroll
        for (int mb = 0; mb < 4; ++mb)
          af[mb] = *reinterpret_cast<const uint4*>(
              &Wt[(i_base + mb * 32 + l32) * kDxLds + kk * 16 + 8 * half]);
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
          bf[nb] = *reinterpret_cast<const uint4*>(&A1[(nb * 32 + l32) * kDxLds + kk * 16 + 8 * half]);
#pragma unroll
        for (int mb = 0; mb < 4; ++mb)
#pragma unroll
          for (int nb = 0; nb < 2; ++nb)
            acc[mb][nb] = mfma_32x32x16(af[mb], bf[nb], acc[mb][nb], Bf16Tag{});
      }
    }
    __syncthreads();
  }

  if (i_base >= d) return;
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const int n = n0 + nb * 32 + l32;
    if (n >= B) continue;
    float* out = dx_part + ((int64_t)split * B + n) * d;
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int i = i_base + mb * 32 + 8 * g + 4 * half;
        if (i < d)
          *reinterpret_cast<float4*>(out + i) =
              make_float4(acc[mb][nb][4 * g], acc[mb][nb][4 * g + 1], acc[mb][nb][4 * g + 2],
                          acc[mb][nb][4 * g + 3]);
      }
  }
}

// Sum the split partials of a row in split order and apply the normalisation
// backward: dx = (dX_hat - x_hat (x_hat . dX_hat)) / ||x||, dX_hat = (s/B) * sum.
template <typename Tag>
__device__ __forceinline__ float load_x(const void* X, int64_t idx);
template <>
__device__ __forceinline__ float load_x<Bf16Tag>(const void* X, int64_t idx) {
  return bf16_to_float(((const uint16_t*)X)[idx]);
}
template <>
__device__ __forceinline__ float load_x<F16Tag>(const void* X, int64_t idx) {
  return f16_to_float(((const uint16_t*)X)[idx]);
}
struct F32Tag {};
template <>
__device__ __forceinline__ float load_x<F32Tag>(const void* X, int64_t idx) {
  return ((const float*)X)[idx];
}

template <typename Tag>
__global__ void __launch_bounds__(256) k_dx_final(const float* __restrict__ dx_part, int n_split,
                                                  const void* __restrict__ X,
                                                  const float* __restrict__ inv_x, int B, int d,
                                                  float sB, float* __restrict__ dX) {
  constexpr int kMaxPer = 16;  // d <= 1024
  const int lane = threadIdx.x & 63;
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (n >= B) return;
  const float ix = inv_x[n];
  float v[kMaxPer], xh[kMaxPer];
  float dot = 0.0f;
#pragma unroll
  for (int k = 0; k < kMaxPer; ++k) {
    const int i = lane + 64 * k;
    v[k] = 0.0f;
    xh[k] = 0.0f;
    if (i < d) {
      float sum = 0.0f;
      for (int s = 0; s < n_split; ++s) sum += dx_part[((int64_t)s * B + n) * d + i];
      v[k] = sB * sum;
      xh[k] = load_x<Tag>(X, (int64_t)n * d + i) * ix;
      dot = fmaf(xh[k], v[k], dot);
    }
  }
  dot = wave_sum(dot);
#pragma unroll
  for (int k = 0; k < kMaxPer; ++k) {
    const int i = lane + 64 * k;
    if (i < d) dX[(int64_t)n * d + i] = ix * (v[k] - xh[k] * dot);
  }
}

template <typename Tag>
__global__ void __launch_bounds__(256) k_dw16(
    const uint16_t* __restrict__ xT, int ldb, uint16_t* __restrict__ W,
    float* __restrict__ W_master, float* __restrict__ M, const int32_t* __restrict__ active,
    const int32_t* __restrict__ n_active_p, const int32_t* __restrict__ yhat,
    const float* __restrict__ row_lse, const float* __restrict__ inv_x,
    const float* __restrict__ inv_w, const int16_t* __restrict__ cosq, int64_t ld_cos, int B,
    int d, Margin mg, float sB, float lr, float mu) {
  const int K = *n_active_p;
  const int64_t j0 = (int64_t)blockIdx.x * kDwJT;
  if (j0 >= K) return;

  __shared__ __attribute__((aligned(16))) uint16_t Xs[kDMax * kDwLds];   // [i][n]
  __shared__ __attribute__((aligned(16))) uint16_t A2[kDwJT * kDwLds];   // [j][n]
  __shared__ float dred[4][kDwJT];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, l32 = lane & 31;
  // X-load role: 8 batch rows of 8 columns of d each.
  const int part = tid & 3;
  const int irow = tid >> 2;
  // Coefficient role: one batch row, 8 consecutive classes.
  const int rl = tid >> 3;
  const int jc = (tid & 7) * 8;

  const uint4 zero = make_uint4(0, 0, 0, 0);
  uint4 xv[8];
  uint4 cq;
  float lse_n = 0.0f, ix_n = 0.0f;
  int yh = -1;
  bool rvalid = false;
  auto gload = [&](int n0) {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int i = irow + 64 * u;
      xv[u] = i < d ? *reinterpret_cast<const uint4*>(xT + (int64_t)i * ldb + n0 + 8 * part) : zero;
    }
    const int rn = n0 + rl;
    rvalid = rn < B;
    cq = rvalid ? *reinterpret_cast<const uint4*>(cosq + (int64_t)rn * ld_cos + j0 + jc) : zero;
    lse_n = rvalid ? row_lse[rn] : 0.0f;
    ix_n = rvalid ? inv_x[rn] : 0.0f;
    yh = rvalid ? yhat[rn] : -1;
  };
  auto swrite = [&]() {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int i = irow + 64 * u;
      if (i < d) *reinterpret_cast<uint4*>(&Xs[i * kDwLds + 8 * part]) = xv[u];
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int64_t j = j0 + jc + k;
      float coef = 0.0f;
      if (rvalid && j < K) {
        const float cd = dequantise_cos((int16_t)u16_at(cq, k));
        coef = grad_coef(mg, cd, j == yh, lse_n) * ix_n;
      }
      A2[(jc + k) * kDwLds + rl] = float_to_bf16(coef);
    }
  };

  f32x16_t acc[4][2];
#pragma unroll
  for (int mb = 0; mb < 4; ++mb)
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mb][nb][r] = 0.0f;
  const int i_base = wave * 128;

  gload(0);
  for (int n0 = 0; n0 < ldb; n0 += kDwNK) {
    swrite();
    __syncthreads();
    if (n0 + kDwNK < ldb) gload(n0 + kDwNK);
    if (i_base < d) {
#pragma unroll
      for (int kk = 0; kk < kDwNK / 16; ++kk) {
        uint4 af[4], bf[2];
#pragma unroll
        for (int mb = 0; mb < 4; ++mb)
          af[mb] = *reinterpret_cast<const uint4*>(
              &Xs[(i_base + mb * 32 + l32) * kDwLds + kk * 16 + 8 * half]);
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
          bf[nb] = *reinterpret_cast<const uint4*>(&A2[(nb * 32 + l32) * kDwLds + kk * 16 + 8 * half]);
#pragma unroll
        for (int mb = 0; mb < 4; ++mb)
#pragma unroll
          for (int nb = 0; nb < 2; ++nb)
            acc[mb][nb] = mfma_32x32x16(af[mb], bf[nb], acc[mb][nb], Bf16Tag{});
      }
    }
    __syncthreads();
  }

  // ---- epilogue: lane owns class j (per nb) and 64 of its d entries.
  int64_t arow[2];
  float iwj[2];
  bool jvalid[2];
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const int64_t j = j0 + nb * 32 + l32;
    jvalid[nb] = j < K;
    arow[nb] = jvalid[nb] ? (int64_t)active[j] : 0;
    iwj[nb] = jvalid[nb] ? inv_w[j] : 0.0f;
    float dot = 0.0f;
    if (jvalid[nb] && i_base < d) {
      const uint16_t* wrow = W + arow[nb] * d;
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int i = i_base + mb * 32 + 8 * g + 4 * half;
          if (i >= d) continue;
          const uint2 w4 = *reinterpret_cast<const uint2*>(wrow + i);
          const uint16_t* wh = reinterpret_cast<const uint16_t*>(&w4);
#pragma unroll
          for (int e = 0; e < 4; ++e)
            dot = fmaf(to_float<Tag>(wh[e]) * iwj[nb], sB * acc[mb][nb][4 * g + e], dot);
        }
    }
    dot += __shfl_xor(dot, 32, 64);
    if (half == 0) dred[wave][nb * 32 + l32] = dot;
  }
  __syncthreads();
  if (i_base >= d) return;
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    if (!jvalid[nb]) continue;
    const int jl = nb * 32 + l32;
    const float dot = dred[0][jl] + dred[1][jl] + dred[2][jl] + dred[3][jl];
    uint16_t* wrow = W + arow[nb] * d;
    float* mrow = M + arow[nb] * d;
    float* prow = W_master ? W_master + arow[nb] * d : nullptr;
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int i = i_base + mb * 32 + 8 * g + 4 * half;
        if (i >= d) continue;
        const uint2 w4 = *reinterpret_cast<const uint2*>(wrow + i);
        const uint16_t* wh = reinterpret_cast<const uint16_t*>(&w4);
        float4 m4 = *reinterpret_cast<const float4*>(mrow + i);
        float* mv = reinterpret_cast<float*>(&m4);
        float wnew[4];
        float4 p4;
        float* pv = reinterpret_cast<float*>(&p4);
        if (prow) p4 = *reinterpret_cast<const float4*>(prow + i);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float w = to_float<Tag>(wh[e]);
          const float gr = iwj[nb] * (sB * acc[mb][nb][4 * g + e] - w * iwj[nb] * dot);
          mv[e] = mu * mv[e] + gr;
          if (prow) {
            pv[e] = pv[e] - lr * mv[e];
            wnew[e] = pv[e];
          } else {
            wnew[e] = w - lr * mv[e];
          }
        }
        *reinterpret_cast<float4*>(mrow + i) = m4;
        if (prow) *reinterpret_cast<float4*>(prow + i) = p4;
        uint2 o;
        o.x = (uint32_t)from_float<Tag>(wnew[0]) | ((uint32_t)from_float<Tag>(wnew[1]) << 16);
        o.y = (uint32_t)from_float<Tag>(wnew[2]) | ((uint32_t)from_float<Tag>(wnew[3]) << 16);
        *reinterpret_cast<uint2*>(wrow + i) = o;
      }
  }
}

// ---------------------------------------------------------------- fp32 path
// Small problems only (parity scale): plain loops, one output per thread.

__global__ void __launch_bounds__(256) k_dx32(const float* __restrict__ W,
                                              const int32_t* __restrict__ active,
                                              const int32_t* __restrict__ n_active_p,
                                              const int32_t* __restrict__ yhat,
                                              const float* __restrict__ row_lse,
                                              const float* __restrict__ inv_w,
                                              const float* __restrict__ cos32, int64_t ld_cos,
                                              int B, int d, Margin mg, float* __restrict__ out) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  const int n = blockIdx.y;
  if (i >= d || n >= B) return;
  const int K = *n_active_p;
  const int yh = yhat[n];
  const float lse = row_lse[n];
  float acc = 0.0f;
  for (int j = 0; j < K; ++j) {
    const float coef = grad_coef(mg, cos32[(int64_t)n * ld_cos + j], j == yh, lse) * inv_w[j];
    acc = fmaf(coef, W[(int64_t)active[j] * d + i], acc);
  }
  out[(int64_t)n * d + i] = acc;
}

__global__ void __launch_bounds__(256) k_dw32(const float* __restrict__ X, float* __restrict__ W,
                                              float* __restrict__ W_master, float* __restrict__ M,
                                              const int32_t* __restrict__ active,
                                              const int32_t* __restrict__ n_active_p,
                                              const int32_t* __restrict__ yhat,
                                              const float* __restrict__ row_lse,
                                              const float* __restrict__ inv_x,
                                              const float* __restrict__ inv_w,
                                              const float* __restrict__ cos32, int64_t ld_cos,
                                              int B, int d, Margin mg, float sB, float lr,
                                              float mu) {
  constexpr int kMaxB = 4096;
  constexpr int kMaxPer = 4;  // d <= 1024
  __shared__ float coef[kMaxB];
  __shared__ float red[4];
  const int64_t j = blockIdx.x;
  if (j >= *n_active_p) return;
  const float iw = inv_w[j];
  for (int n = threadIdx.x; n < B; n += blockDim.x)
    coef[n] = grad_coef(mg, cos32[(int64_t)n * ld_cos + j], j == yhat[n], row_lse[n]) * inv_x[n];
  __syncthreads();
  const int64_t a = active[j];
  float dw[kMaxPer];
  float dot = 0.0f;
#pragma unroll
  for (int k = 0; k < kMaxPer; ++k) {
    const int i = threadIdx.x + 256 * k;
    dw[k] = 0.0f;
    if (i < d) {
      float acc = 0.0f;
      for (int n = 0; n < B; ++n) acc = fmaf(coef[n], X[(int64_t)n * d + i], acc);
      dw[k] = sB * acc;
      dot = fmaf(W[a * d + i] * iw, dw[k], dot);
    }
  }
  dot = wave_sum(dot);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = dot;
  __syncthreads();
  dot = red[0] + red[1] + red[2] + red[3];
#pragma unroll
  for (int k = 0; k < kMaxPer; ++k) {
    const int i = threadIdx.x + 256 * k;
    if (i >= d) continue;
    const float w = W[a * d + i];
    const float gr = iw * (dw[k] - w * iw * dot);
    const float m = mu * M[a * d + i] + gr;
    M[a * d + i] = m;
    if (W_master) {
      const float p = W_master[a * d + i] - lr * m;
      W_master[a * d + i] = p;
      W[a * d + i] = p;
    } else {
      W[a * d + i] = w - lr * m;
    }
  }
}

}  // namespace

hipError_t launch_backward(const StepArgs& a, const StepWs& w, hipStream_t stream) {
  const int B = (int)a.B, d = (int)a.d;
  Margin mg{a.s, a.m, cosf(a.m), sinf(a.m), a.margin};
  const float sB = a.s / (float)a.B;
  if (a.dtype == 0) {
    timing_start(4, stream);
    hipLaunchKernelGGL(k_dx32, dim3((unsigned)ceil_div(d, 256), (unsigned)B), dim3(256), 0,
                       stream, (const float*)a.W, a.active, a.n_active, a.labels_mapped,
                       a.row_lse, w.inv_w, (const float*)w.cosq, w.ld_cos, B, d, mg, w.dx_part);
    timing_stop(4, stream);
    timing_start(5, stream);
    hipLaunchKernelGGL(k_dx_final<F32Tag>, dim3((unsigned)ceil_div(B, 4)), dim3(256), 0, stream,
                       w.dx_part, 1, a.X, w.inv_x, B, d, sB, a.dX);
    timing_stop(5, stream);
    timing_start(6, stream);
    hipLaunchKernelGGL(k_dw32, dim3((unsigned)a.cap), dim3(256), 0, stream, (const float*)a.X,
                       (float*)a.W, a.W_master, a.M, a.active, a.n_active, a.labels_mapped,
                       a.row_lse, w.inv_x, w.inv_w, (const float*)w.cosq, w.ld_cos, B, d, mg, sB,
                       a.lr, a.mu);
    timing_stop(6, stream);
    return hipGetLastError();
  }
  const int n_rt = (int)ceil_div(B, kDxNT);
  const int64_t n_tiles = (int64_t)n_rt * w.n_split;
  const int64_t per_xcd = ceil_div(n_tiles, 8);
  const unsigned dx_grid = (unsigned)(8 * per_xcd);
  const unsigned dw_grid = (unsigned)ceil_div(a.cap, kDwJT);
  if (a.dtype == 1) {
    timing_start(4, stream);
    hipLaunchKernelGGL(k_dx16<Bf16Tag>, dim3(dx_grid), dim3(256), 0, stream,
                       (const uint16_t*)a.W, a.active, a.n_active, a.labels_mapped, a.row_lse,
                       w.inv_w, (const int16_t*)w.cosq, w.ld_cos, B, d, n_rt, w.n_split, n_tiles,
                       per_xcd, mg, w.dx_part);
    timing_stop(4, stream);
    timing_start(5, stream);
    hipLaunchKernelGGL(k_dx_final<Bf16Tag>, dim3((unsigned)ceil_div(B, 4)), dim3(256), 0, stream,
                       w.dx_part, w.n_split, a.X, w.inv_x, B, d, sB, a.dX);
    timing_stop(5, stream);
    timing_start(6, stream);
    hipLaunchKernelGGL(k_dw16<Bf16Tag>, dim3(dw_grid), dim3(256), 0, stream,
                       (const uint16_t*)w.xT, (int)w.ldb, (uint16_t*)a.W, a.W_master, a.M,
                       a.active, a.n_active, a.labels_mapped, a.row_lse, w.inv_x, w.inv_w,
                       (const int16_t*)w.cosq, w.ld_cos, B, d, mg, sB, a.lr, a.mu);
  } else {
    timing_start(4, stream);
    hipLaunchKernelGGL(k_dx16<F16Tag>, dim3(dx_grid), dim3(256), 0, stream,
                       (const uint16_t*)a.W, a.active, a.n_active, a.labels_mapped, a.row_lse,
                       w.inv_w, (const int16_t*)w.cosq, w.ld_cos, B, d, n_rt, w.n_split, n_tiles,
                       per_xcd, mg, w.dx_part);
    timing_stop(4, stream);
    timing_start(5, stream);
    hipLaunchKernelGGL(k_dx_final<F16Tag>, dim3((unsigned)ceil_div(B, 4)), dim3(256), 0, stream,
                       w.dx_part, w.n_split, a.X, w.inv_x, B, d, sB, a.dX);
    timing_stop(5, stream);
    timing_start(6, stream);
    hipLaunchKernelGGL(k_dw16<F16Tag>, dim3(dw_grid), dim3(256), 0, stream,
                       (const uint16_t*)w.xT, (int)w.ldb, (uint16_t*)a.W, a.W_master, a.M,
                       a.active, a.n_active, a.labels_mapped, a.row_lse, w.inv_x, w.inv_w,
                       (const int16_t*)w.cosq, w.ld_cos, B, d, mg, sB, a.lr, a.mu);
  }
  timing_stop(6, stream);
  return hipGetLastError();
}

}  // namespace pfc
