// Stages 4-5: the cosine-logit contraction cos = x_hat . w_hat over the
// active classes (Partial FC Sec. 3.3.3, Eq. mp_gemm: [B x d][d x |S|]), the
// target margin and the row-wise log-sum-exp cross-entropy over S
// (Sec. 3.1, Eq. sampled_probability; max / sum decomposition of Sec. 3.2.1).
//
// 16-bit path: one MFMA GEMM kernel, tile 128 classes (MFMA M) x 128 batch
// rows (MFMA N) x 64 of d, double-buffered LDS.  Classes sit on the MFMA M
// axis so that each lane holds one batch row and 32 of its classes: the row
// max / sum-exp of the epilogue is mostly in-register.  The epilogue scales
// by 1/||x_n|| and 1/||w_j||, stores the unmargined cosine once as 16-bit
// fixed point (the logits' only write), applies the margin at the target,
// and emits one (max, sum exp) pair per (row, class tile).  A small kernel
// merges the pairs into lse_n and the loss.
#include "pfc_device.h"

namespace pfc {
namespace {

constexpr int kFwdBM = 128;                   // classes per tile
constexpr int kFwdBN = 128;                   // batch rows per tile
constexpr int kFwdBK = 64;                    // reduction slice of d per stage
constexpr int kFwdLds = kFwdBK + 8;           // padded LDS row (uint16 elements)

template <typename Tag>
__global__ void __launch_bounds__(256) k_fwd16(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ W,
    const int32_t* __restrict__ active, const int32_t* __restrict__ n_active_p,
    const int32_t* __restrict__ yhat, const float* __restrict__ inv_x,
    const float* __restrict__ inv_w, int B, int d, int64_t ld_cos, int64_t n_ctiles, int n_rt,
    int64_t n_tiles, int64_t per_xcd, Margin mg, int16_t* __restrict__ cosq,
    float2* __restrict__ stats, float* __restrict__ tgt) {
  // Tiles of one class tile (all batch-row tiles) run on the same XCD, so the
  // gathered W rows are fetched from HBM once and re-read from that XCD's L2.
  const int64_t t = (int64_t)(blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  if (t >= n_tiles) return;
  const int64_t ct = t / n_rt;
  const int rt = (int)(t % n_rt);
  const int K = *n_active_p;
  const int64_t j0 = ct * kFwdBM;
  if (j0 >= K) return;
  const int n0 = rt * kFwdBN;

  __shared__ __attribute__((aligned(16))) uint16_t As[2][kFwdBM * kFwdLds];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[2][kFwdBN * kFwdLds];
  __shared__ float2 red[2][kFwdBN];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int half = lane >> 5, l32 = lane & 31;

  const int lrow = tid >> 3;
  const int lcol = (tid & 7) * 8;
  const uint16_t* a_ptr[4];
  const uint16_t* b_ptr[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int64_t jr = j0 + lrow + 32 * q;
    a_ptr[q] = jr < K ? W + (int64_t)active[jr] * d + lcol : nullptr;
    const int nr = n0 + lrow + 32 * q;
    b_ptr[q] = nr < B ? X + (int64_t)nr * d + lcol : nullptr;
  }
  uint4 ra[4], rb[4];
  const uint4 zero = make_uint4(0, 0, 0, 0);
  auto gload = [&](int k0) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      ra[q] = a_ptr[q] ? *reinterpret_cast<const uint4*>(a_ptr[q] + k0) : zero;
      rb[q] = b_ptr[q] ? *reinterpret_cast<const uint4*>(b_ptr[q] + k0) : zero;
    }
  };
  auto swrite = [&](int s) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      *reinterpret_cast<uint4*>(&As[s][(lrow + 32 * q) * kFwdLds + lcol]) = ra[q];
      *reinterpret_cast<uint4*>(&Bs[s][(lrow + 32 * q) * kFwdLds + lcol]) = rb[q];
    }
  };

  f32x16_t acc[2][2];
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mb][nb][r] = 0.0f;

  const int nk = d / kFwdBK;
  gload(0);
  swrite(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int s = kt & 1;
    if (kt + 1 < nk) gload((kt + 1) * kFwdBK);
#pragma unroll
    for (int kk = 0; kk < kFwdBK / 16; ++kk) {
      uint4 af[2], bf[2];
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
        af[mb] = *reinterpret_cast<const uint4*>(
            &As[s][(wm * 64 + mb * 32 + l32) * kFwdLds + kk * 16 + 8 * half]);
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
        bf[nb] = *reinterpret_cast<const uint4*>(
            &Bs[s][(wn * 64 + nb * 32 + l32) * kFwdLds + kk * 16 + 8 * half]);
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) acc[mb][nb] = mfma_32x32x16(af[mb], bf[nb], acc[mb][nb], Tag{});
    }
    if (kt + 1 < nk) swrite(s ^ 1);
    __syncthreads();
  }

  // ---- epilogue
  float iw[2][16];
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int64_t j = j0 + wm * 64 + mb * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
      iw[mb][r] = j < K ? inv_w[j] : 0.0f;
    }
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const int nl = wn * 64 + nb * 32 + l32;
    const int n = n0 + nl;
    const bool nvalid = n < B;
    const float ix = nvalid ? inv_x[n] : 0.0f;
    const int yh = nvalid ? yhat[n] : -1;
    float fv[2][16];
    float mx = -INFINITY;
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        int16_t q4[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = 4 * g + e;
          const int64_t j = j0 + wm * 64 + mb * 32 + 8 * g + 4 * half + e;
          float f = -INFINITY;
          int16_t q = 0;
          if (j < K) {
            q = quantise_cos(acc[mb][nb][r] * ix * iw[mb][r]);
            const float c = dequantise_cos(q);
            if (j == yh) {
              f = target_logit(mg, c);
              if (nvalid) tgt[n] = f;
            } else {
              f = mg.s * c;
            }
          }
          q4[e] = q;
          fv[mb][r] = f;
          mx = fmaxf(mx, f);
        }
        if (nvalid) {
          uint2 packed;
          packed.x = (uint32_t)(uint16_t)q4[0] | ((uint32_t)(uint16_t)q4[1] << 16);
          packed.y = (uint32_t)(uint16_t)q4[2] | ((uint32_t)(uint16_t)q4[3] << 16);
          *reinterpret_cast<uint2*>(&cosq[(int64_t)n * ld_cos + j0 + wm * 64 + mb * 32 + 8 * g +
                                          4 * half]) = packed;
        }
      }
    }
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    float sm = 0.0f;
    if (mx != -INFINITY) {
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int r = 0; r < 16; ++r) sm += __expf(fv[mb][r] - mx);
    }
    sm += __shfl_xor(sm, 32, 64);
    if (half == 0) red[wm][nl] = make_float2(mx, sm);
  }
  __syncthreads();
  if (tid < kFwdBN) {
    const int n = n0 + tid;
    if (n < B) stats[(int64_t)n * n_ctiles + ct] = lse_merge(red[0][tid], red[1][tid]);
  }
}

// Merge the per-tile (max, sum) pairs of a row: lse_n, and the row's loss term.
__global__ void __launch_bounds__(256) k_lse16(const float2* __restrict__ stats, int64_t n_ctiles,
                                               const int32_t* __restrict__ n_active_p,
                                               const int32_t* __restrict__ yhat,
                                               const float* __restrict__ tgt, int B,
                                               float* __restrict__ row_lse,
                                               float* __restrict__ loss_part) {
  const int lane = threadIdx.x & 63;
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (n >= B) return;
  const int64_t nct = ceil_div((int64_t)*n_active_p, (int64_t)kFwdBM);
  float2 acc = make_float2(-INFINITY, 0.0f);
  for (int64_t c = lane; c < nct; c += 64) acc = lse_merge(acc, stats[(int64_t)n * n_ctiles + c]);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    float2 o;
    o.x = __shfl_xor(acc.x, off, 64);
    o.y = __shfl_xor(acc.y, off, 64);
    acc = lse_merge(acc, o);
  }
  if (lane == 0) {
    const float lse = acc.x + __logf(acc.y);
    row_lse[n] = lse;
    loss_part[n] = yhat[n] >= 0 ? lse - tgt[n] : 0.0f;
  }
}

// fp32 path (small problems): one thread per (row, class) dot product.
__global__ void __launch_bounds__(256) k_fwd32(const float* __restrict__ X,
                                               const float* __restrict__ W,
                                               const int32_t* __restrict__ active,
                                               const int32_t* __restrict__ n_active_p,
                                               const float* __restrict__ inv_x,
                                               const float* __restrict__ inv_w, int B, int d,
                                               int64_t cap, int64_t ld_cos,
                                               float* __restrict__ cos32) {
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int n = blockIdx.y;
  if (j >= cap || j >= *n_active_p || n >= B) return;
  const float* x = X + (int64_t)n * d;
  const float* w = W + (int64_t)active[j] * d;
  float acc = 0.0f;
  for (int i = 0; i < d; ++i) acc = fmaf(x[i], w[i], acc);
  cos32[(int64_t)n * ld_cos + j] = acc * inv_x[n] * inv_w[j];
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
                       (const float*)a.W, a.active, a.n_active, w.inv_x, w.inv_w, B, d, a.cap,
                       w.ld_cos, (float*)w.cosq);
    timing_stop(2, stream);
    timing_start(3, stream);
    hipLaunchKernelGGL(k_lse32, dim3((unsigned)ceil_div(B, 4)), dim3(256), 0, stream,
                       (const float*)w.cosq, w.ld_cos, a.n_active, a.labels_mapped, B, mg,
                       a.row_lse_out, w.loss_part);
  } else {
    const int n_rt = (int)ceil_div(B, kFwdBN);
    const int64_t n_tiles = w.n_ctiles * n_rt;
    const int64_t per_xcd = ceil_div(n_tiles, 8);
    const unsigned grid = (unsigned)(8 * per_xcd);
    timing_start(2, stream);
    if (a.dtype == 1)
      hipLaunchKernelGGL(k_fwd16<Bf16Tag>, dim3(grid), dim3(256), 0, stream,
                         (const uint16_t*)a.X, (const uint16_t*)a.W, a.active, a.n_active,
                         a.labels_mapped, w.inv_x, w.inv_w, B, d, w.ld_cos, w.n_ctiles, n_rt,
                         n_tiles, per_xcd, mg, (int16_t*)w.cosq, w.stats, w.tgt);
    else
      hipLaunchKernelGGL(k_fwd16<F16Tag>, dim3(grid), dim3(256), 0, stream,
                         (const uint16_t*)a.X, (const uint16_t*)a.W, a.active, a.n_active,
                         a.labels_mapped, w.inv_x, w.inv_w, B, d, w.ld_cos, w.n_ctiles, n_rt,
                         n_tiles, per_xcd, mg, (int16_t*)w.cosq, w.stats, w.tgt);
    timing_stop(2, stream);
    timing_start(3, stream);
    hipLaunchKernelGGL(k_lse16, dim3((unsigned)ceil_div(B, 4)), dim3(256), 0, stream, w.stats,
                       w.n_ctiles, a.n_active, a.labels_mapped, w.tgt, B, a.row_lse_out,
                       w.loss_part);
  }
  hipLaunchKernelGGL(k_loss, dim3(1), dim3(1024), 0, stream, w.loss_part, B, a.loss);
  timing_stop(3, stream);
  return hipGetLastError();
}

}  // namespace pfc
