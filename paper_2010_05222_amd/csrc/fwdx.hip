// Stages 3-5 and the feature-gradient contraction of stage 6, fused, on the
// 16-bit paths: the cosine logits against the active classes (Partial FC
// Sec. 3.3.3, Eq. mp_gemm: [B x d][d x |S|]), the target margin, the row-wise
// log-sum-exp statistics (Sec. 3.1, Eq. sampled_probability; the max / sum
// decomposition of Sec. 3.2.1) and dX_hat = P W_hat (Eq. proxy_update, the
// matrix form of Sec. 3.2.1), in one pass over the gathered class rows.
//
// A workgroup owns 64 batch rows and a slice of the active classes, walked in
// chunks of 32 classes.  The batch rows stay in registers for the whole
// slice; each chunk's gathered W rows go straight from HBM into a four-stage
// LDS ring (direct-to-LDS loads, three chunks in flight) and are used twice:
// as the class operand of the cosine contraction (16x16x32 MFMA, each wave 16
// batch rows over all of d) and, read transposed, as the W operand of the
// dX contraction (32x32x16 MFMA, each wave a quarter of d for all 64 rows).
//
// The softmax probabilities of the dX contraction need each row's full
// log-sum-exp, which is only known after every class.  The kernel keeps per
// row a running reference m (base 2) instead, accumulates
// O = sum_j 2^(f_j - m) W_j / ||w_j|| and sum_j 2^(f_j - m), and rescales both
// when m moves; m moves only when a chunk's maximum exceeds it by more than
// kRefSlack, so values stay <= 2^kRefSlack and rescales are rare.  The final
// kernels merge the per-slice (m, sum) pairs into lse and scale each slice's
// O by 2^(m - lse) (exactly the decomposition of Sec. 3.2.1).
//
// The same pass writes the logit store the class-gradient kernel reads:
// E = 2^(f - m) in fp16 per (row, class), relative to the row's reference for
// each group of 128 classes (E = 0 at the row's target and past |S|), and the
// group references.  A group's four chunks are held in registers until the
// group ends, and rescaled there if m moved inside the group.
#include "pfc_gemm.h"

namespace pfc {
namespace {

constexpr int kFxRows = 64;      // batch rows of a workgroup
constexpr int kFxCls = 32;       // active classes per chunk
constexpr int kFxStages = 4;     // W ring depth
constexpr int kFxThreads = 256;  // four waves
constexpr int kFxPLd = 40;       // coefficient tile row stride, 16-bit elements (80 B)
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kEpsNormW = 1e-12f;
constexpr float kRefSlack = 8.0f;
// Largest fp16 coefficient of the dX contraction: P' = 2^(f - m) / ||w|| * sigma
// <= 2^kRefSlack * 2^7 = 2^15, below the fp16 maximum.
constexpr float kFp16CoefHeadroom = 128.0f;

// W ring, sized for d = 512: stage s, row r at fxW + (s * 32 + r) * (d + 16).
// Row r of a stage holds chunk class sigma(r) (below), and its 16-byte piece
// p is stored at position p ^ ((r >> 3) & 1).  With the 32-byte row padding,
// the sixteen rows of one cosine-operand read and the four rows of one
// transposing read each hit distinct banks.
__shared__ __attribute__((aligned(1024))) uint16_t fxW[kFxStages * kFxCls * (512 + 16)];
// Coefficients P' of the chunk for the dX contraction, [64 rows][32 classes].
__shared__ __attribute__((aligned(16))) uint16_t fxP[kFxRows * kFxPLd];
// Per-row rescale factor of the dX accumulators for the chunk.
__shared__ __attribute__((aligned(16))) float fxFac[kFxRows];
// Partial squared norms of the chunk's class rows (one quarter of d per wave),
// and each wave's own copy of the inverse norms.
__shared__ __attribute__((aligned(16))) float fxNrm[4][kFxCls];
__shared__ __attribute__((aligned(16))) float fxIw[4][kFxCls];
// Active-row ids of the chunks in flight: wave w's eight rows, four slots.
__shared__ __attribute__((aligned(16))) int32_t fxIds[4][4][8];

// Stage row r holds class sigma(r) of its chunk.  With this order the 16x16
// cosine tile of a lane (M index 4 (l / 16) + i of blocks 0 and 1) covers the
// eight consecutive classes 8 (l / 16) .. + 7.
__host__ __device__ constexpr int fx_sigma(int r) {
  return 8 * ((r & 15) >> 2) + 4 * (r >> 4) + (r & 3);
}
__host__ __device__ constexpr int fx_sigma_inv(int k) {
  return 16 * ((k >> 2) & 1) + 4 * (k >> 3) + (k & 3);
}
static_assert(fx_sigma(fx_sigma_inv(13)) == 13 && fx_sigma_inv(fx_sigma(21)) == 21, "sigma");

template <int OFF>
__device__ __forceinline__ void ds_write_32(uint32_t addr, uint32_t v) {
  asm volatile("ds_write_b32 %0, %1 offset:%2" ::"v"(addr), "v"(v), "i"(OFF) : "memory");
}

typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));

// D(16x16, fp32) += A(16x32) * B(32x16): lane l supplies A[l % 16][8 (l / 16) .. + 7]
// and B[8 (l / 16) .. + 7][l % 16]; accumulator register i of lane l is
// D[4 (l / 16) + i][l % 16].
__device__ __forceinline__ f32x4_t mfma_16x16x32(const u32x4_t& a, const u32x4_t& b, f32x4_t c,
                                                 Bf16Tag) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}
__device__ __forceinline__ f32x4_t mfma_16x16x32(const u32x4_t& a, const u32x4_t& b, f32x4_t c,
                                                 F16Tag) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8_t, a),
                                                __builtin_bit_cast(f16x8_t, b), c, 0, 0, 0);
}

// a0^2 + a1^2 + acc for a packed pair of 16-bit values.
__device__ __forceinline__ float sumsq2(uint32_t v, float acc, F16Tag) {
  const f16x2_t h = __builtin_bit_cast(f16x2_t, v);
  return __builtin_amdgcn_fdot2(h, h, acc, false);
}
__device__ __forceinline__ float sumsq2(uint32_t v, float acc, Bf16Tag) {
  const bf16x2_t h = __builtin_bit_cast(bf16x2_t, v);
  return __builtin_amdgcn_fdot2_f32_bf16(h, h, acc, false);
}

template <typename Tag>
__device__ __forceinline__ uint32_t pack2(float a, float b);
template <>
__device__ __forceinline__ uint32_t pack2<Bf16Tag>(float a, float b) {
  const bf16x2_t v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}
template <>
__device__ __forceinline__ uint32_t pack2<F16Tag>(float a, float b) {
  const f16x2_t v = {(_Float16)a, (_Float16)b};
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ uint4 as_uint4(const u32x4_t& v) { return make_uint4(v.x, v.y, v.z, v.w); }

// Eight fp16 values of a packed 16-byte group, times f, repacked.
__device__ __forceinline__ u32x4_t scale_f16x8(const u32x4_t& v, float f) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
  uint32_t o[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) o[k] = pack_f16x2(f16_lo(w[k]) * f, f16_hi(w[k]) * f);
  return u32x4_t{o[0], o[1], o[2], o[3]};
}

// One workgroup: batch rows [n0, n0 + 64) x the class slice of `split`, all of
// d (= 32 KS).  Outputs: the logit store and group references of its rows
// and classes, 1/||w|| of its classes (first row tile only), the row's
// margined target logit and cosine where the target lies in the slice, and,
// per (row, split), the pair (m, sum 2^(f - m)) and the dX partial
// O / sigma (O relative to the same m).
template <typename Tag, int D, bool FILT>
__global__ void __launch_bounds__(kFxThreads, 1) k_fwdx16(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ W,
    const int32_t* __restrict__ act_pad, const int32_t* __restrict__ n_active_p,
    const int32_t* __restrict__ yhat, const float* __restrict__ inv_x, int B, int n_rt,
    int n_split, int64_t n_tiles, int64_t per_xcd, Margin mg, float tau, int64_t ld_cos,
    int64_t ld_g, uint16_t* __restrict__ lbuf, float* __restrict__ gmax,
    float* __restrict__ inv_w, float2* __restrict__ stats, float* __restrict__ tgt,
    float* __restrict__ tgtc, float* __restrict__ dx_part) {
  constexpr int KS = D / 32;          // 16x16x32 k-steps of the cosine contraction
  constexpr int KSW = KS / 4;         // k-steps whose squares each wave sums for the norms
  constexpr int MB = D / 128;         // 32-wide d blocks of a wave's quarter of dX
  constexpr int RLD = D + 16;         // W stage row stride, elements
  constexpr uint32_t RB = RLD * 2;    // ... bytes
  constexpr uint32_t SB = kFxCls * RB;
  constexpr bool kF16 = std::is_same<Tag, F16Tag>::value;

  // All row tiles of a split run on one XCD, so the split's W rows are
  // fetched from HBM once and re-read from that XCD's L2.
  const int64_t t = (int64_t)(blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  if (t >= n_tiles) return;
  const int split = (int)(t / n_rt);
  const int rt = (int)(t % n_rt);
  const int n0 = rt * kFxRows;
  const int K = *n_active_p;
  const int64_t n_ch = ceil_div((int64_t)K, (int64_t)kFxCls);
  const int64_t n_grp = ceil_div(n_ch, (int64_t)4);
  const int64_t per = ceil_div(n_grp, (int64_t)n_split);
  const int64_t g_begin = (int64_t)split * per < n_grp ? (int64_t)split * per : n_grp;
  const int64_t g_end = g_begin + per < n_grp ? g_begin + per : n_grp;
  const int64_t c_begin = 4 * g_begin;
  const int64_t c_end = 4 * g_end < n_ch ? 4 * g_end : n_ch;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r16 = lane & 15, q = lane >> 4;   // cosine layout: row 16 wave + r16, classes 8q..8q+7
  const int l32 = lane & 31, h = lane >> 5;   // dX layout: row 32 nb + l32
  const int rho = 16 * wave + r16;
  const int n_row = n0 + rho;
  const int dbase = wave * (D / 4);           // the wave's quarter of d in the dX contraction

  // The wave's 16 batch rows as the cosine contraction's B operand, for the
  // whole slice: lane l holds X[row][32 ks + 8 q .. + 7].
  u32x4_t xr[KS];
  {
    const int nr = n_row < B ? n_row : B - 1;
    const u32x4_t* xp = reinterpret_cast<const u32x4_t*>(X + (int64_t)nr * D + 8 * q);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) xr[ks] = xp[4 * ks];
  }
  float ix = n_row < B ? inv_x[n_row] : 0.0f;
  int yh = n_row < B ? yhat[n_row] : -1;
  wait_vmcnt<0>();
  pin_reg(xr);
  pin_reg(ix);
  pin_reg(yh);

  f32x16_t acc[MB][2];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mb][nb][r] = 0.0f;
  float mref = -INFINITY;   // the row's running reference (base 2)
  float lpart = 0.0f;       // sum of 2^(f - mref) over the lane's classes so far
  float sig = kF16 ? INFINITY : 1.0f;   // fp16 coefficient scale (power of two)

  if (c_begin < c_end) {
    const uint32_t wring = lds_addr(fxW);
    // Ids of chunk c: two runs of four classes per wave (sigma(8 wave) .. + 3
    // and + 8 .. + 11), from the padded copy, into ring slot c & 3.
    auto dma_ids = [&](int64_t c) __attribute__((always_inline)) {
      const int64_t cc = c < c_end ? c : c_end - 1;
      if (lane < 2)
        dma16(act_pad + cc * kFxCls + fx_sigma(8 * wave) + 8 * lane, &fxIds[wave][c & 3][0]);
    };
    // W rows of chunk c into stage s: row 8 wave + v, one load per row, from
    // the ids in slot c & 3 (landed).
    auto dma_w = [&](int64_t c, int s) __attribute__((always_inline)) {
      u32x4_t i0, i1;
      ds_read_128<0>(i0, lds_addr(&fxIds[wave][c & 3][0]));
      ds_read_128<16>(i1, lds_addr(&fxIds[wave][c & 3][0]));
      lgkm_wait<0>(i0, i1);
      const int rows[8] = {(int)i0.x, (int)i0.y, (int)i0.z, (int)i0.w,
                           (int)i1.x, (int)i1.y, (int)i1.z, (int)i1.w};
      uint16_t* st = fxW + (s * kFxCls + 8 * wave) * RLD;
#pragma unroll
      for (int v = 0; v < 8; ++v) {
        const int row = __builtin_amdgcn_readfirstlane(rows[v]);
        if (lane < D / 8) dma16(W + (int64_t)row * D + 8 * (lane ^ (wave & 1)), st + v * RLD);
      }
    };
    // Ids of the first three chunks, then three virtual iterations of the
    // steady pattern (ids of chunk c + 5 and W rows of chunk c + 3), so that
    // every iteration finds the same load counts in flight.
    dma_ids(c_begin);
    dma_ids(c_begin + 1);
    dma_ids(c_begin + 2);
    wait_vmcnt<0>();
    dma_ids(c_begin + 2);
    dma_w(c_begin, 0);
    dma_ids(c_begin + 3);
    dma_w(c_begin + 1, 1);
    dma_ids(c_begin + 4);
    dma_w(c_begin + 2, 2);

    // Per-lane LDS byte offsets.  Cosine operand: stage row 16 mb + r16, piece
    // 4 ks + q (stored at (4 ks + q) ^ f, f = (r16 >> 3) & 1).
    const uint32_t a_cos = r16 * RB + 16 * (q ^ ((r16 >> 3) & 1));
    // Transposing W reads of the dX contraction (see frag_mn_major): the
    // addressing lane 4 e + p of 16-lane group fg points at class
    // kappa = 16 kk + 8 (fg >> 1) + e (stage row sigma_inv(kappa)) and, for
    // the hi half, kappa + 4 (that row + 16), columns dbase + 16 (fg & 1) + 4 p.
    const int fg = lane >> 4, fsrc = lane & 15;
    const int chunk0 = dbase / 8 + 2 * (fg & 1) + ((fsrc & 3) >> 1);
    uint32_t a_tr[2];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int r_lo = 8 * kk + 4 * (fg >> 1) + (fsrc >> 2);
      a_tr[kk] = r_lo * RB + 16 * (chunk0 ^ kk) + 8 * (fsrc & 1);
    }
    // Coefficient tile reads (B operand of dX): row 32 nb + l32, classes 16 kk + 8 h.
    const uint32_t b_p = lds_addr(fxP) + l32 * (kFxPLd * 2) + 16 * h;
    const uint32_t p_w = lds_addr(fxP) + rho * (kFxPLd * 2) + 16 * q;

    const float s2 = mg.s * kLog2e;
    u32x4_t eb[4];      // fp16 E of the group's chunks
    float gm[4];        // the reference each was computed with
    for (int64_t g = g_begin; g < g_end; ++g) {
      static_for<0, 4>([&](auto sl) {
        constexpr int S = decltype(sl)::value;
        const int64_t c = 4 * g + S;
        if (c >= c_end) return;
        const uint32_t stg = wring + S * SB;
        // Landed: this wave's W rows of chunk c and the ids of chunk c + 3;
        // after the barrier everyone's rows, and every wave is done with
        // chunk c - 1 (its stage and the coefficient tile are free).
        wait_vmcnt<17>();
        stage_barrier();
        dma_ids(c + 5);
        dma_w(c + 3, (S + 3) % 4);

        // ---- cosine contraction of the wave's 16 rows x 32 classes.
        f32x4_t cs[2];
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
          for (int i = 0; i < 4; ++i) cs[mb][i] = 0.0f;
        float nrm[2] = {0.0f, 0.0f};
        u32x4_t af[2][2][2];   // [buffer][k-step of the pair][mb]
        static_for<0, KS / 2>([&](auto pp) {
          constexpr int P = decltype(pp)::value;
          constexpr int BUF = P & 1;
          if constexpr (P == 0) {
            static_for<0, 2>([&](auto kq) {
              constexpr int k2 = decltype(kq)::value;
              ds_read_128<(2 * P + k2) * 64>(af[BUF][k2][0], stg + a_cos);
              ds_read_128<(2 * P + k2) * 64 + 16 * RB>(af[BUF][k2][1], stg + a_cos);
            });
          }
          if constexpr (P + 1 < KS / 2) {
            static_for<0, 2>([&](auto kq) {
              constexpr int k2 = decltype(kq)::value;
              ds_read_128<(2 * (P + 1) + k2) * 64>(af[BUF ^ 1][k2][0], stg + a_cos);
              ds_read_128<(2 * (P + 1) + k2) * 64 + 16 * RB>(af[BUF ^ 1][k2][1], stg + a_cos);
            });
            lgkm_wait<4>(af[BUF][0][0], af[BUF][0][1], af[BUF][1][0], af[BUF][1][1]);
          } else {
            lgkm_wait<0>(af[BUF][0][0], af[BUF][0][1], af[BUF][1][0], af[BUF][1][1]);
          }
          static_for<0, 2>([&](auto kq) {
            constexpr int k2 = decltype(kq)::value;
            constexpr int ks = 2 * P + k2;
            if (ks >= wave * KSW && ks < (wave + 1) * KSW) {
#pragma unroll
              for (int mb = 0; mb < 2; ++mb) {
                nrm[mb] = sumsq2(af[BUF][k2][mb].x, nrm[mb], Tag{});
                nrm[mb] = sumsq2(af[BUF][k2][mb].y, nrm[mb], Tag{});
                nrm[mb] = sumsq2(af[BUF][k2][mb].z, nrm[mb], Tag{});
                nrm[mb] = sumsq2(af[BUF][k2][mb].w, nrm[mb], Tag{});
              }
            }
#pragma unroll
            for (int mb = 0; mb < 2; ++mb) cs[mb] = mfma_16x16x32(af[BUF][k2][mb], xr[ks], cs[mb], Tag{});
          });
        });
        // Partial squared norms of stage rows 16 mb + r16 over the wave's
        // quarter of d: the four lanes q of a row meet, lanes q = 0 publish.
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) {
          nrm[mb] += __shfl_xor(nrm[mb], 16, 64);
          nrm[mb] += __shfl_xor(nrm[mb], 32, 64);
        }
        if (q == 0) {
          ds_write_32<0>(lds_addr(&fxNrm[wave][r16]), __float_as_uint(nrm[0]));
          ds_write_32<64>(lds_addr(&fxNrm[wave][r16]), __float_as_uint(nrm[1]));
        }
        wait_lgkm0();
        stage_barrier();

        // ---- inverse norms of the chunk's rows (every wave its own copy).
        float iwr = 0.0f;
        if (lane < kFxCls) {
          uint32_t p0, p1, p2, p3;
          ds_read_32<0>(p0, lds_addr(&fxNrm[0][lane]));
          ds_read_32<0>(p1, lds_addr(&fxNrm[1][lane]));
          ds_read_32<0>(p2, lds_addr(&fxNrm[2][lane]));
          ds_read_32<0>(p3, lds_addr(&fxNrm[3][lane]));
          lgkm_wait<0>(p0, p1, p2, p3);
          const float ss = (__uint_as_float(p0) + __uint_as_float(p1)) +
                           (__uint_as_float(p2) + __uint_as_float(p3));
          iwr = 1.0f / fmaxf(sqrtf(ss), kEpsNormW);
          ds_write_32<0>(lds_addr(&fxIw[wave][lane]), __float_as_uint(iwr));
          // 1/||w_j|| for the backward (one row tile per split writes them).
          if (rt == 0 && wave == S) {
            const int64_t j = c * kFxCls + fx_sigma(lane);
            inv_w[j] = j < K ? iwr : 0.0f;
          }
        }
        float ratio = 1.0f;   // change of the fp16 coefficient scale
        if constexpr (kF16) {
          const float iw_max = wave_max(iwr);
          if (!(iw_max * sig <= kFp16CoefHeadroom)) {
            const float sn = exp2f(floorf(log2f(kFp16CoefHeadroom / fmaxf(iw_max, 1e-30f))));
            ratio = sn / sig;
            sig = sn;
          }
        }
        wait_lgkm0();
        u32x4_t iv0, iv1;   // 1/||w|| of classes 8q..8q+3 (rows 4q..) and 8q+4.. (rows 16+4q..)
        ds_read_128<0>(iv0, lds_addr(&fxIw[wave][4 * q]));
        ds_read_128<64>(iv1, lds_addr(&fxIw[wave][4 * q]));
        lgkm_wait<0>(iv0, iv1);
        const float iw[8] = {__uint_as_float(iv0.x), __uint_as_float(iv0.y),
                             __uint_as_float(iv0.z), __uint_as_float(iv0.w),
                             __uint_as_float(iv1.x), __uint_as_float(iv1.y),
                             __uint_as_float(iv1.z), __uint_as_float(iv1.w)};

        // ---- epilogue of the lane's row and classes j = 32 c + 8 q + e.
        const int64_t jb = c * kFxCls + 8 * q;
        const int tpos = yh - (int)jb;   // the row's target among the lane's classes, if in [0, 8)
        float f2[8];
        float ct = 0.0f;
        bool has_t = false;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float cv = cs[e >> 2][e & 3] * ix * iw[e];
          float v = cv * s2;
          if (jb + e >= K) v = -INFINITY;
          if (FILT && cv > tau) v = -INFINITY;   // PFC* drops the negative (Eq. noise_filtering)
          if (tpos == e) {
            ct = cv;
            has_t = true;
            v = -INFINITY;   // the margined target logit is merged separately
          }
          f2[e] = v;
        }
        float ft2 = -INFINITY;
        if (has_t) {
          const float ft = target_logit(mg, ct);
          ft2 = ft * kLog2e;
          if (n_row < B) {
            tgt[n_row] = ft;
            tgtc[n_row] = ct;
          }
        }
        float mc = ft2;
#pragma unroll
        for (int e = 0; e < 8; ++e) mc = fmaxf(mc, f2[e]);
        mc = fmaxf(mc, __shfl_xor(mc, 16, 64));
        mc = fmaxf(mc, __shfl_xor(mc, 32, 64));
        float fac = 1.0f;
        if (mc > mref + kRefSlack || (mref == -INFINITY && mc > -INFINITY)) {
          fac = exp2f(mref - mc);   // 0 when there was no reference yet
          mref = mc;
          lpart *= fac;
        }
        const float mr = mref == -INFINITY ? 0.0f : mref;
        float ev[8];
        float lsum = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          ev[e] = __builtin_amdgcn_exp2f(f2[e] - mr);
          lsum += ev[e];
        }
        if (has_t) lsum += __builtin_amdgcn_exp2f(ft2 - mr);
        lpart += lsum;
        eb[S] = u32x4_t{pack_f16x2(ev[0], ev[1]), pack_f16x2(ev[2], ev[3]),
                        pack_f16x2(ev[4], ev[5]), pack_f16x2(ev[6], ev[7])};
        gm[S] = mref;
        // Coefficients of the dX contraction: 2^(f - m) / ||w_j|| (times the
        // fp16 scale), in the operand type.
        {
          float pv[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) pv[e] = ev[e] * (iw[e] * sig);
          const u32x4_t pk{pack2<Tag>(pv[0], pv[1]), pack2<Tag>(pv[2], pv[3]),
                           pack2<Tag>(pv[4], pv[5]), pack2<Tag>(pv[6], pv[7])};
          ds_write_128<0>(p_w, pk);
        }
        if (q == 0) ds_write_32<0>(lds_addr(&fxFac[rho]), __float_as_uint(fac * ratio));
        wait_lgkm0();
        stage_barrier();

        // ---- dX contraction: O[d quarter][64 rows] += W^T[.][32 classes] P'^T.
        uint32_t fv0, fv1;
        ds_read_32<0>(fv0, lds_addr(&fxFac[l32]));
        ds_read_32<128>(fv1, lds_addr(&fxFac[l32]));
        u32x2_t alo[2][MB], ahi[2][MB];
        u32x4_t bq[2][2];
        static_for<0, 2>([&](auto kq) {
          constexpr int kk = decltype(kq)::value;
          static_for<0, MB>([&](auto mm) {
            constexpr int mb = decltype(mm)::value;
            ds_read_tr_b64<64 * mb>(alo[kk][mb], stg + a_tr[kk]);
            ds_read_tr_b64<64 * mb + 16 * RB>(ahi[kk][mb], stg + a_tr[kk]);
          });
          ds_read_128<32 * kk>(bq[kk][0], b_p);
          ds_read_128<32 * kk + 32 * kFxPLd * 2>(bq[kk][1], b_p);
        });
        lgkm_wait<0>(fv0, fv1, alo, ahi, bq[0][0], bq[0][1], bq[1][0], bq[1][1]);
        const float fr[2] = {__uint_as_float(fv0), __uint_as_float(fv1)};
        if (__any(fr[0] != 1.0f || fr[1] != 1.0f)) {
#pragma unroll
          for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int nb = 0; nb < 2; ++nb)
#pragma unroll
              for (int r = 0; r < 16; ++r) acc[mb][nb][r] *= fr[nb];
        }
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
          for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int nb = 0; nb < 2; ++nb)
              acc[mb][nb] = mfma_32x32x16(make_uint4(alo[kk][mb].x, alo[kk][mb].y, ahi[kk][mb].x,
                                                     ahi[kk][mb].y),
                                          as_uint4(bq[kk][nb]), acc[mb][nb], Tag{});
      });
      // ---- end of a 128-class group: E of its chunks relative to the final
      // reference, the reference itself (0 when the row has no live logit).
      const int nv = (int)(c_end - 4 * g < 4 ? c_end - 4 * g : 4);
      const float mr = mref == -INFINITY ? 0.0f : mref;
      if (n_row < B) {
        uint16_t* erow = lbuf + (int64_t)n_row * ld_cos + 4 * g * kFxCls + 8 * q;
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          // Chunks past |S| in the last group hold E = 0.
          u32x4_t v = u32x4_t{0u, 0u, 0u, 0u};
          if (s < nv) {
            v = eb[s];
            if (gm[s] != mref) v = scale_f16x8(v, exp2f((gm[s] == -INFINITY ? 0.0f : gm[s]) - mr));
          }
          __builtin_nontemporal_store(v, reinterpret_cast<u32x4_t*>(erow + s * kFxCls));
        }
        if (q == 0) gmax[g * ld_g + n_row] = mr;
      }
    }
    wait_vmcnt<0>();
  }

  // ---- per (row, split): the reference and the sum, and O / sigma.
  float lt = lpart;
  lt += __shfl_xor(lt, 16, 64);
  lt += __shfl_xor(lt, 32, 64);
  if (q == 0 && n_row < B) stats[(int64_t)n_row * n_split + split] = make_float2(mref, lt);
  const float inv_sig = kF16 ? (sig == INFINITY ? 0.0f : 1.0f / sig) : 1.0f;
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const int n = n0 + 32 * nb + l32;
    if (n >= B) continue;
    float* out = dx_part + ((int64_t)split * B + n) * D;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int i = dbase + 32 * mb + 8 * g4 + 4 * h;
        *reinterpret_cast<float4*>(out + i) =
            make_float4(acc[mb][nb][4 * g4] * inv_sig, acc[mb][nb][4 * g4 + 1] * inv_sig,
                        acc[mb][nb][4 * g4 + 2] * inv_sig, acc[mb][nb][4 * g4 + 3] * inv_sig);
      }
  }
}

template <typename Tag, int D>
void launch_fwdx_d(const StepArgs& a, const StepWs& w, const Margin& mg, hipStream_t stream) {
  const int B = (int)a.B;
  const int n_rt = (int)ceil_div(B, kFxRows);
  const int64_t n_tiles = (int64_t)n_rt * w.n_split;
  const int64_t per_xcd = ceil_div(n_tiles, 8);
  const dim3 grid((unsigned)(8 * per_xcd)), block(kFxThreads);
  if (a.tau < 1.0f)
    hipLaunchKernelGGL((k_fwdx16<Tag, D, true>), grid, block, 0, stream, (const uint16_t*)a.X,
                       (const uint16_t*)a.W, w.act_pad, a.n_active, a.labels_mapped, w.inv_x, B,
                       n_rt, w.n_split, n_tiles, per_xcd, mg, a.tau, w.ld_cos, w.ld_g,
                       (uint16_t*)w.lbuf, w.gmax, w.inv_w, w.stats, w.tgt, w.tgtc, w.dx_part);
  else
    hipLaunchKernelGGL((k_fwdx16<Tag, D, false>), grid, block, 0, stream, (const uint16_t*)a.X,
                       (const uint16_t*)a.W, w.act_pad, a.n_active, a.labels_mapped, w.inv_x, B,
                       n_rt, w.n_split, n_tiles, per_xcd, mg, a.tau, w.ld_cos, w.ld_g,
                       (uint16_t*)w.lbuf, w.gmax, w.inv_w, w.stats, w.tgt, w.tgtc, w.dx_part);
}

template <typename Tag>
void launch_fwdx_tag(const StepArgs& a, const StepWs& w, const Margin& mg, hipStream_t stream) {
  switch (a.d) {
    case 128: launch_fwdx_d<Tag, 128>(a, w, mg, stream); break;
    case 256: launch_fwdx_d<Tag, 256>(a, w, mg, stream); break;
    default: launch_fwdx_d<Tag, 512>(a, w, mg, stream); break;
  }
}

}  // namespace

void launch_fwdx16(const StepArgs& a, const StepWs& w, const Margin& mg, hipStream_t stream) {
  if (a.dtype == 1)
    launch_fwdx_tag<Bf16Tag>(a, w, mg, stream);
  else
    launch_fwdx_tag<F16Tag>(a, w, mg, stream);
}

}  // namespace pfc
