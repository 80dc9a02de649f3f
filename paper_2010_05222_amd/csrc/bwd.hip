// Stage 6: backward through the sampled margin softmax and both
// normalisations, and lazy momentum SGD on the active rows
// (Partial FC Eq. proxy_update, Eq. pfc_center_update, Sec. 3.2.1 matrix form:
// G = (P - Y)/B, dW = X^T G, dX = G W^T, restricted to the active set S).
//
// With dcos = (s/B) g and g_{nj} = (p_{nj} - [j = y_n]) * slope_{nj}, the
// contractions run over the non-target part p_{nj} only (p <= 1, which keeps
// the 16-bit operands in range), rebuilt on the fly from the forward's logit
// store as p = E * gscale (E = 2^(f - m) per row and 128-class group, zero at
// targets and past |S|; gscale = 2^(m - lse log2 e) per row and group).  The
// single target term of each row, (p_t - 1) * slope_t, is added exactly in
// fp32 outside the MFMA loops.
//
// dX (k_dx16): split-K MFMA contraction over classes, dX_hat^T[i][n] =
//   sum_j W[S_j][i] * p_{nj} / ||w_j||.  A workgroup owns 128 batch rows x all
//   of d and a slice of the classes.  The gathered W rows go straight from
//   HBM into a three-stage LDS ring (direct-to-LDS loads) and are read as MFMA
//   operands with transposing LDS reads, so they are never staged in
//   registers.  k_dx_final sums the split partials in a fixed order, adds the
//   target terms and applies the normalisation backward of x.
// dW + update (k_dw16): a workgroup (eight waves, two per SIMD) owns 128
//   active classes x all of d and reduces over the whole batch, so its
//   epilogue has complete rows: target terms, tangent projection, momentum,
//   weight step and the scatter into the persistent W / momentum rows (unique
//   rows, no atomics).  It runs after the dX kernels, which read the old W.
#include <atomic>

#include "pfc_gemm.h"

namespace pfc {
namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr int kBwKC = 32;          // reduction chunk: classes (dX) or batch rows (dW)
constexpr int kRowLd = 528;        // LDS row stride of a DMA'd row of up to 512 (1 KB + 32 B)
constexpr int kRowStage = kBwKC * kRowLd;
constexpr int kDxRows = 128;       // batch rows of a dX workgroup
constexpr int kDwCls = 128;        // classes of a dW workgroup
constexpr int kTLd = 260;         // LDS row stride (floats) of the update's staged gradient rows
constexpr int kHitCap = 256;      // target rows listed per wave of a dW workgroup
constexpr int kGateSpins = 512;   // polls of a dW start gate before the workgroup goes ahead anyway

// Every operand reaches LDS through direct-to-LDS loads into three-stage
// rings (one array per stage, so the compiler can keep later stages in
// flight while a stage is read); the coefficient producer reads the raw
// logit-store values from LDS and writes the 16-bit MFMA operand back to LDS.
//
// dX: W rows, raw logit-store values [128 rows x 32 classes], 1/||w|| of the
// chunk, the rows' scales, and the coefficient tile (K-major, 64-byte rows).
__shared__ __attribute__((aligned(1024))) uint16_t xW0[kRowStage], xW1[kRowStage], xW2[kRowStage];
__shared__ __attribute__((aligned(1024))) int16_t xR0[kDxRows * kBwKC], xR1[kDxRows * kBwKC],
    xR2[kDxRows * kBwKC];
__shared__ __attribute__((aligned(16))) float xI0[kBwKC], xI1[kBwKC], xI2[kBwKC];
__shared__ __attribute__((aligned(16))) float xS0[kDxRows], xS1[kDxRows], xS2[kDxRows];
__shared__ __attribute__((aligned(1024))) uint16_t xG0[kDxRows * kBwKC], xG1[kDxRows * kBwKC],
    xG2[kDxRows * kBwKC];
// dX: active row ids of four chunks (a ring: chunk c in slot c % 4).
__shared__ __attribute__((aligned(16))) int32_t xIds[4][kBwKC];
// dW: X^T rows (K-major: d rows of 32 batch rows, bf16), raw logit-store
// values [32 rows x 128 classes] (16-byte pieces swizzled per row), the rows'
// scales, and the coefficient tile G^T (K-major: 128 class rows of 32 batch
// rows).  After the loop the X^T stages (33 KB each) hold the update's staged
// gradient rows, a coefficient stage the target-row lists.
__shared__ __attribute__((aligned(1024))) uint16_t wX0[kRowStage], wX1[kRowStage], wX2[kRowStage];
__shared__ __attribute__((aligned(1024))) int16_t wR0[kBwKC * kDwCls], wR1[kBwKC * kDwCls],
    wR2[kBwKC * kDwCls];
__shared__ __attribute__((aligned(16))) float wQ0[kBwKC], wQ1[kBwKC], wQ2[kBwKC];
__shared__ __attribute__((aligned(1024))) uint16_t wG0[kDwCls * kBwKC], wG1[kDwCls * kBwKC],
    wG2[kDwCls * kBwKC];

#define PFC_STAGE3(name, T, a0, a1, a2)          \
  template <int S>                               \
  __device__ __forceinline__ T* name() {         \
    if constexpr (S == 0) return a0;             \
    else if constexpr (S == 1) return a1;        \
    else return a2;                              \
  }
PFC_STAGE3(dx_w, uint16_t, xW0, xW1, xW2)
PFC_STAGE3(dx_r, int16_t, xR0, xR1, xR2)
PFC_STAGE3(dx_i, float, xI0, xI1, xI2)
PFC_STAGE3(dx_s, float, xS0, xS1, xS2)
PFC_STAGE3(dx_g, uint16_t, xG0, xG1, xG2)
PFC_STAGE3(dw_x, uint16_t, wX0, wX1, wX2)
PFC_STAGE3(dw_r, int16_t, wR0, wR1, wR2)
PFC_STAGE3(dw_q, float, wQ0, wQ1, wQ2)
PFC_STAGE3(dw_g, uint16_t, wG0, wG1, wG2)
#undef PFC_STAGE3

template <typename Tag>
__device__ __forceinline__ float load16(const void* p, int64_t idx) {
  return to_float<Tag>(((const uint16_t*)p)[idx]);
}

// Target term of a row, (p_t - 1) * slope_t, from its unmargined target cosine.
__device__ __forceinline__ float target_coef(const Margin& mg, float c, float lse) {
  const float p = __expf(target_logit(mg, c) - lse);
  return (p - 1.0f) * target_slope(mg, c);
}

// Scale of the fp16 coefficient operand of dX: a power of two that keeps
// p / ||w_j|| * scale inside the fp16 range for every active class (p <= 1).
__device__ __forceinline__ float dx_operand_scale(F16Tag, float inv_w_max) {
  return exp2f(floorf(log2f(60000.0f / fmaxf(inv_w_max, 1e-30f))));
}
__device__ __forceinline__ float dx_operand_scale(Bf16Tag, float) { return 1.0f; }

// Two floats to a packed pair of 16-bit values, round to nearest even
// (v_cvt_pk_bf16_f32 / v_cvt_f16_f32 on gfx950).
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
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

template <typename Tag>
__device__ __forceinline__ uint4 pack8(const float (&v)[8]) {
  uint4 o;
  o.x = pack2<Tag>(v[0], v[1]);
  o.y = pack2<Tag>(v[2], v[3]);
  o.z = pack2<Tag>(v[4], v[5]);
  o.w = pack2<Tag>(v[6], v[7]);
  return o;
}

// An MFMA operand from the two halves of a transposing read pair.
__device__ __forceinline__ uint4 frag_of(const u32x2_t& lo, const u32x2_t& hi) {
  return make_uint4(lo.x, lo.y, hi.x, hi.y);
}
__device__ __forceinline__ uint4 as_uint4(const u32x4_t& v) { return make_uint4(v.x, v.y, v.z, v.w); }

template <typename T>
__device__ __forceinline__ void zero_acc(T (&acc)[4][2]) {
#pragma unroll
  for (int mb = 0; mb < 4; ++mb)
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mb][nb][r] = 0.0f;
}

// ------------------------------------------------------------------ dX

// D = 128 * WI; 2 * WI waves: wave (wi, wn) owns d entries [128 wi, +128) and
// batch rows [64 wn, +64) of the workgroup's 128 (4 x 2 MFMA blocks).
// Pipeline per chunk c (32 classes): the raw cosines and 1/||w|| of chunk
// c + 3 and the W rows of chunk c + 2 are requested, the coefficients of
// chunk c + 1 are produced, and chunk c is contracted.
template <typename Tag, int WI>
__global__ void __launch_bounds__(128 * WI) k_dx16(
    const uint16_t* __restrict__ W, const int32_t* __restrict__ act_pad,
    const int32_t* __restrict__ n_active_p, const float* __restrict__ inv_w,
    const float* __restrict__ inv_w_max, const uint16_t* __restrict__ lbuf, int64_t ld_cos,
    const float* __restrict__ gscale, int64_t ld_g, int B, int n_rt, int n_split,
    int64_t n_tiles, int64_t per_xcd, float* __restrict__ dx_part) {
  constexpr int D = 128 * WI;
  constexpr int NT = 128 * WI;              // threads
  constexpr int NW = 2 * WI;                // waves
  constexpr int WROWS = kBwKC / NW;         // W rows DMA'd by each wave per chunk
  constexpr int RDMA = 8 / NW;              // 1-KB logit-store blocks DMA'd by each wave
  constexpr int GROUPS = 512 / NT;          // 8-coefficient groups per thread per chunk
  constexpr int PER_ITER = WROWS + RDMA + 3;  // DMAs a wave issues per chunk
  const int64_t t = (int64_t)(blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  if (t >= n_tiles) return;
  // The batch-row tiles of one split share its class range: they run on one
  // XCD so the split's W rows are fetched from HBM once.
  const int split = (int)(t / n_rt);
  const int n0 = (int)(t % n_rt) * kDxRows;
  const int K = *n_active_p;
  const int64_t n_chunks = ceil_div((int64_t)K, (int64_t)kBwKC);
  const int64_t per = ceil_div(n_chunks, (int64_t)n_split);
  const int64_t c_begin = split * per;
  const int64_t c_end = c_begin + per < n_chunks ? c_begin + per : n_chunks;
  const int64_t c_stop =
      c_begin + ceil_div(c_end > c_begin ? c_end - c_begin : 0, (int64_t)3) * 3;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wi = wave >> 1, wn = wave & 1;
  const float scale = dx_operand_scale(Tag{}, *inv_w_max);

  // Coefficient-producer slots of this thread (fixed for the whole kernel):
  // row prow, classes 8 pchunk .. + 7 of each chunk.
  int prow[GROUPS], pchunk[GROUPS];
#pragma unroll
  for (int u = 0; u < GROUPS; ++u) {
    const int q = tid + NT * u;
    prow[u] = q >> 2;
    pchunk[u] = q & 3;
  }
  // Logit-store DMA of this lane: block b holds rows 16 b .. 16 b + 15.
  int64_t rsrc[RDMA];
#pragma unroll
  for (int v = 0; v < RDMA; ++v) {
    const int r = 16 * (wave * RDMA + v) + (lane >> 2);
    const int n = n0 + r < B ? n0 + r : B - 1;
    rsrc[v] = (int64_t)n * ld_cos + 8 * (lane & 3);
  }

  auto dma_raw = [&](auto st, int64_t c) {
    constexpr int S = decltype(st)::value;
    const int64_t jb = (c < n_chunks ? c : n_chunks - 1) * kBwKC;
#pragma unroll
    for (int v = 0; v < RDMA; ++v)
      dma16(lbuf + rsrc[v] + jb, dx_r<S>() + 512 * (wave * RDMA + v));
    // 1/||w|| of the chunk's 32 classes: 8 / NW 16-byte pieces per wave.
    if (lane < 8 / NW) dma16(inv_w + jb + 4 * (wave * (8 / NW) + lane), dx_i<S>() + 4 * wave * (8 / NW));
    // Row scales of the chunk's 128-class group for the 128 rows: 32 / NW pieces per wave.
    const float* gs = gscale + (jb / kLogitGroup) * ld_g + n0;
    if (lane < 32 / NW) dma16(gs + 4 * (wave * (32 / NW) + lane), dx_s<S>() + 4 * wave * (32 / NW));
  };
  // Active-set indices of the W rows this wave DMAs for a chunk.  The first
  // two chunks' come from scalar loads; later chunks' travel with the loads,
  // four chunks ahead, into the index ring (their wait is then the chunk's
  // load wait, not a scalar-load round trip inside the loop).  The padded copy
  // holds a valid row id at every index of a chunk.
  int32_t rows_pf[WROWS];
  auto load_rows = [&](int64_t c) {
    const int64_t jb = (c < n_chunks ? c : n_chunks - 1) * kBwKC;
#pragma unroll
    for (int v = 0; v < WROWS; ++v)
      rows_pf[v] = act_pad[__builtin_amdgcn_readfirstlane((int)(jb + wave * WROWS + v))];
  };
  auto dma_ids = [&](int64_t c) {
    const int64_t jb = (c < n_chunks ? c : n_chunks - 1) * kBwKC;
    if (lane < WROWS / 4) dma16(act_pad + jb + wave * WROWS + 4 * lane, &xIds[c & 3][wave * WROWS]);
  };
  auto read_ids = [&](int64_t c, u32x4_t (&iv)[WROWS / 4]) {
#pragma unroll
    for (int q = 0; q < WROWS / 4; ++q)
      ds_read_128<0>(iv[q], lds_addr(&xIds[c & 3][wave * WROWS + 4 * q]));
  };
  auto rows_of = [&](u32x4_t (&iv)[WROWS / 4]) {
#pragma unroll
    for (int q = 0; q < WROWS / 4; ++q) {
      rows_pf[4 * q + 0] = __builtin_amdgcn_readfirstlane((int)iv[q].x);
      rows_pf[4 * q + 1] = __builtin_amdgcn_readfirstlane((int)iv[q].y);
      rows_pf[4 * q + 2] = __builtin_amdgcn_readfirstlane((int)iv[q].z);
      rows_pf[4 * q + 3] = __builtin_amdgcn_readfirstlane((int)iv[q].w);
    }
  };
  auto dma_w = [&](auto st) {
    constexpr int S = decltype(st)::value;
#pragma unroll
    for (int v = 0; v < WROWS; ++v) {
      const int r = wave * WROWS + v;
      if (lane < D / 8) dma16(W + (int64_t)rows_pf[v] * D + 8 * lane, dx_w<S>() + r * kRowLd);
    }
  };
  // Coefficients of chunk c (K-major, rows of 32 classes): the LDS reads are
  // issued first (produce_load) and consumed later (produce_store), after an
  // lgkm wait that covers them.
  // Coefficient of (row, class): p / ||w_j|| * scale = E * gscale_row * scale * (1/||w_j||);
  // E is 0 at the row's target and past |S|, gscale 0 past the batch, so only
  // chunks past the split's end need masking.
  struct ProdIn {
    u32x4_t qv[GROUPS], i0v[GROUPS], i1v[GROUPS];
    uint32_t sv[GROUPS];
  };
  auto produce_load = [&](auto st, ProdIn& in) {
    constexpr int S = decltype(st)::value;
#pragma unroll
    for (int u = 0; u < GROUPS; ++u) {
      ds_read_128<0>(in.qv[u], lds_addr(dx_r<S>()) + (prow[u] * kBwKC + 8 * pchunk[u]) * 2);
      ds_read_128<0>(in.i0v[u], lds_addr(dx_i<S>()) + 32 * pchunk[u]);
      ds_read_128<16>(in.i1v[u], lds_addr(dx_i<S>()) + 32 * pchunk[u]);
      ds_read_32<0>(in.sv[u], lds_addr(dx_s<S>()) + 4 * prow[u]);
    }
  };
  auto produce_store = [&](auto st, int64_t c, ProdIn& in) {
    constexpr int S = decltype(st)::value;
    const bool cvalid = c < c_end;   // wave-uniform
#pragma unroll
    for (int u = 0; u < GROUPS; ++u) {
      pin_reg(in.qv[u]);
      pin_reg(in.i0v[u]);
      pin_reg(in.i1v[u]);
      pin_reg(in.sv[u]);
      const uint4 q = as_uint4(in.qv[u]);
      const uint32_t qw[4] = {q.x, q.y, q.z, q.w};
      const float iw[8] = {__uint_as_float(in.i0v[u].x), __uint_as_float(in.i0v[u].y),
                           __uint_as_float(in.i0v[u].z), __uint_as_float(in.i0v[u].w),
                           __uint_as_float(in.i1v[u].x), __uint_as_float(in.i1v[u].y),
                           __uint_as_float(in.i1v[u].z), __uint_as_float(in.i1v[u].w)};
      const float sc = cvalid ? __uint_as_float(in.sv[u]) * scale : 0.0f;
      float v[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float ev = (e & 1) ? f16_hi(qw[e >> 1]) : f16_lo(qw[e >> 1]);
        v[e] = ev * (sc * iw[e]);
      }
      const uint4 o = pack8<Tag>(v);
      ds_write_128<0>(lds_addr(dx_g<S>()) + k_major32_offset(prow[u], pchunk[u]) * 2,
                      u32x4_t{o.x, o.y, o.z, o.w});
    }
  };

  // Per-lane byte offsets of the fragment reads (see frag_mn_major and
  // frag_k_major32): W rows MN-major, coefficients K-major.
  const int fg = lane >> 4, fsrc = lane & 15;
  const uint32_t a_lane =
      ((8 * (fg >> 1) + (fsrc >> 2)) * kRowLd + 16 * (fg & 1) + 4 * (fsrc & 3) + 128 * wi) * 2;
  const uint32_t b_lane0 = k_major32_offset(64 * wn + (lane & 31), lane >> 5) * 2;
  const uint32_t b_lane1 = k_major32_offset(64 * wn + (lane & 31), 2 + (lane >> 5)) * 2;

  f32x16_t acc[4][2];
  zero_acc(acc);

  if (c_begin < c_stop) {
    using S0 = std::integral_constant<int, 0>;
    using S1 = std::integral_constant<int, 1>;
    using S2 = std::integral_constant<int, 2>;
    // Prologue: raw data of chunks 0..2, W rows of chunks 0, 1; coefficients of chunk 0.
    load_rows(c_begin);
    dma_raw(S0{}, c_begin);
    dma_w(S0{});
    load_rows(c_begin + 1);
    dma_raw(S1{}, c_begin + 1);
    dma_ids(c_begin + 2);
    dma_ids(c_begin + 3);
    dma_w(S1{});
    dma_raw(S2{}, c_begin + 2);
    wait_vmcnt_lgkm0<2 * (RDMA + 1) + WROWS + 2>();
    stage_barrier();
    ProdIn in0;
    produce_load(S0{}, in0);
    lgkm_wait<0>();
    produce_store(S0{}, c_begin, in0);
    for (int64_t c = c_begin; c < c_stop; c += 3) {
      static_for<0, 3>([&](auto uu) {
        constexpr int u = decltype(uu)::value;
        const int64_t cu = c + u;
        // Landed: W rows of chunk cu, raw data of chunk cu + 1; this wave's
        // coefficient writes of the previous iteration are complete.
        wait_vmcnt_lgkm0<PER_ITER>();
        stage_barrier();
        // The row ids of chunk cu + 2 (landed: requested before the W rows of
        // chunk cu) and the producer's reads of chunk cu + 1 go first
        // (consumed while the first k-step's MFMAs run), then the fragments of
        // chunk cu...
        u32x4_t idv[WROWS / 4];
        read_ids(cu + 2, idv);
        ProdIn pin;
        produce_load(std::integral_constant<int, (u + 1) % 3>{}, pin);
        const uint32_t wb = lds_addr(dx_w<u>()) + a_lane;
        const uint32_t gb0 = lds_addr(dx_g<u>()) + b_lane0;
        const uint32_t gb1 = lds_addr(dx_g<u>()) + b_lane1;
        u32x2_t alo[2][4], ahi[2][4];
        u32x4_t bq[2][2];
        static_for<0, 4>([&](auto mm) {
          constexpr int mb = decltype(mm)::value;
          ds_read_tr_b64<(0 * kRowLd + 32 * mb) * 2>(alo[0][mb], wb);
          ds_read_tr_b64<(4 * kRowLd + 32 * mb) * 2>(ahi[0][mb], wb);
        });
        ds_read_128<0>(bq[0][0], gb0);
        ds_read_128<32 * 64>(bq[0][1], gb0);
        static_for<0, 4>([&](auto mm) {
          constexpr int mb = decltype(mm)::value;
          ds_read_tr_b64<(16 * kRowLd + 32 * mb) * 2>(alo[1][mb], wb);
          ds_read_tr_b64<(20 * kRowLd + 32 * mb) * 2>(ahi[1][mb], wb);
        });
        ds_read_128<0>(bq[1][0], gb1);
        ds_read_128<32 * 64>(bq[1][1], gb1);
        // ... then later chunks' loads; the next coefficients are produced
        // while the first k-step's MFMAs run.
        dma_raw(std::integral_constant<int, u>{}, cu + 3);
        dma_ids(cu + 4);
        static_for<0, 2>([&](auto kq) {
          constexpr int kk = decltype(kq)::value;
          if constexpr (kk == 0) {
            lgkm_wait<10>(alo[0][0], alo[0][1], alo[0][2], alo[0][3], ahi[0][0], ahi[0][1],
                          ahi[0][2], ahi[0][3], bq[0][0], bq[0][1], idv);
            // W rows of chunk cu + 2, from the ids read above.
            rows_of(idv);
            dma_w(std::integral_constant<int, (u + 2) % 3>{});
          } else {
            produce_store(std::integral_constant<int, (u + 1) % 3>{}, cu + 1, pin);
            lgkm_wait<0>(alo[1][0], alo[1][1], alo[1][2], alo[1][3], ahi[1][0], ahi[1][1],
                         ahi[1][2], ahi[1][3], bq[1][0], bq[1][1]);
          }
#pragma unroll
          for (int mb = 0; mb < 4; ++mb)
#pragma unroll
            for (int nb = 0; nb < 2; ++nb)
              acc[mb][nb] = mfma_32x32x16(frag_of(alo[kk][mb], ahi[kk][mb]), as_uint4(bq[kk][nb]),
                                          acc[mb][nb], Tag{});
        });
      });
    }
    wait_vmcnt<0>();
  }

  const float inv_scale = 1.0f / scale;
  const int half = lane >> 5, l32 = lane & 31;
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const int n = n0 + 64 * wn + 32 * nb + l32;
    if (n >= B) continue;
    float* out = dx_part + ((int64_t)split * B + n) * D;
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int i = 128 * wi + 32 * mb + 8 * g + 4 * half;
        *reinterpret_cast<float4*>(out + i) =
            make_float4(acc[mb][nb][4 * g] * inv_scale, acc[mb][nb][4 * g + 1] * inv_scale,
                        acc[mb][nb][4 * g + 2] * inv_scale, acc[mb][nb][4 * g + 3] * inv_scale);
      }
  }
}

// Row scales of the logit store: gscale[g][n] = 2^(m_gn - lse_n log2 e), so that
// E * gscale is the softmax probability (0 for rows past the batch).  A row
// with an empty denominator (lse = -inf: its label is outside the shard and the
// PFC* filter dropped every logit, so all its E are 0) gets scale 0, and with
// it no gradient.  Groups past |S| are never read and are skipped.
__global__ void __launch_bounds__(256) k_scales(const float* __restrict__ gmax,
                                                const float* __restrict__ row_lse, int B,
                                                int64_t ld_g, int64_t n_groups,
                                                const int32_t* __restrict__ n_active_p,
                                                float* __restrict__ gscale) {
  // Four consecutive entries per thread (ld_g is a multiple of 4, so the four
  // rows share one group and the 16-byte accesses are aligned).
  const int64_t i = 4 * ((int64_t)blockIdx.x * blockDim.x + threadIdx.x);
  const int64_t K = *n_active_p;
  if (i >= n_groups * ld_g) return;
  const int64_t g = i / ld_g;
  const int n = (int)(i - g * ld_g);
  if (g * kLogitGroup >= K) return;
  const float4 m4 = *reinterpret_cast<const float4*>(gmax + i);
  const float mv[4] = {m4.x, m4.y, m4.z, m4.w};
  float v[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float lse = n + e < B ? row_lse[n + e] : -INFINITY;
    v[e] = lse > -INFINITY ? __builtin_amdgcn_exp2f(mv[e] - lse * kLog2e) : 0.0f;
  }
  *reinterpret_cast<float4*>(gscale + i) = make_float4(v[0], v[1], v[2], v[3]);
}

// Sum the split partials of a row in split order, add the row's target term
// g_t * W[S_t] / ||w_t||, and apply the normalisation backward:
// dx = (dX_hat - x_hat (x_hat . dX_hat)) / ||x||, dX_hat = (s/B) * sum.  A
// mapped label outside [0, |S|) counts as unowned: no target term, and no
// row of W or of the id list is read for it.
template <typename Tag>
__global__ void __launch_bounds__(256) k_dx_final(
    const float* __restrict__ dx_part, int n_split, const void* __restrict__ X,
    const void* __restrict__ W, const int32_t* __restrict__ active,
    const int32_t* __restrict__ n_active_p,
    const int32_t* __restrict__ yhat, const float* __restrict__ row_lse,
    const float* __restrict__ inv_x, const float* __restrict__ inv_w,
    const float* __restrict__ tgtc, int B, int d, Margin mg, float sB, float* __restrict__ dX) {
  // One workgroup per batch row, thread t owns entries t and t + 256 (d <= 512):
  // the split partials are independent loads, summed in split order.
  __shared__ float red[4];
  const int n = blockIdx.x;
  const int t = threadIdx.x, lane = t & 63;
  const float ix = inv_x[n];
  const int K = *n_active_p;
  const int yt = yhat[n] < K ? yhat[n] : -1;
  float gt = 0.0f;
  int64_t wbase = 0;
  if (yt >= 0) {
    gt = target_coef(mg, tgtc[n], row_lse[n]) * inv_w[yt];
    wbase = (int64_t)active[yt] * d;
  }
  float v[2] = {0.0f, 0.0f}, xh[2] = {0.0f, 0.0f};
  float dot = 0.0f;
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int i = t + 256 * k;
    if (i >= d) continue;
    const float* p = dx_part + (int64_t)n * d + i;
    const int64_t stride = (int64_t)B * d;
    float sum = 0.0f;
    int s = 0;
    for (; s + 8 <= n_split; s += 8) {
      float q[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) q[u] = p[(int64_t)(s + u) * stride];
#pragma unroll
      for (int u = 0; u < 8; ++u) sum += q[u];
    }
    for (; s < n_split; ++s) sum += p[(int64_t)s * stride];
    if (yt >= 0) sum = fmaf(gt, load16<Tag>(W, wbase + i), sum);
    v[k] = sB * sum;
    xh[k] = load16<Tag>(X, (int64_t)n * d + i) * ix;
    dot = fmaf(xh[k], v[k], dot);
  }
  dot = wave_sum(dot);
  if (lane == 0) red[t >> 6] = dot;
  __syncthreads();
  dot = red[0] + red[1] + red[2] + red[3];
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int i = t + 256 * k;
    if (i < d) dX[(int64_t)n * d + i] = ix * (v[k] - xh[k] * dot);
  }
}

// ------------------------------------------------------------------ dW

// D = 128 * WI; eight waves, two per SIMD: wave w owns d entries
// [D/4 (w % 4), +D/4) and classes [64 (w / 4), +64) of the workgroup (MB x 2
// accumulator tiles of 32 x 32), so that a SIMD's second wave issues while
// the first waits at a barrier or on its loads.  Both MFMA operands are
// K-major in LDS, so every fragment is one 16-byte read: X^T from the
// transposed bf16 copy of the batch, and G^T written by the producer.
// Pipeline per chunk c (32 batch rows): raw logit-store values and row
// scales of chunk c + 3 and X^T of chunk c + 2 requested, coefficients of
// chunk c + 1 produced, chunk c contracted.  The second k-step of chunk c is
// contracted at the start of the next chunk, from fragments read in this
// one, so that the matrix pipe is busy while the next fragments arrive.
template <typename Tag, int WI, bool MASTER>
__global__ void __launch_bounds__(512) k_dw16(
    const uint16_t* __restrict__ xbT, int64_t ld_xt, const void* __restrict__ X,
    uint16_t* __restrict__ W, float* __restrict__ W_master, float* __restrict__ M,
    const int32_t* __restrict__ active, const int32_t* __restrict__ n_active_p,
    const int32_t* __restrict__ yhat, const float* __restrict__ row_lse,
    const float* __restrict__ inv_x, const float* __restrict__ inv_w,
    const float* __restrict__ tgtc, const uint16_t* __restrict__ lbuf, int64_t ld_cos,
    const float* __restrict__ gscale, int64_t ld_g, int B, Margin mg, float sB, float lr,
    float mu, int32_t* __restrict__ gate, int n_gate, int epoch) {
  constexpr int D = 128 * WI;
  constexpr int NW = 8;
  constexpr int DW = D / 4;             // d entries of a wave
  constexpr int CW = kDwCls / 2;        // classes of a wave
  constexpr int MB = DW / 32;           // 32-entry d blocks of a wave
  constexpr int NB = CW / 32;           // 32-class blocks of a wave
  constexpr int XDMA = D / 16 / NW;     // X^T loads (16 d rows each) per wave per chunk
  constexpr int RDMA = 8 / NW;          // logit-store loads (4 rows each) per wave
  constexpr int QL = 8 / NW;            // row-scale pieces (4 rows each) per wave
  constexpr int GROUPS = 1;             // producer slots per thread (512 / 512)
  constexpr int PER_ITER = XDMA + RDMA + 1;
  constexpr int NF = MB + NB;           // fragment reads per k-step
  static_assert(PER_ITER + 2 * (RDMA + 1) < 64, "vmcnt range");
  const int K = *n_active_p;
  const int64_t j0 = (int64_t)blockIdx.x * kDwCls;
  if (j0 >= K) return;
  // Start gates (n_gate > 0 on a long grid, one workgroup per CU): workgroup
  // 2 i + 1 of the first wave starts once workgroup 2 i has finished its
  // contraction, which it signals by writing this launch's number to gate[i].
  // Otherwise all CUs run the contraction and then the memory-bound update in
  // step for the first few hundred microseconds, and the updates, all at
  // once, saturate HBM; with the gates about half of the CUs update at any
  // time from the start.  The wait is bounded (kGateSpins polls), and the
  // results never depend on it: a gate that is never opened, or holds the
  // number by chance, only changes when the workgroup starts.
  const bool gated = (int)blockIdx.x < 2 * n_gate;
  if (gated && (blockIdx.x & 1)) {
    if (threadIdx.x == 0) {
      const int32_t* g = gate + blockIdx.x / 2;
      for (int it = 0; it < kGateSpins; ++it) {
        if (__hip_atomic_load(g, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == epoch) break;
        __builtin_amdgcn_s_sleep(8);
      }
    }
    __syncthreads();
  }

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wd = wave & 3, wc = wave >> 2;   // the wave's d quarter and class half
  const int half = lane >> 5, l32 = lane & 31;
  const int n_chunks = (int)ceil_div(B, kBwKC);
  const int c_stop = (int)ceil_div(n_chunks, 3) * 3;
  // The tile is one 128-class group of the logit store: its row scales.
  const float* gsc = gscale + (j0 / kLogitGroup) * ld_g;
  // Row ids and 1/||w|| of the tile's classes for the update, requested now
  // so that they have long arrived when the update forms its row addresses:
  // lane l holds classes l (u = 0) and 64 + l (u = 1).
  int act_l[2];
  float iw_l[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int64_t j = j0 + 64 * u + lane;
    act_l[u] = j < K ? active[j] : 0;
    iw_l[u] = j < K ? inv_w[j] : 0.0f;
  }

  // Producer slots: a 16-lane group owns 16 classes x 8 batch rows of a chunk;
  // lane gi of the group owns class 16 cb + gi.
  const int grp = lane >> 4, gi = lane & 15;
  int pcls[GROUPS], prg[GROUPS];
  uint32_t ptr_off[GROUPS];   // byte offset of the lane's transposing raw read
#pragma unroll
  for (int u = 0; u < GROUPS; ++u) {
    const int s = 4 * wave + grp + 16 * u;
    const int cb = s >> 2;
    pcls[u] = 16 * cb + gi;
    prg[u] = s & 3;
    // Lane 4 e + q of the group points at row 8 rg + e, classes 16 cb + 4 q .. + 3
    // (16-byte piece 2 cb + q / 2, stored at piece ^ 2 (row & 3)), half q & 1.
    const int e = gi >> 2, q = gi & 3;
    const int r = 8 * prg[u] + e;
    ptr_off[u] = (uint32_t)(r * kDwCls * 2 + 16 * ((2 * cb + (q >> 1)) ^ (2 * (r & 3))) + 8 * (q & 1));
  }

  // Raw logit-store values: load v of this wave covers rows 4 b .. 4 b + 3
  // (b = wave RDMA + v); lane l fills piece l % 16 of row 4 b + l / 16 with
  // source piece (l % 16) ^ 2 (row & 3).
  auto dma_raw_piece = [&](auto st, int c, int v) __attribute__((always_inline)) {
    constexpr int S = decltype(st)::value;
    const int cc = c < n_chunks ? c : n_chunks - 1;
    const int blk = wave * RDMA + v;
    const int r = 4 * blk + (lane >> 4);
    int n = cc * kBwKC + r;
    n = n < B ? n : B - 1;
    const int piece = (lane & 15) ^ (2 * (r & 3));
    dma16(lbuf + (int64_t)n * ld_cos + j0 + 8 * piece, dw_r<S>() + 512 * blk);
  };
  // Row scales of the chunk: QL 16-byte pieces (4 rows each) per wave; rows < ld_g always.
  auto dma_scale = [&](auto st, int c) __attribute__((always_inline)) {
    constexpr int S = decltype(st)::value;
    const int cc = c < n_chunks ? c : n_chunks - 1;
    if (lane < QL) dma16(gsc + cc * kBwKC + 4 * (QL * wave + lane), dw_q<S>() + 4 * QL * wave);
  };
  auto dma_raw = [&](auto st, int c) __attribute__((always_inline)) {
#pragma unroll
    for (int v = 0; v < RDMA; ++v) dma_raw_piece(st, c, v);
    dma_scale(st, c);
  };
  // X^T: block cc of the transposed batch ([d][32], contiguous); load v of this
  // wave covers d rows 16 m .. 16 m + 15 (m = wave XDMA + v), 4 pieces each;
  // lane l fills piece l & 3 of row 16 m + l / 4 with source piece
  // (l & 3) ^ ((row >> 2) & 3).
  auto dma_x_piece = [&](auto st, int c, int v) __attribute__((always_inline)) {
    constexpr int S = decltype(st)::value;
    const int cc = c < n_chunks ? c : n_chunks - 1;
    const int m = wave * XDMA + v;
    const int i = 16 * m + (lane >> 2);
    const int piece = (lane & 3) ^ ((i >> 2) & 3);
    dma16(xbT + ((int64_t)cc * D + i) * kBwKC + 8 * piece, dw_x<S>() + 512 * m);
  };
  auto dma_x = [&](auto st, int c) __attribute__((always_inline)) {
#pragma unroll
    for (int v = 0; v < XDMA; ++v) dma_x_piece(st, c, v);
  };
  // Coefficients of chunk c: G^T[class][row] = p = E * gscale_row (the operand
  // X^T holds x_hat, so no 1/||x|| here).  E is 0 at targets and past |S|,
  // gscale 0 past the batch.  The LDS reads are issued first (produce_load)
  // and consumed later (produce_store), after an lgkm wait that covers them.
  struct ProdIn {
    u32x2_t qlo[GROUPS], qhi[GROUPS];
    u32x4_t sq[GROUPS][2];
  };
  auto produce_load = [&](auto st, ProdIn& in) {
    constexpr int S = decltype(st)::value;
#pragma unroll
    for (int u = 0; u < GROUPS; ++u) {
      const uint32_t ra = lds_addr(dw_r<S>()) + ptr_off[u];
      ds_read_tr_b64<0>(in.qlo[u], ra);
      ds_read_tr_b64<4 * kDwCls * 2>(in.qhi[u], ra);
      const uint32_t qa = lds_addr(dw_q<S>()) + 32 * prg[u];
      ds_read_128<0>(in.sq[u][0], qa);
      ds_read_128<16>(in.sq[u][1], qa);
    }
  };
  auto pin_group = [&](ProdIn& in, int u) __attribute__((always_inline)) {
    pin_reg(in.qlo[u]);
    pin_reg(in.qhi[u]);
    pin_reg(in.sq[u][0]);
    pin_reg(in.sq[u][1]);
  };
  // Group u's coefficients into stage S; gmask 0 writes zeros (a chunk past
  // the batch, whose MFMAs then add nothing).
  auto produce_group = [&](auto st, ProdIn& in, int u, uint32_t gmask) __attribute__((always_inline)) {
    constexpr int S = decltype(st)::value;
    const uint32_t qw[4] = {in.qlo[u].x, in.qlo[u].y, in.qhi[u].x, in.qhi[u].y};
    const float sc[8] = {__uint_as_float(in.sq[u][0].x), __uint_as_float(in.sq[u][0].y),
                         __uint_as_float(in.sq[u][0].z), __uint_as_float(in.sq[u][0].w),
                         __uint_as_float(in.sq[u][1].x), __uint_as_float(in.sq[u][1].y),
                         __uint_as_float(in.sq[u][1].z), __uint_as_float(in.sq[u][1].w)};
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float ev = (e & 1) ? f16_hi(qw[e >> 1]) : f16_lo(qw[e >> 1]);
      v[e] = ev * sc[e];
    }
    const uint4 o = pack8<Bf16Tag>(v);
    const int cl = pcls[u];
    ds_write_128<0>(lds_addr(dw_g<S>()) + cl * kBwKC * 2 + 16 * (prg[u] ^ ((cl >> 2) & 3)),
                    u32x4_t{o.x & gmask, o.y & gmask, o.z & gmask, o.w & gmask});
  };

  // Fragment byte offsets: operand row (d entry or class) 32 q + l32 of the
  // wave's block, chunk 2 kk + half stored at chunk ^ ((row >> 2) & 3).
  const int sw = (l32 >> 2) & 3;
  const uint32_t a_lane0 = (uint32_t)((DW * wd + l32) * kBwKC * 2 + 16 * ((0 + half) ^ sw));
  const uint32_t a_lane1 = (uint32_t)((DW * wd + l32) * kBwKC * 2 + 16 * ((2 + half) ^ sw));
  const uint32_t b_lane0 = (uint32_t)((CW * wc + l32) * kBwKC * 2 + 16 * ((0 + half) ^ sw));
  const uint32_t b_lane1 = (uint32_t)((CW * wc + l32) * kBwKC * 2 + 16 * ((2 + half) ^ sw));

  f32x16_t acc[MB][NB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mb][nb][r] = 0.0f;
  // Second k-step fragments, carried from one chunk to the next.
  u32x4_t a1[MB], b1[NB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) a1[mb] = u32x4_t{0, 0, 0, 0};
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) b1[nb] = u32x4_t{0, 0, 0, 0};

  {
    using S0 = std::integral_constant<int, 0>;
    using S1 = std::integral_constant<int, 1>;
    using S2 = std::integral_constant<int, 2>;
    dma_raw(S0{}, 0);
    dma_x(S0{}, 0);
    dma_raw(S1{}, 1);
    dma_x(S1{}, 1);
    dma_raw(S2{}, 2);
    wait_vmcnt_lgkm0<2 * (RDMA + 1) + XDMA>();
    stage_barrier();
    ProdIn in0;
    produce_load(S0{}, in0);
    lgkm_wait<0>();
#pragma unroll
    for (int u = 0; u < GROUPS; ++u) {
      pin_group(in0, u);
      produce_group(S0{}, in0, u, 0xFFFFFFFFu);
    }
  }
  // Instruction slots of a chunk: NMF MFMAs per k-step, each followed by
  // the work placed after it, so that the wave issues its other instructions
  // while the matrix pipe works through the MFMAs already issued.
  constexpr int NMF = MB * NB;
  constexpr int W_AT = NMF >= 16 ? 3 : NMF / 4;      // wait for the chunk's fragment and producer reads
  constexpr int G0_AT = NMF / 2 - 1;                 // coefficient group 0 written
  constexpr int G1_AT = NMF - 2 > G0_AT ? NMF - 2 : G0_AT + 1;  // group 1 written
  constexpr int NITEM = RDMA + 1 + XDMA + NF;        // loads and reads spread over the second k-step
  static_assert(G1_AT < NMF, "slots");
  for (int c = 0; c < c_stop; c += 3) {
    static_for<0, 3>([&](auto uu) {
      constexpr int u = decltype(uu)::value;
      using SU = std::integral_constant<int, u>;
      using SN = std::integral_constant<int, (u + 1) % 3>;
      using SX = std::integral_constant<int, (u + 2) % 3>;
      const int cu = c + u;
      // Landed: X^T of chunk cu, raw data of chunk cu + 1; this wave's
      // coefficient writes and second k-step reads of the previous chunk are
      // complete.
      wait_vmcnt_lgkm0<PER_ITER>();
      stage_barrier();
      const uint32_t xs = lds_addr(dw_x<u>());
      const uint32_t gs = lds_addr(dw_g<u>());
      u32x4_t a0[MB], b0[NB];
      static_for<0, MB>([&](auto mm) {
        constexpr int mb = decltype(mm)::value;
        ds_read_128<32 * mb * kBwKC * 2>(a0[mb], xs + a_lane0);
      });
      static_for<0, NB>([&](auto nn) {
        constexpr int nb = decltype(nn)::value;
        ds_read_128<32 * nb * kBwKC * 2>(b0[nb], gs + b_lane0);
      });
      ProdIn pin;
      produce_load(SN{}, pin);
      const uint32_t gmask = cu + 1 < n_chunks ? 0xFFFFFFFFu : 0u;
      // Second k-step of the previous chunk (fragments landed before the
      // barrier), with the next chunk's coefficients produced alongside.
      pin_reg(a1);
      pin_reg(b1);
      static_for<0, NMF>([&](auto ii) {
        constexpr int i = decltype(ii)::value;
        acc[i / NB][i % NB] = mfma_32x32x16(as_uint4(a1[i / NB]), as_uint4(b1[i % NB]), acc[i / NB][i % NB], Bf16Tag{});
        if constexpr (i == W_AT) {
          lgkm_wait<0>(a0, b0);
          pin_group(pin, 0);
        }
        if constexpr (i == G0_AT) produce_group(SN{}, pin, 0, gmask);
        if constexpr (GROUPS > 1 && i == G0_AT + 1) pin_group(pin, 1);
        if constexpr (GROUPS > 1 && i == G1_AT) produce_group(SN{}, pin, 1, gmask);
      });
      // First k-step of this chunk, with the loads of later chunks and this
      // chunk's second k-step reads spread over its slots.
      static_for<0, NMF>([&](auto ii) {
        constexpr int i = decltype(ii)::value;
        acc[i / NB][i % NB] = mfma_32x32x16(as_uint4(a0[i / NB]), as_uint4(b0[i % NB]), acc[i / NB][i % NB], Bf16Tag{});
        static_for<(i * NITEM + NMF - 1) / NMF, ((i + 1) * NITEM + NMF - 1) / NMF>([&](auto kk) {
          constexpr int k = decltype(kk)::value;
          if constexpr (k < RDMA) {
            dma_raw_piece(SU{}, cu + 3, k);
          } else if constexpr (k == RDMA) {
            dma_scale(SU{}, cu + 3);
          } else if constexpr (k < RDMA + 1 + XDMA) {
            dma_x_piece(SX{}, cu + 2, k - RDMA - 1);
          } else if constexpr (k < RDMA + 1 + XDMA + MB) {
            constexpr int mb = k - RDMA - 1 - XDMA;
            ds_read_128<32 * mb * kBwKC * 2>(a1[mb], xs + a_lane1);
          } else {
            constexpr int nb = k - RDMA - 1 - XDMA - MB;
            ds_read_128<32 * nb * kBwKC * 2>(b1[nb], gs + b_lane1);
          }
        });
      });
    });
  }
  wait_vmcnt<0>();
  wait_lgkm0();
  // Second k-step of the last chunk (zero coefficients past the batch).
  pin_reg(a1);
  pin_reg(b1);
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
      acc[mb][nb] = mfma_32x32x16(as_uint4(a1[mb]), as_uint4(b1[nb]), acc[mb][nb], Bf16Tag{});
  if (gated && !(blockIdx.x & 1) && threadIdx.x == 0)
    __hip_atomic_store(gate + blockIdx.x / 2, epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);

  // ---- update: the tile goes through LDS in four passes of 32 classes so
  // that each wave then owns whole rows: W, momentum and master rows are read
  // and written in full contiguous segments.  Pass p holds the classes
  // 32 p + r (r < 32); entry d of row r sits in stage array d / 256 at
  // r * kTLd + d % 256.  Wave w owns rows 4 w .. 4 w + 3 of each pass; lane l
  // owns d = 256 h + 4 l .. + 3.  A wave's rows of a pass are loaded while
  // the previous pass is updated, one row after each row written.
  constexpr int NH = D > 256 ? 2 : 1;         // 256-entry halves of a row
  constexpr int LPH = (D > 256 ? 256 : D) / 4;  // lanes that own entries
  constexpr int RPW = 32 / NW;                // rows of a pass per wave
  float* const tlo = reinterpret_cast<float*>(wX0);
  float* const thi = reinterpret_cast<float*>(wX1);
  const bool lane_on = LPH == 64 || lane < LPH;
  const int kt = (int)(K - j0);               // classes of the tile that exist (>= 1)
  int* const hits = reinterpret_cast<int*>(wG0);   // NW lists of kHitCap entries
  int* const hit_n = reinterpret_cast<int*>(wQ0);  // their lengths
  static_assert(NW * kHitCap * 4 <= kDwCls * kBwKC * 2, "hit lists fit a coefficient stage");

  // A wave's rows of one pass.  Row ids, 1/||w|| and the count of rows that
  // exist are wave-uniform; a row past |S| reads row 0 and is not updated.
  struct Rows {
    uint2 wv[RPW][NH];   // four 16-bit weights
    float4 mv[RPW][NH], pv[MASTER ? RPW : 1][NH];
    int row[RPW];
    float iwr[RPW];
    int nv;              // rows k < nv exist
  };
  auto set_rows = [&](Rows& bt, int p) __attribute__((always_inline)) {
    const int cb = 32 * p + RPW * wave;   // tile offset of the wave's first class of the pass
    bt.nv = kt - cb < 0 ? 0 : (kt - cb > RPW ? RPW : kt - cb);
  };
  auto load_row = [&](Rows& bt, int p, int k) __attribute__((always_inline)) {
    const int src = 32 * (p & 1) + RPW * wave + k;   // lane that holds class 32 p + RPW wave + k
    bt.row[k] = __builtin_amdgcn_readlane(act_l[p >> 1], src);
    bt.iwr[k] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(iw_l[p >> 1]), src));
    const int64_t rb = (int64_t)bt.row[k] * D;   // uniform row base
#pragma unroll
    for (int h = 0; h < NH; ++h) {
      const uint32_t o = 256u * h + 4u * (uint32_t)lane;
      bt.wv[k][h] = make_uint2(0, 0);
      bt.mv[k][h] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
      if constexpr (MASTER) bt.pv[k][h] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
      if (lane_on) {
        // Non-temporal: each row is read once here and written back once.
        const u32x2_t w2 = __builtin_nontemporal_load(
            reinterpret_cast<const u32x2_t*>(reinterpret_cast<const char*>(W + rb) + 2 * o));
        const f32x4_t m4 = __builtin_nontemporal_load(
            reinterpret_cast<const f32x4_t*>(reinterpret_cast<const char*>(M + rb) + 4 * o));
        bt.wv[k][h] = make_uint2(w2.x, w2.y);
        bt.mv[k][h] = make_float4(m4.x, m4.y, m4.z, m4.w);
        if constexpr (MASTER) {
          const f32x4_t p4 = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(
              reinterpret_cast<const char*>(W_master + rb) + 4 * o));
          bt.pv[k][h] = make_float4(p4.x, p4.y, p4.z, p4.w);
        }
      }
    }
  };
  auto load_rows = [&](Rows& bt, int p) __attribute__((always_inline)) {
    set_rows(bt, p);
#pragma unroll
    for (int k = 0; k < RPW; ++k) load_row(bt, p, k);
  };
  // Pass p's classes are block p % 2 of the waves of class half p / 2.
  auto park = [&](auto pp) __attribute__((always_inline)) {
    constexpr int p = decltype(pp)::value;
    if (wc != p / 2) return;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int d0 = DW * wd + 32 * mb + 8 * g + 4 * half;
        *reinterpret_cast<float4*>((d0 >= 256 ? thi : tlo) + l32 * kTLd + (d0 & 255)) =
            make_float4(acc[mb][p % 2][4 * g], acc[mb][p % 2][4 * g + 1],
                        acc[mb][p % 2][4 * g + 2], acc[mb][p % 2][4 * g + 3]);
      }
  };
  // Target term of batch row nn added to staged row r (this wave's own row).
  auto add_target = [&](int nn, int r) {
    const float gt = target_coef(mg, tgtc[nn], row_lse[nn]) * inv_x[nn];
    if (!lane_on) return;
#pragma unroll
    for (int h = 0; h < NH; ++h) {
      const uint2 x4 = *reinterpret_cast<const uint2*>(
          reinterpret_cast<const uint16_t*>(X) + (int64_t)nn * D + 256 * h + 4 * lane);
      float4* t = reinterpret_cast<float4*>((h ? thi : tlo) + r * kTLd + 4 * lane);
      float4 a = *t;
      a.x = fmaf(gt, to_float<Tag>((uint16_t)(x4.x & 0xFFFF)), a.x);
      a.y = fmaf(gt, to_float<Tag>((uint16_t)(x4.x >> 16)), a.y);
      a.z = fmaf(gt, to_float<Tag>((uint16_t)(x4.y & 0xFFFF)), a.z);
      a.w = fmaf(gt, to_float<Tag>((uint16_t)(x4.y >> 16)), a.w);
      *t = a;
    }
  };
  auto wf_of = [&](uint2 w4) __attribute__((always_inline)) {
    return make_float4(to_float<Tag>((uint16_t)(w4.x & 0xFFFF)), to_float<Tag>((uint16_t)(w4.x >> 16)),
                       to_float<Tag>((uint16_t)(w4.y & 0xFFFF)), to_float<Tag>((uint16_t)(w4.y >> 16)));
  };
  // Row update, with a = the staged row (dL/dw_hat = sB a), w_hat = w / ||w||:
  // g_w = (sB a - w_hat (w_hat . sB a)) / ||w|| = ga a - gb w,
  // ga = sB / ||w||, gb = ga (w . a) / ||w||^2; then momentum and the step.
  // With PN < 4 each row's registers are refilled, right after the row is
  // written, with the same row of pass PN: the next pass's loads spread over
  // this pass's arithmetic and stores instead of queueing behind them.
  auto update_rows = [&](Rows& bt, auto pn_c) __attribute__((always_inline)) {
    constexpr int PN = decltype(pn_c)::value;
    // The dots w . a of all of this wave's rows first, then their reductions.
    float dots[RPW];
#pragma unroll
    for (int k = 0; k < RPW; ++k) {
      const int r = RPW * wave + k;
      float dot = 0.0f;
#pragma unroll
      for (int h = 0; h < NH; ++h) {
        if (!lane_on) continue;
        const float4 wf = wf_of(bt.wv[k][h]);
        const float4 a4 = *reinterpret_cast<const float4*>((h ? thi : tlo) + r * kTLd + 4 * lane);
        dot = fmaf(wf.x, a4.x, dot);
        dot = fmaf(wf.y, a4.y, dot);
        dot = fmaf(wf.z, a4.z, dot);
        dot = fmaf(wf.w, a4.w, dot);
      }
      dots[k] = dot;
    }
#pragma unroll
    for (int k = 0; k < RPW; ++k) dots[k] = wave_total(dots[k]);
    const int nv = bt.nv;
    if constexpr (PN < 4) set_rows(bt, PN);
#pragma unroll
    for (int k = 0; k < RPW; ++k) {
      const int r = RPW * wave + k;
      if (k < nv) {
        const float ga = sB * bt.iwr[k];
        const float gb = ga * bt.iwr[k] * bt.iwr[k] * dots[k];
        // Uniform row base, made opaque so that the stores below address it as
        // base + lane offset instead of sharing the loads' 64-bit addresses.
        int rw = bt.row[k];
        asm volatile("" : "+s"(rw));
        const int64_t rb = (int64_t)rw * D;
#pragma unroll
        for (int h = 0; h < NH; ++h) {
          if (!lane_on) continue;
          const uint32_t o = 256u * h + 4u * (uint32_t)lane;
          const float4 wf = wf_of(bt.wv[k][h]);
          const float4 a4 = *reinterpret_cast<const float4*>((h ? thi : tlo) + r * kTLd + 4 * lane);
          const float wo[4] = {wf.x, wf.y, wf.z, wf.w};
          const float ao[4] = {a4.x, a4.y, a4.z, a4.w};
          float mo[4] = {bt.mv[k][h].x, bt.mv[k][h].y, bt.mv[k][h].z, bt.mv[k][h].w};
          float po[4] = {0.0f, 0.0f, 0.0f, 0.0f};
          if constexpr (MASTER) {
            po[0] = bt.pv[k][h].x;
            po[1] = bt.pv[k][h].y;
            po[2] = bt.pv[k][h].z;
            po[3] = bt.pv[k][h].w;
          }
          float wn[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float gr = fmaf(-gb, wo[e], ga * ao[e]);
            mo[e] = fmaf(mu, mo[e], gr);
            if constexpr (MASTER) {
              po[e] = fmaf(-lr, mo[e], po[e]);
              wn[e] = po[e];
            } else {
              wn[e] = fmaf(-lr, mo[e], wo[e]);
            }
          }
          *reinterpret_cast<float4*>(reinterpret_cast<char*>(M + rb) + 4 * o) =
              make_float4(mo[0], mo[1], mo[2], mo[3]);
          if constexpr (MASTER)
            *reinterpret_cast<float4*>(reinterpret_cast<char*>(W_master + rb) + 4 * o) =
                make_float4(po[0], po[1], po[2], po[3]);
          uint2 ov;
          ov.x = pack2<Tag>(wn[0], wn[1]);
          ov.y = pack2<Tag>(wn[2], wn[3]);
          *reinterpret_cast<uint2*>(reinterpret_cast<char*>(W + rb) + 2 * o) = ov;
        }
      }
      if constexpr (PN < 4) load_row(bt, PN, k);
    }
  };

  // One row set in registers: pass p's rows, refilled row by row with pass
  // p + 1 (requesting two passes ahead measured no faster: the update's
  // loads and stores are bound by the HBM read-modify-write rate).
  Rows bat;
  load_rows(bat, 0);
  stage_barrier();  // every wave's fragment reads of the stage arrays are done
  // Target terms: wave w lists, in row order, the rows n of its quarter of the
  // batch whose label is one of the tile's classes (entry n * 128 + class
  // offset).  A quarter with more than kHitCap such rows makes each wave scan
  // all labels instead.  Either way the terms are added to the staged
  // gradient rows by the wave that owns the row, in increasing n.
  {
    const int q0 = (int)((int64_t)B * wave / NW), q1 = (int)((int64_t)B * (wave + 1) / NW);
    int cnt = 0;
    for (int nbase = q0; nbase < q1; nbase += 64) {
      const int n = nbase + lane;
      const int yv = n < q1 ? yhat[n] : -1;
      const bool hit = yv >= j0 && yv < j0 + kDwCls;
      const uint64_t mask = __ballot(hit);
      const int pos = cnt + __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                                      __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0));
      if (hit && pos < kHitCap) hits[kHitCap * wave + pos] = n * kDwCls + (int)(yv - j0);
      cnt += __popcll(mask);
    }
    if (lane == 0) hit_n[wave] = cnt;
  }
  park(std::integral_constant<int, 0>{});
  wait_lgkm0();
  stage_barrier();
  int hn[NW];
  bool hit_scan = false;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    hn[w] = __builtin_amdgcn_readfirstlane(hit_n[w]);
    hit_scan |= hn[w] > kHitCap;
  }
  static_for<0, 4>([&](auto pp) {
    constexpr int p = decltype(pp)::value;
    if constexpr (p > 0) {
      wait_lgkm0();
      stage_barrier();  // the stage arrays are rewritten by this pass
      park(pp);
      wait_lgkm0();
      stage_barrier();
    }
    // This wave's rows of the pass: class offsets c0 .. c0 + RPW - 1.
    const int c0 = 32 * p + RPW * wave;
    if (!hit_scan) {
      for (int w = 0; w < NW; ++w)
        for (int i = 0; i < hn[w]; ++i) {
          const int ent = hits[kHitCap * w + i];
          const int ct = ent & (kDwCls - 1);
          if (ct >= c0 && ct < c0 + RPW) add_target(ent / kDwCls, ct & 31);
        }
    } else {
      for (int nbase = 0; nbase < B; nbase += 64) {
        const int n = nbase + lane;
        const int yv = n < B ? yhat[n] : -1;
        uint64_t mask = __ballot(yv >= j0 + c0 && yv < j0 + c0 + RPW);
        while (mask) {
          const int bit = __ffsll((unsigned long long)mask) - 1;
          mask &= mask - 1;
          const int yt = __shfl(yv, bit, 64);
          add_target(nbase + bit, (int)(yt - j0) & 31);
        }
      }
    }
    update_rows(bat, std::integral_constant<int, p + 1>{});
  });
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

__global__ void __launch_bounds__(256) k_dx_final32(const float* __restrict__ dx_part,
                                                    const float* __restrict__ X,
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
      v[k] = sB * dx_part[(int64_t)n * d + i];
      xh[k] = X[(int64_t)n * d + i] * ix;
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

// Compute units of the current device (0 if the query fails).
int device_cu_count() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  return n;
}

template <typename Tag, int WI>
void launch_bwd16(const StepArgs& a, const StepWs& w, const Margin& mg, float sB,
                  hipStream_t stream) {
  const int B = (int)a.B;
  // Start gates on grids of at least four waves of one workgroup per CU; each
  // launch writes a number of its own to the gates it opens.
  static std::atomic<int> launches{0};
  const int n_cu = device_cu_count();
  const int64_t dw_grid = ceil_div(a.cap, kDwCls);
  const int n_gate = (n_cu > 0 && dw_grid >= 4LL * n_cu) ? (n_cu / 2 < kDwGates ? n_cu / 2 : kDwGates) : 0;
  const int epoch = 1 + (launches.fetch_add(1, std::memory_order_relaxed) & 0x3FFFFFFF);
  const int n_rt = (int)ceil_div(B, kDxRows);
  const int64_t n_tiles = (int64_t)n_rt * w.n_split;
  const int64_t per_xcd = ceil_div(n_tiles, 8);
  timing_start(4, stream);
  // Row scales of the logit store from the lse the gradient is normalised with.
  hipLaunchKernelGGL(k_scales, dim3((unsigned)ceil_div(w.n_groups * w.ld_g, 4 * 256)), dim3(256), 0,
                     stream, w.gmax, a.row_lse, B, w.ld_g, w.n_groups, a.n_active, w.gscale);
  hipLaunchKernelGGL((k_dx16<Tag, WI>), dim3((unsigned)(8 * per_xcd)), dim3(128 * WI), 0, stream,
                     (const uint16_t*)a.W, w.act_pad, a.n_active, w.inv_w, w.inv_w_max,
                     (const uint16_t*)w.lbuf, w.ld_cos, w.gscale, w.ld_g, B, n_rt, w.n_split,
                     n_tiles, per_xcd, w.dx_part);
  timing_stop(4, stream);
  timing_start(5, stream);
  hipLaunchKernelGGL(k_dx_final<Tag>, dim3((unsigned)B), dim3(256), 0, stream,
                     w.dx_part, w.n_split, a.X, a.W, a.active, a.n_active, a.labels_mapped,
                     a.row_lse, w.inv_x, w.inv_w, w.tgtc, B, (int)a.d, mg, sB, a.dX);
  timing_stop(5, stream);
  timing_start(6, stream);
  if (a.W_master)
    hipLaunchKernelGGL((k_dw16<Tag, WI, true>), dim3((unsigned)dw_grid), dim3(512),
                       0, stream, (const uint16_t*)w.xbT, w.ld_xt, a.X, (uint16_t*)a.W, a.W_master,
                       a.M, a.active, a.n_active, a.labels_mapped, a.row_lse, w.inv_x, w.inv_w,
                       w.tgtc, (const uint16_t*)w.lbuf, w.ld_cos, w.gscale, w.ld_g, B, mg, sB, a.lr,
                       a.mu, w.dw_gate, n_gate, epoch);
  else
    hipLaunchKernelGGL((k_dw16<Tag, WI, false>), dim3((unsigned)dw_grid), dim3(512),
                       0, stream, (const uint16_t*)w.xbT, w.ld_xt, a.X, (uint16_t*)a.W, a.W_master,
                       a.M, a.active, a.n_active, a.labels_mapped, a.row_lse, w.inv_x, w.inv_w,
                       w.tgtc, (const uint16_t*)w.lbuf, w.ld_cos, w.gscale, w.ld_g, B, mg, sB, a.lr,
                       a.mu, w.dw_gate, n_gate, epoch);
  timing_stop(6, stream);
}

template <typename Tag>
void launch_bwd16_d(const StepArgs& a, const StepWs& w, const Margin& mg, float sB,
                    hipStream_t stream) {
  switch (a.d) {
    case 128: launch_bwd16<Tag, 1>(a, w, mg, sB, stream); break;
    case 256: launch_bwd16<Tag, 2>(a, w, mg, sB, stream); break;
    default: launch_bwd16<Tag, 4>(a, w, mg, sB, stream); break;
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
                       a.row_lse, w.inv_w, (const float*)w.lbuf, w.ld_cos, B, d, mg, w.dx_part);
    timing_stop(4, stream);
    timing_start(5, stream);
    hipLaunchKernelGGL(k_dx_final32, dim3((unsigned)ceil_div(B, 4)), dim3(256), 0, stream,
                       w.dx_part, (const float*)a.X, w.inv_x, B, d, sB, a.dX);
    timing_stop(5, stream);
    timing_start(6, stream);
    hipLaunchKernelGGL(k_dw32, dim3((unsigned)a.cap), dim3(256), 0, stream, (const float*)a.X,
                       (float*)a.W, a.W_master, a.M, a.active, a.n_active, a.labels_mapped,
                       a.row_lse, w.inv_x, w.inv_w, (const float*)w.lbuf, w.ld_cos, B, d, mg, sB,
                       a.lr, a.mu);
    timing_stop(6, stream);
  } else if (a.dtype == 1) {
    launch_bwd16_d<Bf16Tag>(a, w, mg, sB, stream);
  } else {
    launch_bwd16_d<F16Tag>(a, w, mg, sB, stream);
  }
  return hipGetLastError();
}

}  // namespace pfc
