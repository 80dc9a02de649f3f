// Stages 4-5: the cosine-logit contraction cos = x_hat . w_hat over the
// active classes (Partial FC Sec. 3.3.3, Eq. mp_gemm: [B x d][d x |S|]), the
// target margin and the row-wise log-sum-exp cross-entropy over S
// (Sec. 3.1, Eq. sampled_probability; max / sum decomposition of Sec. 3.2.1).
//
// 16-bit path: one MFMA GEMM workgroup per 128 active classes (MFMA M, one
// 128-class group of the logit store) x 256 batch rows (MFMA N), d streamed
// in 32-wide chunks through a three-stage direct-to-LDS ring; two workgroups
// share a CU.  A stage holds 8 KB of gathered W rows (64-byte pieces of 128
// different rows) and 16 KB of batch rows (one contiguous run): of the two
// operands the gathered one moves fewer bytes, as its short pieces cost the
// L2 more per byte than the contiguous run.  Classes sit on the MFMA M axis
// so that each lane holds one batch row and 64 of its classes: the row
// max / sum-exp of the epilogue is mostly in-register.  The epilogue scales
// by 1/||x_n|| and 1/||w_j|| (the class-row norms are summed from the
// contraction's own class fragments), applies the margin at the target and
// the optional PFC* conflict filter, and writes each logit once, as its fp16
// softmax numerator E = 2^(f - m) relative to the maximum m of its row and
// 128-class group, the tile's (the tile is assembled in the idle LDS ring
// and stored as whole rows), with one (max, sum E) pair per (row, class
// tile).  A small
// kernel merges the pairs into lse_n and the loss.
#include "pfc_gemm.h"

namespace pfc {
namespace {

constexpr int kFwdBM = 128;       // classes per tile (MFMA M): one 128-class group
constexpr int kFwdBN = 256;       // batch rows per tile (MFMA N)
constexpr int kFwdKC = 32;        // slice of d per pipeline stage
constexpr int kFwdThreads = 256;  // 4 waves, one per 64 batch rows, 128 classes x 64 each
constexpr int kFwdStageA = kFwdBM * kFwdKC;  // uint16 elements per stage, class operand
constexpr int kFwdStageB = kFwdBN * kFwdKC;  // uint16 elements per stage, batch operand
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kEpsNormW = 1e-12f;  // ||w|| floor of the normalisation

// Three-stage LDS ring per operand (24 KB per stage; 72 KB in all, so two
// workgroups share a CU and one's epilogue overlaps the other's MFMA loop).
// One array per stage, so the compiler can keep the direct-to-LDS loads of
// later stages in flight while a stage is read.  Row r of a stage holds 32
// elements (64 B) as four 16-byte chunks; chunk c is stored at position
// c ^ ((r >> 2) & 3), so the sixteen lanes of a 16-byte LDS read that
// address sixteen consecutive rows hit distinct banks (64 banks).
__shared__ __attribute__((aligned(1024))) uint16_t fA0[kFwdStageA], fA1[kFwdStageA],
    fA2[kFwdStageA];
__shared__ __attribute__((aligned(1024))) uint16_t fB0[kFwdStageB], fB1[kFwdStageB],
    fB2[kFwdStageB];
__shared__ float2 fRed[1][kFwdBN];
__shared__ __attribute__((aligned(16))) float fIw[kFwdBM];
__shared__ int32_t fIds[kFwdBM];   // the tile's class-row ids
__shared__ float fNrm[2][kFwdBM];

template <int S>
__device__ __forceinline__ uint16_t* fwd_a() {
  if constexpr (S == 0) return fA0;
  else if constexpr (S == 1) return fA1;
  else return fA2;
}
template <int S>
__device__ __forceinline__ uint16_t* fwd_b() {
  if constexpr (S == 0) return fB0;
  else if constexpr (S == 1) return fB1;
  else return fB2;
}

// Row r (0..255) of the epilogue's cosine tile, rows of 128 elements: rows
// 0..95 in the class-operand stages (32 each), 96..255 in the batch-operand
// stages (64 each).  Every caller's r >> 5 is wave-uniform.
__device__ __forceinline__ uint16_t* fwd_tile_row(int r) {
  uint16_t* base;
  if (r < 32) base = fA0 + r * kFwdBM;
  else if (r < 64) base = fA1 + (r - 32) * kFwdBM;
  else if (r < 96) base = fA2 + (r - 64) * kFwdBM;
  else if (r < 160) base = fB0 + (r - 96) * kFwdBM;
  else if (r < 224) base = fB1 + (r - 160) * kFwdBM;
  else base = fB2 + (r - 224) * kFwdBM;
  return base;
}

// DMA of one stage: class operand rows 16 (2 wave + u) + lane / 4 (u < 2),
// batch operand rows 16 (4 wave + u) + lane / 4 (u < 4).
template <int S>
__device__ __forceinline__ void fwd_issue_a(const uint16_t* const ap[2], int k0, int wave) {
#pragma unroll
  for (int u = 0; u < 2; ++u) dma16(ap[u] + k0, fwd_a<S>() + (2 * wave + u) * 16 * kFwdKC);
}
template <int S>
__device__ __forceinline__ void fwd_issue_b(const uint16_t* const bp[4], int64_t kb, int wave) {
#pragma unroll
  for (int u = 0; u < 4; ++u) dma16(bp[u] + kb, fwd_b<S>() + (4 * wave + u) * 16 * kFwdKC);
}
template <int S>
__device__ __forceinline__ void fwd_issue(const uint16_t* const ap[2], const uint16_t* const bp[4],
                                          int k0, int64_t kb, int wave) {
  fwd_issue_a<S>(ap, k0, wave);
  fwd_issue_b<S>(bp, kb, wave);
}

// a0^2 + a1^2 + acc for a packed pair of 16-bit values (v_dot2_f32_*).
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ float sumsq2(uint32_t v, float acc, F16Tag) {
  const f16x2_t h = __builtin_bit_cast(f16x2_t, v);
  return __builtin_amdgcn_fdot2(h, h, acc, false);
}
__device__ __forceinline__ float sumsq2(uint32_t v, float acc, Bf16Tag) {
  const bf16x2_t h = __builtin_bit_cast(bf16x2_t, v);
  return __builtin_amdgcn_fdot2_f32_bf16(h, h, acc, false);
}

// Fragments of both 16-wide k-steps of a stage are requested first, then
// consumed: lane l reads row 32 q + l % 32 of its operand block, chunk
// 2 kk + l / 32 (stored at chunk ^ ((row >> 2) & 3)).  The class-operand
// fragments also feed the class-row norms: the wave with wn == kk adds the
// squares of its k-step's fragments to wss[mb] (class row 128 wm + 32 mb +
// l % 32, elements 8 (l / 32) .. + 7 of the k-step).
template <int S, typename Tag>
__device__ __forceinline__ void fwd_compute(f32x16_t (&acc)[4][2], int wm, int wn, int lane,
                                            float (&wss)[4]) {
  const int r32 = lane & 31;
  const int sw = (lane >> 2) & 3;
  const uint32_t arow = lds_addr(fwd_a<S>()) + (128 * wm + r32) * kFwdKC * 2;
  const uint32_t brow = lds_addr(fwd_b<S>()) + (64 * wn + r32) * kFwdKC * 2;
  u32x4_t af[2][4], bf[2][2];
  static_for<0, 2>([&](auto kq) {
    constexpr int kk = decltype(kq)::value;
    const uint32_t chunk = (uint32_t)(((2 * kk + (lane >> 5)) ^ sw) * 16);
    static_for<0, 4>([&](auto mm) {
      constexpr int mb = decltype(mm)::value;
      ds_read_128<32 * mb * kFwdKC * 2>(af[kk][mb], arow + chunk);
    });
    static_for<0, 2>([&](auto nn) {
      constexpr int nb = decltype(nn)::value;
      ds_read_128<32 * nb * kFwdKC * 2>(bf[kk][nb], brow + chunk);
    });
  });
  static_for<0, 2>([&](auto kq) {
    constexpr int kk = decltype(kq)::value;
    if constexpr (kk == 0)
      lgkm_wait<6>(af[0][0], af[0][1], af[0][2], af[0][3], bf[0][0], bf[0][1]);
    else
      lgkm_wait<0>(af[1][0], af[1][1], af[1][2], af[1][3], bf[1][0], bf[1][1]);
    if (wn == kk) {
#pragma unroll
      for (int mb = 0; mb < 4; ++mb) {
        wss[mb] = sumsq2(af[kk][mb].x, wss[mb], Tag{});
        wss[mb] = sumsq2(af[kk][mb].y, wss[mb], Tag{});
        wss[mb] = sumsq2(af[kk][mb].z, wss[mb], Tag{});
        wss[mb] = sumsq2(af[kk][mb].w, wss[mb], Tag{});
      }
    }
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
        acc[mb][nb] = mfma_32x32x16(make_uint4(af[kk][mb].x, af[kk][mb].y, af[kk][mb].z, af[kk][mb].w),
                                    make_uint4(bf[kk][nb].x, bf[kk][nb].y, bf[kk][nb].z, bf[kk][nb].w),
                                    acc[mb][nb], Tag{});
  });
}

// The 8-byte piece (classes 32 mb + 8 g + 4 half .. + 3) of a tile row: its
// 16-byte block b = bbase + 4 mb + g sits at position b ^ bsw (bbase a
// multiple of 16, bsw < 16), split here into the mb and g parts of the XOR.
__device__ __forceinline__ uint16_t* tile_block(uint16_t* trow, int bbase, int bsw, int mb, int g,
                                                int half) {
  return trow + 8 * bbase + 32 * (mb ^ (bsw >> 2)) + 8 * (g ^ (bsw & 3)) + 4 * half;
}

// Epilogue of one lane for one 32-row block (nb): the lane's row n and its
// 64 classes j = jb + 32 mb + 8 g + e (jb = first class of the lane's
// pattern, e < 4); with the partner lane (half ^ 1) they are the row's 128
// classes of one group.  Computes the base-2 logits f2 = s c log2 e (-inf at
// the target, whose margined logit is merged separately, past |S|, and with
// FILT at a negative whose cosine exceeds tau: the PFC* conflict filter,
// Sec. 3.3.4, Eq. noise_filtering, so E = 0 there and the backward's
// coefficient too), the
// group maximum m (the target's margined logit included), and writes
// E = 2^(f2 - m) as fp16 to the LDS tile row trow (16-byte block b of the row
// at position b ^ bsw).  Returns the pair's (m, sum of E and the target term).
template <bool CHECK_J, bool CHECK_T, bool FILT>
__device__ __forceinline__ void fwd_epilogue_rows(f32x16_t (&acc)[4][2], int nb, float ix,
                                                  const float* iwp, int K, int64_t jb, int tpos,
                                                  const Margin& mg, float tau, uint16_t* trow,
                                                  int bbase, int bsw, int half, float* mx_out,
                                                  float* sm_out, float* tgt_out, float* tgtc_out) {
  const float s2 = mg.s * kLog2e;
  float mx = -INFINITY;
  float ct = 0.0f;
#pragma unroll
  for (int mb = 0; mb < 4; ++mb) {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int o = 32 * mb + 8 * g;
      const float4 iw4 = *reinterpret_cast<const float4*>(iwp + o);
      const float iwv[4] = {iw4.x, iw4.y, iw4.z, iw4.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float c = acc[mb][nb][4 * g + e] * ix * iwv[e];
        float f2 = c * s2;
        if (CHECK_J && jb + o + e >= K) f2 = -INFINITY;
        if (FILT && c > tau) f2 = -INFINITY;   // PFC* drops the negative (not the target: below)
        if (CHECK_T && tpos == o + e) {
          ct = c;
          f2 = -INFINITY;   // the margined target logit is merged below
        }
        acc[mb][nb][4 * g + e] = f2;
        mx = fmaxf(mx, f2);
      }
    }
  }
  float ft2 = -INFINITY;
  if (CHECK_T && tgt_out) {
    const float ft = target_logit(mg, ct);
    *tgt_out = ft;
    *tgtc_out = ct;
    ft2 = ft * kLog2e;
    mx = fmaxf(mx, ft2);
  }
  mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
  // A group with no live logit keeps reference 0 (all its E are 0).
  const float mref = mx == -INFINITY ? 0.0f : mx;
  float sm = 0.0f;
#pragma unroll
  for (int mb = 0; mb < 4; ++mb) {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      float ev[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        ev[e] = __builtin_amdgcn_exp2f(acc[mb][nb][4 * g + e] - mref);
        sm += ev[e];
      }
      uint2 packed;
      packed.x = pack_f16x2(ev[0], ev[1]);
      packed.y = pack_f16x2(ev[2], ev[3]);
      *reinterpret_cast<uint2*>(tile_block(trow, bbase, bsw, mb, g, half)) = packed;
    }
  }
  if (CHECK_T && tgt_out) sm += __builtin_amdgcn_exp2f(ft2 - mref);
  sm += __shfl_xor(sm, 32, 64);
  *mx_out = mx;
  *sm_out = sm;
}

// The common case of fwd_epilogue_rows: every class of the lane's pattern
// exists, none is a row's target, no filter.  With q = s log2 e / ||x|| >= 0
// the group maximum is q max_j u_j over u_j = acc_j / ||w_j||, and
// E_j = 2^(u_j q - m) takes one fused multiply-add.
__device__ __forceinline__ void fwd_epilogue_rows_plain(f32x16_t (&acc)[4][2], int nb, float q,
                                                        const float* iwp, uint16_t* trow,
                                                        int bbase, int bsw, int half,
                                                        float* mx_out, float* sm_out) {
  float mu = -INFINITY;
#pragma unroll
  for (int mb = 0; mb < 4; ++mb) {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const float4 iw4 = *reinterpret_cast<const float4*>(iwp + 32 * mb + 8 * g);
      const float iwv[4] = {iw4.x, iw4.y, iw4.z, iw4.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float u = acc[mb][nb][4 * g + e] * iwv[e];
        acc[mb][nb][4 * g + e] = u;
        mu = fmaxf(mu, u);
      }
    }
  }
  mu = fmaxf(mu, __shfl_xor(mu, 32, 64));
  const float mx = mu * q;
  float sm = 0.0f;
#pragma unroll
  for (int mb = 0; mb < 4; ++mb) {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      float ev[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        ev[e] = __builtin_amdgcn_exp2f(fmaf(acc[mb][nb][4 * g + e], q, -mx));
        sm += ev[e];
      }
      uint2 packed;
      packed.x = pack_f16x2(ev[0], ev[1]);
      packed.y = pack_f16x2(ev[2], ev[3]);
      *reinterpret_cast<uint2*>(tile_block(trow, bbase, bsw, mb, g, half)) = packed;
    }
  }
  sm += __shfl_xor(sm, 32, 64);
  *mx_out = mx;
  *sm_out = sm;
}

// Tile: 128 active classes x 256 batch rows, the whole of d (= 32 * NK).
// Epilogue, per (row, class): c = acc / (||x|| ||w||) and the base-2 logit
// s c log2 e (the margined logit at the target, which also goes to tgt[n],
// its cosine to tgtc[n]); per row the tile's maximum m (the row's reference
// for this 128-class group), written to gmax, and E = 2^(f - m) in fp16, and
// the pair (m, sum E), merged by k_lse16.  The batch operand comes from the
// column-blocked copy of X (block k = [ld_xb][32]), so a stage's 256 batch
// rows are one contiguous 16 KB run.
template <typename Tag, int NK, bool FILT>
__global__ void __launch_bounds__(kFwdThreads, 2) k_fwd16(
    const uint16_t* __restrict__ Xb, int64_t ld_xb, const uint16_t* __restrict__ W,
    const int32_t* __restrict__ act_pad, const int32_t* __restrict__ n_active_p,
    const int32_t* __restrict__ yhat, const float* __restrict__ inv_x,
    float* __restrict__ inv_w, float* __restrict__ inv_w_max, int B, int64_t ld_cos,
    int64_t n_ctiles, int n_rt, int64_t n_tiles, int64_t per_xcd, Margin mg, float tau,
    uint16_t* __restrict__ lbuf, float2* __restrict__ stats, float* __restrict__ tgt,
    float* __restrict__ tgtc, float* __restrict__ gmax, int64_t ld_g) {
  constexpr int D = NK * kFwdKC;
  // All batch-row tiles of a class tile run on one XCD: the gathered W rows
  // come from HBM once and are re-read from that XCD's L2.
  const int64_t t = (int64_t)(blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  if (t >= n_tiles) return;
  const int64_t ct = t / n_rt;
  const int rt = (int)(t % n_rt);
  const int64_t j0 = ct * kFwdBM;
  const int n0 = rt * kFwdBN;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = 0, wn = wave;   // every wave: all 128 classes, its 64 batch rows
  const int half = lane >> 5, l32 = lane & 31;

  // Per-lane source rows of the DMA segments.  The class rows come from the
  // padded id list (entries past |S| repeat the last active id, so their
  // results are valid numbers, masked in the epilogue), which needs no wait
  // for |S|: the ids of the wave's 32 class rows go straight to LDS first,
  // then the batch rows of the first two stages are requested (rows past the
  // end clamped to a valid row), then the ids are read back and the class
  // rows requested.
  const int cidx = (lane & 3) ^ ((lane >> 4) & 3);
  if (lane < 32)
    __builtin_amdgcn_global_load_lds(act_pad + j0 + 32 * wave + lane, (lds_void_t)(fIds + 32 * wave),
                                     4, 0, 0);
  const uint16_t* ap[2];
  const uint16_t* bp[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int row = 16 * (4 * wave + u) + (lane >> 2);
    const int nr = n0 + row < B ? n0 + row : B - 1;
    bp[u] = Xb + (int64_t)nr * kFwdKC + 8 * cidx;
  }
  fwd_issue_b<0>(bp, 0, wave);
  if constexpr (NK > 1) fwd_issue_b<1>(bp, (int64_t)kFwdKC * ld_xb, wave);
  const int K = *n_active_p;
  if (j0 >= K) {   // no active class in the tile: drain the wave's loads into LDS, leave
    wait_vmcnt<0>();
    return;
  }
  wait_vmcnt<(NK > 1 ? 8 : 4)>();   // the id load, older than the batch-row loads, has landed
  uint32_t ids[2];
  ds_read_32<0>(ids[0], lds_addr(fIds + 32 * wave + (lane >> 2)));
  ds_read_32<64>(ids[1], lds_addr(fIds + 32 * wave + (lane >> 2)));
  lgkm_wait<0>(ids[0], ids[1]);
#pragma unroll
  for (int u = 0; u < 2; ++u) ap[u] = W + (int64_t)ids[u] * D + 8 * cidx;

  f32x16_t acc[4][2];
#pragma unroll
  for (int mb = 0; mb < 4; ++mb)
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mb][nb][r] = 0.0f;

  // Epilogue inputs, requested before the main loop and not used before the
  // epilogue (so nothing waits for them here): each lane's row data, from a
  // valid row for rows past the batch (whose results are never stored).
  float ixr[2];
  int yraw[2];
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const int n = n0 + 64 * wn + 32 * nb + l32;
    const int nc = n < B ? n : B - 1;
    ixr[nb] = inv_x[nc];
    yraw[nb] = yhat[nc];
  }

  float wss[4] = {0.0f, 0.0f, 0.0f, 0.0f};  // partial ||w||^2 of the lane's class rows
  constexpr int kPerStage = 6;  // DMAs per thread per stage (2 class-row, 4 batch-row)
  fwd_issue_a<0>(ap, 0, wave);
  if constexpr (NK > 1) fwd_issue_a<1>(ap, kFwdKC, wave);
  static_for<0, NK>([&](auto cc) {
    constexpr int c = decltype(cc)::value;
    constexpr int ahead = (NK - 1 - c) < 1 ? (NK - 1 - c) : 1;
    // Loads still in flight that belong to later chunks: stage 1's class rows
    // (issued last) at chunk 0, the next stage's six loads after that.
    constexpr int later = c == 0 ? 2 * ahead : kPerStage * ahead;
    // This wave's loads of chunk c have landed; after the barrier everyone's
    // have, and every wave is done with chunk c - 1, whose stage is refilled.
    wait_vmcnt<later>();
    stage_barrier();
    if constexpr (c + 2 < NK) fwd_issue<(c + 2) % 3>(ap, bp, (c + 2) * kFwdKC, (int64_t)(c + 2) * kFwdKC * ld_xb, wave);
    fwd_compute<c % 3, Tag>(acc, wm, wn, lane, wss);
  });

  // Inverse norms of the tile's class rows (stage 3 of the step, computed from
  // the rows this kernel streams anyway): the four partial sums of a row
  // (lane halves, and the two waves wn = 0, 1) meet in LDS; the norms stay in
  // LDS for the epilogue, and the first batch-row tile of each class tile
  // also publishes them, and their running maximum, for the backward kernels.
  {
#pragma unroll
    for (int mb = 0; mb < 4; ++mb) {
      const float s = wss[mb] + __shfl_xor(wss[mb], 32, 64);
      if (half == 0 && wn < 2) fNrm[wn][128 * wm + 32 * mb + l32] = s;
    }
    wait_lgkm0();
    stage_barrier();
    if (tid < kFwdBM) {   // waves 0 and 1: one class each
      const float inv = 1.0f / fmaxf(sqrtf(fNrm[0][tid] + fNrm[1][tid]), kEpsNormW);
      fIw[tid] = inv;
      if (rt == 0) {
        const bool jok = j0 + tid < (int64_t)K;
        inv_w[j0 + tid] = jok ? inv : 0.0f;
        const float m = wave_max(jok ? inv : 0.0f);
        if (lane == 0) atomicMax(reinterpret_cast<int*>(inv_w_max), __float_as_int(m));
      }
    }
  }

  // ---- epilogue.  The fp16 128-class x 256-row tile of E values is
  // assembled in the (now idle) LDS ring (rows of 256 B, 16-byte block b of
  // row r at position b ^ (r & 15): conflict-free writes from the MFMA layout
  // and reads along rows); each wave writes out its rows, 32 at a time, in
  // whole rows as soon as they are done.
  wait_lgkm0();
  stage_barrier();  // all fragment reads of the ring are done
  const int64_t jlo = j0 + 128 * wm;
  const bool full = jlo + 128 <= (int64_t)K;   // wave-uniform: no class past |S|
  const float* iwp = fIw + 128 * wm + 4 * half;
  // Rows of the lane, and whether the lane's class pattern holds a row's target.
  int tpos[2];
  bool has_t[2];
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const int n = n0 + 64 * wn + 32 * nb + l32;
    const int yh = n < B && yraw[nb] < K ? yraw[nb] : -1;   // past |S|: unowned
    tpos[nb] = yh - (int)(jlo + 4 * half);   // target's offset in this lane's class pattern
    has_t[nb] = yh >= jlo && yh < jlo + 128 && ((tpos[nb] & 4) == 0);
  }
  auto finish = [&](int nb, float mx, float sm) __attribute__((always_inline)) {
    const int nl = 64 * wn + 32 * nb + l32;
    const int n = n0 + nl;
    if (half == 0) {
      fRed[wm][nl] = make_float2(mx, sm);
      // reference of the row's 128-class group, the tile's
      if (n < B) gmax[ct * ld_g + n] = mx == -INFINITY ? 0.0f : mx;
    }
  };
  // Rows 64 wave + 32 nb .. + 31 of the tile, which this wave alone wrote:
  // read back along rows (the wave's LDS accesses complete in order) and
  // stored as whole 256-byte rows, four rows per store, while the wave goes
  // on with its next row block.  The stores are non-temporal: the logit
  // store is read back only by later kernels, after gigabytes of other
  // traffic, so it should not take L2 space from the operands this kernel
  // re-reads.
  auto store_rows = [&](int nb) __attribute__((always_inline)) {
    wait_lgkm0();
    asm volatile("" ::: "memory");   // the tile writes above are not moved below the reads
    const int b = lane & 15;
    u32x4_t v[8];
    static_for<0, 8>([&](auto ii) {
      constexpr int i = decltype(ii)::value;
      const int r = 64 * wave + 32 * nb + 4 * i + (lane >> 4);
      ds_read_128<0>(v[i], lds_addr(fwd_tile_row(r) + 8 * (b ^ (r & 15))));
    });
    lgkm_wait<0>(v);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int n = n0 + 64 * wave + 32 * nb + 4 * i + (lane >> 4);
      if (n < B)
        __builtin_nontemporal_store(
            v[i], reinterpret_cast<u32x4_t*>(lbuf + (int64_t)n * ld_cos + j0 + 8 * b));
    }
  };
  // Two separate paths over both row blocks, so that the masking work of
  // the checked one (classes past |S|, targets) stays out of the common one.
  if (full && !__any(has_t[0] || has_t[1])) {
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      const int nl = 64 * wn + 32 * nb + l32;
      float mx, sm;
      if constexpr (FILT)
        fwd_epilogue_rows<false, false, true>(acc, nb, ixr[nb], iwp, K, jlo + 4 * half, tpos[nb],
                                              mg, tau, fwd_tile_row(nl), 16 * wm, nl & 15, half,
                                              &mx, &sm, nullptr, nullptr);
      else
        fwd_epilogue_rows_plain(acc, nb, ixr[nb] * (mg.s * kLog2e), iwp, fwd_tile_row(nl),
                                16 * wm, nl & 15, half, &mx, &sm);
      finish(nb, mx, sm);
      store_rows(nb);
    }
  } else {
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      const int nl = 64 * wn + 32 * nb + l32;
      const int n = n0 + nl;
      float mx, sm;
      fwd_epilogue_rows<true, true, FILT>(acc, nb, ixr[nb], iwp, K, jlo + 4 * half, tpos[nb], mg,
                                          tau, fwd_tile_row(nl), 16 * wm, nl & 15, half, &mx,
                                          &sm, has_t[nb] ? tgt + n : nullptr,
                                          has_t[nb] ? tgtc + n : nullptr);
      finish(nb, mx, sm);
      store_rows(nb);
    }
  }
  // Row r of the pairs was written by lane r % 32 of wave r / 64, this
  // thread's own wave: no barrier.
  for (int r = tid; r < kFwdBN; r += kFwdThreads) {
    const int n = n0 + r;
    if (n < B) stats[(int64_t)n * n_ctiles + ct] = fRed[0][r];
  }
}

// Merge the per-tile (max, sum) pairs of a row: lse_n, and the row's loss
// term.  One workgroup per row, one pass over the row's pairs: each thread
// merges its pairs in tile order (base 2), the waves' pairs meet through
// lane moves and LDS in a fixed order.
__global__ void __launch_bounds__(256) k_lse16(const float2* __restrict__ stats, int64_t n_ctiles,
                                               const int32_t* __restrict__ n_active_p,
                                               const int32_t* __restrict__ yhat,
                                               const float* __restrict__ tgt, int B,
                                               float* __restrict__ row_lse,
                                               float* __restrict__ loss_part) {
  __shared__ float2 red[4];
  const int n = blockIdx.x;
  const int t = threadIdx.x, lane = t & 63;
  const int64_t nct = ceil_div((int64_t)*n_active_p, (int64_t)kFwdBM);
  const float2* row = stats + (int64_t)n * n_ctiles;
  float2 acc = make_float2(-INFINITY, 0.0f);
  // Eight loads in flight per thread, merged in tile order.
  for (int64_t c0 = t; c0 < nct; c0 += 256 * 8) {
    float2 v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int64_t c = c0 + 256 * k;
      v[k] = c < nct ? row[c] : make_float2(-INFINITY, 0.0f);
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) acc = lse_merge2(acc, v[k]);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    float2 o;
    o.x = __shfl_xor(acc.x, off, 64);
    o.y = __shfl_xor(acc.y, off, 64);
    acc = lse_merge2(acc, o);
  }
  if (lane == 0) red[t >> 6] = acc;
  __syncthreads();
  if (t == 0) {
    acc = lse_merge2(lse_merge2(red[0], red[1]), lse_merge2(red[2], red[3]));
    const float lse = acc.x == -INFINITY ? -INFINITY
                                         : (acc.x + log2f(acc.y)) * 0.6931471805599453f;
    row_lse[n] = lse;
    const int yh = yhat[n];
    loss_part[n] = yh >= 0 && yh < *n_active_p ? lse - tgt[n] : 0.0f;   // past |S|: unowned
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
    loss_part[n] = yh >= 0 && yh < K ? lse - ft : 0.0f;
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

template <typename Tag, int NK>
void launch_fwd16_nk(unsigned grid, hipStream_t stream, const StepArgs& a, const StepWs& w, int B,
                     int n_rt, int64_t n_tiles, int64_t per_xcd, const Margin& mg) {
  if (a.tau < 1.0f)
    hipLaunchKernelGGL((k_fwd16<Tag, NK, true>), dim3(grid), dim3(kFwdThreads), 0, stream,
                       (const uint16_t*)w.xblk, w.ld_xt, (const uint16_t*)a.W, w.act_pad, a.n_active,
                       a.labels_mapped, w.inv_x, w.inv_w, w.inv_w_max, B, w.ld_cos, w.n_ctiles,
                       n_rt, n_tiles, per_xcd, mg, a.tau, (uint16_t*)w.lbuf, w.stats, w.tgt,
                       w.tgtc, w.gmax, w.ld_g);
  else
    hipLaunchKernelGGL((k_fwd16<Tag, NK, false>), dim3(grid), dim3(kFwdThreads), 0, stream,
                       (const uint16_t*)w.xblk, w.ld_xt, (const uint16_t*)a.W, w.act_pad, a.n_active,
                       a.labels_mapped, w.inv_x, w.inv_w, w.inv_w_max, B, w.ld_cos, w.n_ctiles,
                       n_rt, n_tiles, per_xcd, mg, a.tau, (uint16_t*)w.lbuf, w.stats, w.tgt,
                       w.tgtc, w.gmax, w.ld_g);
}

template <typename Tag>
void launch_fwd16(int d, unsigned grid, hipStream_t stream, const StepArgs& a, const StepWs& w,
                  int B, int n_rt, int64_t n_tiles, int64_t per_xcd, const Margin& mg) {
  switch (d) {
    case 128: launch_fwd16_nk<Tag, 4>(grid, stream, a, w, B, n_rt, n_tiles, per_xcd, mg); break;
    case 256: launch_fwd16_nk<Tag, 8>(grid, stream, a, w, B, n_rt, n_tiles, per_xcd, mg); break;
    default: launch_fwd16_nk<Tag, 16>(grid, stream, a, w, B, n_rt, n_tiles, per_xcd, mg); break;
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
    const int n_rt = (int)ceil_div(B, kFwdBN);
    const int64_t n_tiles = w.n_ctiles * n_rt;
    const int64_t per_xcd = ceil_div(n_tiles, 8);
    const unsigned grid = (unsigned)(8 * per_xcd);
    timing_start(2, stream);
    if (a.dtype == 1)
      launch_fwd16<Bf16Tag>(d, grid, stream, a, w, B, n_rt, n_tiles, per_xcd, mg);
    else
      launch_fwd16<F16Tag>(d, grid, stream, a, w, B, n_rt, n_tiles, per_xcd, mg);
    timing_stop(2, stream);
    timing_start(3, stream);
    hipLaunchKernelGGL(k_lse16, dim3((unsigned)B), dim3(256), 0, stream, w.stats,
                       w.n_ctiles, a.n_active, a.labels_mapped, w.tgt, B, a.row_lse_out,
                       w.loss_part);
  }
  hipLaunchKernelGGL(k_loss, dim3(1), dim3(1024), 0, stream, w.loss_part, B, a.loss);
  timing_stop(3, stream);
  return hipGetLastError();
}

}  // namespace pfc
