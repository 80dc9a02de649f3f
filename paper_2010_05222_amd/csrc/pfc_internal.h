// Internal declarations shared by the HIP translation units of libpfc.
// Not part of the public ABI (include/pfc.h is).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace pfc {

// ----------------------------------------------------------------- sampler

enum SampleMode : uint32_t { kSelectNone = 0, kSelectKeys = 1, kSelectAll = 2 };

// Device-resident sampler state of one step (lives in the workspace).
struct SampleState {
  uint32_t n_pos;       // |P|: distinct owned labels
  uint32_t mode;        // SampleMode
  uint32_t top_digit;   // value of the top key bits holding the threshold
  int64_t n_neg;        // max(b - |P|, 0)
  int64_t k_rem;        // keys equal to `thresh` still to take (class order)
  uint64_t thresh;      // n_neg-th smallest non-positive key
};

// Compaction works on groups of kCompactClasses consecutive classes.
constexpr int kCompactThreads = 256;
constexpr int kCompactPer = 16;   // classes per thread
constexpr int kCompactClasses = kCompactPer * kCompactThreads;
constexpr int kTopBitsMax = 12;

struct SampleWs {
  uint32_t* bitmap;      // ceil(C/32) words: bit c set iff class c is positive
  uint32_t* hist;        // 2^kTopBitsMax bins
  SampleState* state;
  uint16_t* digits;      // C top-bit digits of the keys (only in kSelectKeys mode)
  uint64_t* cand_key;    // C: the full keys of compaction group g's non-positive classes
                         // in the threshold's top bucket at [g * kCompactClasses, + count)
  uint32_t* grp_sure;    // per compaction group: classes surely selected
  uint32_t* grp_tie;     // per compaction group: its candidate count, then (once the
                         // threshold is resolved) its non-positive keys == thresh
  uint32_t* grp_out;     // per compaction group: output offset
  uint32_t* grp_tie_off; // per compaction group: ties before the group
};

// ----------------------------------------------------------------- step

// Class tile of the forward contraction (one softmax-statistics pair per row and tile).
constexpr int kFwdClassTile = 128;
// Class group of the logit store: the forward keeps one base-2 reference per
// (row, group of 128 active classes).
constexpr int kLogitGroup = 128;

struct StepWs {
  float* inv_x;          // [B]      1/max(||x_n||, eps)
  void* xbT;             // [ld_xt / 32][d][32] x_hat (normalised rows) transposed in blocks of
                         // 32 rows, bf16, zero past B (the class-gradient operand)
  int64_t ld_xt;         // B rounded up to 32
  void* xblk;            // [d / 32][ld_xt][32] the raw 16-bit batch rows in 32-wide column
                         // blocks, zero past B (the forward's batch operand: one block is
                         // a contiguous run of whole rows)
  float* inv_w_max;      // [1] max_j 1/||W[S_j]|| (scale of the fp16 feature-gradient operand)
  float* inv_w;          // [ld_cos] 1/max(||W[S_j]||, eps), 0 past |S| within the last tile
  void* lbuf;            // [B x ld_cos] logit store.  16-bit paths: fp16 E = 2^(f log2 e - m)
                         // with m the row's reference for the class's 128-class group (E = 0
                         // at the target and past |S|); fp32 path: fp32 cosines
  int64_t ld_cos;        // row stride of lbuf: cap rounded up to 256
  float2* stats;         // [B x n_ctiles] per class tile: (max, sum 2^(f log2 e - max)), base 2
  int64_t n_ctiles;      // class tiles of the forward contraction
  float* tgt;            // [B] margined target logit
  float* tgtc;           // [B] unmargined target cosine
  float* gmax;           // [n_groups x ld_g] reference m of each (group, row)
  float* gscale;         // [n_groups x ld_g] 2^(m - lse log2 e), so p = E * gscale (0 past B)
  int64_t ld_g;          // B rounded up to 128
  int64_t n_groups;      // ld_cos / 128
  float* dx_part;        // [n_split x B x d] split-K partial sums of dX_hat
  int n_split;
  float* loss_part;      // [B] per-row loss terms
  int32_t* act_pad;      // [n_act_pad] the active row ids, padded with the last one
                         // (read a whole 32-class chunk at a time by the dX kernel)
  int64_t n_act_pad;     // cap rounded up to 128
  int32_t* dw_gate;      // [kDwGates] start gates of the class-gradient kernel: entry i holds
                         // the launch number once workgroup 2 i has finished its contraction
};

// Start gates of the class-gradient kernel (pairs of first-wave workgroups).
constexpr int kDwGates = 512;

// Layout of the whole workspace (offsets in bytes from its base).
struct WsLayout {
  size_t bytes;
  size_t sample_bytes;   // prefix used by the sampler
  size_t off_bitmap, off_hist, off_state, off_digits, off_cand_key;
  size_t off_grp_sure, off_grp_tie, off_grp_out, off_grp_tie_off;
  size_t off_inv_x, off_xb, off_xblk, off_wmax, off_inv_w, off_cos, off_stats, off_tgt, off_tgtc,
      off_gmax, off_gscale, off_dx, off_loss, off_act_pad, off_dw_gate;
  int64_t ld_cos, n_ctiles, n_groups, ld_xt, ld_g, n_lgroups, n_act_pad;
  int n_split;
  int top_bits;
};

// Activation budget b of a shard and the capacity max(b, min(B, C)) of S.
int64_t budget_of(double r, int64_t C);
int64_t cap_of(int64_t B, int64_t C, double r);

WsLayout ws_layout(int64_t B, int64_t d, int64_t C, int64_t cap, int compute);
SampleWs sample_ws(void* ws, const WsLayout& L);
StepWs step_ws(void* ws, const WsLayout& L);

hipError_t launch_sample(const int64_t* labels, int64_t B, int64_t C,
                         int64_t a, int64_t budget, uint64_t seed,
                         int top_bits, int64_t n_groups, const SampleWs& w,
                         int32_t* active, int64_t cap, int32_t* n_active,
                         int32_t* labels_mapped, hipStream_t stream);

struct StepArgs {
  const void* X;
  void* W;
  float* W_master;
  float* M;
  const int32_t* active;
  const int32_t* n_active;
  const int32_t* labels_mapped;
  const float* row_lse;
  float* loss;
  float* row_lse_out;
  float* dX;
  int64_t B, d, C, cap;
  int dtype;      // pfc_dtype of X, W and the compute
  float s, m;
  int margin;     // pfc_margin
  float tau;      // PFC* conflict threshold (forward); >= 1: no filtering
  float lr, mu;
};

hipError_t launch_prep(const StepArgs& a, const StepWs& w, hipStream_t stream);
hipError_t launch_forward(const StepArgs& a, const StepWs& w, hipStream_t stream);
hipError_t launch_backward(const StepArgs& a, const StepWs& w, hipStream_t stream);

// Measurement hook (pfc_timing_begin / pfc_timing_end): launchers bracket a
// kernel id's launches with these calls; both are no-ops unless armed.
void timing_start(int kernel, hipStream_t stream);
void timing_stop(int kernel, hipStream_t stream);

__host__ __device__ inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace pfc
