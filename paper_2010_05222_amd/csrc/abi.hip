// extern "C" entry points of libpfc: argument checks, workspace layout and
// dispatch to the kernel launchers.  Declarations and documentation of each
// entry point are in include/pfc.h.
#include <math.h>

#include "pfc.h"
#include "pfc_internal.h"

namespace pfc {
namespace {

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

int64_t round_up(int64_t x, int64_t m) { return ceil_div(x, m) * m; }

int ceil_log2(int64_t x) {
  int b = 0;
  while (((int64_t)1 << b) < x) ++b;
  return b;
}

bool dtype_ok(int t) { return t == PFC_F32 || t == PFC_BF16 || t == PFC_F16; }

bool finite_pos(double v) { return isfinite(v) && v > 0.0; }

// Shape checks shared by every step call.  Returns PFC_OK or the error code.
int check_shape(int64_t B, int64_t d, int64_t C, int compute) {
  if (B < 1 || B > PFC_MAX_BATCH || C < 1 || C > PFC_MAX_CLASSES) return PFC_ERR_INVALID_ARG;
  if (d < 8 || d > 1024 || d % 8 != 0) return PFC_ERR_INVALID_ARG;
  if (!dtype_ok(compute)) return PFC_ERR_UNSUPPORTED;
  if (compute == PFC_F32) {
    if (B > 4096) return PFC_ERR_UNSUPPORTED;      // fp32 path is for parity-scale problems
  } else if (d != 128 && d != 256 && d != 512) {
    return PFC_ERR_UNSUPPORTED;                    // 16-bit MFMA kernels: d in {128, 256, 512}
  }
  return PFC_OK;
}

int check_hparams(float s, float m, int margin) {
  if (!finite_pos(s) || !isfinite(m) || m < 0.0f) return PFC_ERR_INVALID_ARG;
  if (margin != PFC_COSFACE && margin != PFC_ARCFACE) return PFC_ERR_INVALID_ARG;
  if (margin == PFC_ARCFACE && m >= 3.14159265358979f) return PFC_ERR_INVALID_ARG;
  return PFC_OK;
}

}  // namespace

// Activation budget of a shard (Eq. local_sampling): r*C when it is an
// integer within 1e-9 relative, else ceil(r*C).
int64_t budget_of(double r, int64_t C) {
  const double t = r * (double)C;
  const double rt = nearbyint(t);
  if (fabs(t - rt) <= 1e-9 * fmax(1.0, t)) return (int64_t)rt;
  return (int64_t)ceil(t);
}

int64_t cap_of(int64_t B, int64_t C, double r) {
  const int64_t b = budget_of(r, C);
  const int64_t p = B < C ? B : C;
  return b > p ? b : p;
}

WsLayout ws_layout(int64_t B, int64_t d, int64_t C, int64_t cap, int compute) {
  WsLayout L{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align256(off + bytes);
    return o;
  };
  L.n_groups = ceil_div(C, kCompactClasses);
  L.top_bits = ceil_log2(C) - 10;
  L.top_bits = L.top_bits < 1 ? 1 : (L.top_bits > kTopBitsMax ? kTopBitsMax : L.top_bits);
  L.off_bitmap = take((size_t)ceil_div(C, 32) * 4);
  L.off_hist = take((size_t)(1 << kTopBitsMax) * 4);
  L.off_state = take(sizeof(SampleState));
  L.off_digits = take((size_t)round_up(C, kCompactPer) * 2);   // read 16 at a time
  L.off_cand_key = take((size_t)C * 8);
  L.off_grp_sure = take((size_t)L.n_groups * 4);
  L.off_grp_tie = take((size_t)L.n_groups * 4);
  L.off_grp_out = take((size_t)L.n_groups * 4);
  L.off_grp_tie_off = take((size_t)L.n_groups * 4);
  L.sample_bytes = off;

  L.ld_cos = round_up(cap, 256);
  L.n_ctiles = ceil_div(cap, kFwdClassTile);
  L.ld_xt = round_up(B, 32);
  L.ld_g = round_up(B, 128);
  L.n_lgroups = L.ld_cos / kLogitGroup;
  if (compute == PFC_F32) {
    L.n_split = 1;
  } else {
    // Split-K of the feature-gradient contraction: ~256 workgroups of
    // 128 batch rows, one per CU.
    const int64_t n_rt = ceil_div(B, 128);
    const int64_t chunks = ceil_div(cap, 32);
    int64_t ns = ceil_div(256, n_rt);
    ns = ns > chunks ? chunks : ns;
    L.n_split = (int)(ns < 1 ? 1 : ns);
  }
  const size_t cos_elt = compute == PFC_F32 ? 4 : 2;
  L.off_inv_x = take((size_t)B * 4);
  L.off_xb = take(compute == PFC_F32 ? 0 : (size_t)L.ld_xt * d * 2);
  L.off_xblk = take(compute == PFC_F32 ? 0 : (size_t)L.ld_xt * d * 2);
  L.off_wmax = take(4);
  L.off_inv_w = take((size_t)L.ld_cos * 4);
  L.off_cos = take((size_t)B * L.ld_cos * cos_elt);
  L.off_stats = take((size_t)B * L.n_ctiles * 8);
  L.off_tgt = take((size_t)B * 4);
  L.off_dx = take((size_t)L.n_split * B * d * 4);
  L.off_loss = take((size_t)B * 4);
  L.off_tgtc = take((size_t)B * 4);
  L.off_gmax = take(compute == PFC_F32 ? 0 : (size_t)L.n_lgroups * L.ld_g * 4);
  L.off_gscale = take(compute == PFC_F32 ? 0 : (size_t)L.n_lgroups * L.ld_g * 4);
  L.n_act_pad = round_up(cap, 128);   // whole forward class tiles (and dX chunks)
  L.off_act_pad = take(compute == PFC_F32 ? 0 : (size_t)L.n_act_pad * 4);
  L.off_dw_gate = take(compute == PFC_F32 ? 0 : (size_t)kDwGates * 4);
  L.bytes = off;
  return L;
}

SampleWs sample_ws(void* ws, const WsLayout& L) {
  char* b = (char*)ws;
  SampleWs w;
  w.bitmap = (uint32_t*)(b + L.off_bitmap);
  w.hist = (uint32_t*)(b + L.off_hist);
  w.state = (SampleState*)(b + L.off_state);
  w.digits = (uint16_t*)(b + L.off_digits);
  w.cand_key = (uint64_t*)(b + L.off_cand_key);
  w.grp_sure = (uint32_t*)(b + L.off_grp_sure);
  w.grp_tie = (uint32_t*)(b + L.off_grp_tie);
  w.grp_out = (uint32_t*)(b + L.off_grp_out);
  w.grp_tie_off = (uint32_t*)(b + L.off_grp_tie_off);
  return w;
}

StepWs step_ws(void* ws, const WsLayout& L) {
  char* b = (char*)ws;
  StepWs w;
  w.inv_x = (float*)(b + L.off_inv_x);
  w.xbT = b + L.off_xb;
  w.xblk = b + L.off_xblk;
  w.ld_xt = L.ld_xt;
  w.inv_w_max = (float*)(b + L.off_wmax);
  w.inv_w = (float*)(b + L.off_inv_w);
  w.lbuf = b + L.off_cos;
  w.ld_cos = L.ld_cos;
  w.stats = (float2*)(b + L.off_stats);
  w.n_ctiles = L.n_ctiles;
  w.tgt = (float*)(b + L.off_tgt);
  w.dx_part = (float*)(b + L.off_dx);
  w.n_split = L.n_split;
  w.loss_part = (float*)(b + L.off_loss);
  w.tgtc = (float*)(b + L.off_tgtc);
  w.gmax = (float*)(b + L.off_gmax);
  w.gscale = (float*)(b + L.off_gscale);
  w.ld_g = L.ld_g;
  w.n_groups = L.n_lgroups;
  w.act_pad = (int32_t*)(b + L.off_act_pad);
  w.n_act_pad = L.n_act_pad;
  w.dw_gate = (int32_t*)(b + L.off_dw_gate);
  return w;
}

}  // namespace pfc

using namespace pfc;

extern "C" {

int pfc_workspace_bytes(int64_t B, int64_t d, int64_t C, double r, int compute_dtype,
                        size_t* bytes, int64_t* active_cap) {
  if (!bytes || !active_cap) return PFC_ERR_INVALID_ARG;
  if (!(isfinite(r) && r > 0.0 && r <= 1.0)) return PFC_ERR_INVALID_ARG;
  const int st = check_shape(B, d, C, compute_dtype);
  if (st != PFC_OK) return st;
  const int64_t cap = cap_of(B, C, r);
  *active_cap = cap;
  *bytes = ws_layout(B, d, C, cap, compute_dtype).bytes;
  return PFC_OK;
}

int pfc_sample(const int64_t* labels, int64_t B, int64_t C, int64_t class_offset, double r,
               uint64_t seed, int32_t* active, int64_t active_cap, int32_t* n_active,
               int32_t* labels_mapped, void* ws, size_t ws_bytes, void* stream) {
  if (!labels || !active || !n_active || !labels_mapped) return PFC_ERR_INVALID_ARG;
  if (B < 1 || B > PFC_MAX_BATCH || C < 1 || C > PFC_MAX_CLASSES) return PFC_ERR_INVALID_ARG;
  if (class_offset < 0 || class_offset > ((int64_t)1 << 62) - C) return PFC_ERR_INVALID_ARG;
  if (!(isfinite(r) && r > 0.0 && r <= 1.0)) return PFC_ERR_INVALID_ARG;
  if (active_cap < cap_of(B, C, r)) return PFC_ERR_CAPACITY;
  const WsLayout L = ws_layout(B, 8, C, active_cap, PFC_F32);
  if (!ws || ((uintptr_t)ws & 255) != 0) return PFC_ERR_WORKSPACE;
  if (ws_bytes < L.sample_bytes) return PFC_ERR_WORKSPACE;
  (void)hipGetLastError();
  const hipError_t e = launch_sample(labels, B, C, class_offset, budget_of(r, C), seed, L.top_bits,
                                     L.n_groups, sample_ws(ws, L), active, active_cap, n_active,
                                     labels_mapped, (hipStream_t)stream);
  return e == hipSuccess ? PFC_OK : PFC_ERR_HIP;
}

int pfc_forward_loss(const void* X, int x_dtype, int64_t B, int64_t d, const void* W,
                     int w_dtype, int64_t C, const int32_t* active, const int32_t* n_active,
                     int64_t active_cap, const int32_t* labels_mapped, int compute_dtype,
                     float s, float m, int margin, float tau, float* loss, float* row_lse,
                     void* ws, size_t ws_bytes, void* stream) {
  if (!X || !W || !active || !n_active || !labels_mapped || !loss || !row_lse)
    return PFC_ERR_INVALID_ARG;
  int st = check_shape(B, d, C, compute_dtype);
  if (st != PFC_OK) return st;
  if (x_dtype != compute_dtype || w_dtype != compute_dtype) return PFC_ERR_UNSUPPORTED;
  if (active_cap < 1 || active_cap > C) return PFC_ERR_CAPACITY;
  st = check_hparams(s, m, margin);
  if (st != PFC_OK) return st;
  if (tau != tau) return PFC_ERR_INVALID_ARG;   // NaN
  const WsLayout L = ws_layout(B, d, C, active_cap, compute_dtype);
  if (!ws || ((uintptr_t)ws & 255) != 0 || ws_bytes < L.bytes) return PFC_ERR_WORKSPACE;
  StepArgs a{};
  a.X = X;
  a.W = const_cast<void*>(W);
  a.active = active;
  a.n_active = n_active;
  a.labels_mapped = labels_mapped;
  a.loss = loss;
  a.row_lse_out = row_lse;
  a.B = B;
  a.d = d;
  a.C = C;
  a.cap = active_cap;
  a.dtype = compute_dtype;
  a.s = s;
  a.m = m;
  a.margin = margin;
  a.tau = tau;
  (void)hipGetLastError();
  const hipError_t e = launch_forward(a, step_ws(ws, L), (hipStream_t)stream);
  return e == hipSuccess ? PFC_OK : PFC_ERR_HIP;
}

int pfc_backward_update(const void* X, int x_dtype, int64_t B, int64_t d, void* W, int w_dtype,
                        float* W_master, float* momentum, int64_t C, const int32_t* active,
                        const int32_t* n_active, int64_t active_cap,
                        const int32_t* labels_mapped, int compute_dtype, float s, float m,
                        int margin, const float* row_lse, float lr, float mu, float* dX,
                        void* ws, size_t ws_bytes, void* stream) {
  if (!X || !W || !momentum || !active || !n_active || !labels_mapped || !row_lse || !dX)
    return PFC_ERR_INVALID_ARG;
  int st = check_shape(B, d, C, compute_dtype);
  if (st != PFC_OK) return st;
  if (x_dtype != compute_dtype || w_dtype != compute_dtype) return PFC_ERR_UNSUPPORTED;
  if (active_cap < 1 || active_cap > C) return PFC_ERR_CAPACITY;
  st = check_hparams(s, m, margin);
  if (st != PFC_OK) return st;
  if (!finite_pos(lr) || !isfinite(mu) || mu < 0.0f || mu >= 1.0f) return PFC_ERR_INVALID_ARG;
  const WsLayout L = ws_layout(B, d, C, active_cap, compute_dtype);
  if (!ws || ((uintptr_t)ws & 255) != 0 || ws_bytes < L.bytes) return PFC_ERR_WORKSPACE;
  StepArgs a{};
  a.X = X;
  a.W = W;
  a.W_master = W_master;
  a.M = momentum;
  a.active = active;
  a.n_active = n_active;
  a.labels_mapped = labels_mapped;
  a.row_lse = row_lse;
  a.dX = dX;
  a.B = B;
  a.d = d;
  a.C = C;
  a.cap = active_cap;
  a.dtype = compute_dtype;
  a.s = s;
  a.m = m;
  a.margin = margin;
  a.lr = lr;
  a.mu = mu;
  (void)hipGetLastError();
  const hipError_t e = launch_backward(a, step_ws(ws, L), (hipStream_t)stream);
  return e == hipSuccess ? PFC_OK : PFC_ERR_HIP;
}

const char* pfc_status_string(int status) {
  switch (status) {
    case PFC_OK: return "ok";
    case PFC_ERR_INVALID_ARG: return "invalid argument";
    case PFC_ERR_CAPACITY: return "active_cap smaller than the largest possible active set";
    case PFC_ERR_WORKSPACE: return "workspace missing or too small";
    case PFC_ERR_UNSUPPORTED: return "unsupported dtype or shape";
    case PFC_ERR_HIP: return "HIP launch failed";
    case PFC_ERR_SCRATCH: return "problem larger than the static scratch of the no-allocation entry point";
    default: return "unknown status";
  }
}

}  // extern "C"
