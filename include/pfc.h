/*
 * pfc.h - C ABI of the Partial FC classifier-head step on one class shard.
 *
 * Partial FC (arXiv 2010.05222): a class-sharded margin-softmax classifier
 * whose shard activates, per mini-batch, every positive class centre plus a
 * random subset of negatives (Sec. 3.3.1-3.3.2), computes normalised cosine
 * logits against the active centres only (Sec. 3.1, Sec. 3.3.3), and updates
 * only those centres (Eq. pfc_center_update).
 *
 * Conventions for every entry point:
 *  - Pointers are DEVICE pointers unless marked (host).  All device buffers
 *    are owned by the caller; the library never allocates or frees memory and
 *    never synchronises the host with the device.
 *  - Every call only enqueues kernels on `stream` (a hipStream_t passed as
 *    void*; NULL is the null stream) and returns.  Results are valid after the
 *    caller synchronises the stream.
 *  - Row-major layouts.  X is [B x d], W / W_master / momentum are [C x d]
 *    (one class centre per contiguous row of d elements), dX is [B x d] fp32.
 *  - All argument checks run before anything is enqueued.  On a non-zero
 *    return nothing was enqueued, except PFC_ERR_HIP (a launch failed; the
 *    outputs are then undefined).  Nothing is thrown across the ABI.
 *  - `ws` is a caller-owned device workspace of at least the size that
 *    pfc_workspace_bytes() reports.  It carries the sampler state and the
 *    forward pass's intermediates (norms, the logit store, softmax
 *    statistics) into the backward pass of the SAME step: a step's three calls
 *    must use the same workspace, in order, and no other step may use that
 *    workspace concurrently.
 */
#ifndef PFC_H
#define PFC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  PFC_OK = 0,
  PFC_ERR_INVALID_ARG = 1,  /* a size, pointer or hyper-parameter is out of range */
  PFC_ERR_CAPACITY = 2,     /* active_cap smaller than the largest possible |S| */
  PFC_ERR_WORKSPACE = 3,    /* ws is NULL, not 256-byte aligned, or smaller than required */
  PFC_ERR_UNSUPPORTED = 4,  /* dtype combination not implemented */
  PFC_ERR_HIP = 5,          /* a HIP launch failed */
  PFC_ERR_SCRATCH = 6       /* larger than the static scratch of pfc_sample_noalloc */
} pfc_status;

typedef enum { PFC_F32 = 0, PFC_BF16 = 1, PFC_F16 = 2 } pfc_dtype;

/* Target-logit margin (Sec. 3.1; the paper trains with CosFace m = 0.4 and
 * ArcFace m = 0.5 at scale s = 64, Sec. 4.1). */
typedef enum {
  PFC_COSFACE = 0,  /* additive cosine margin:  f_y = s * (cos - m)          */
  PFC_ARCFACE = 1   /* additive angular margin: f_y = s * cos(acos(cos) + m) */
} pfc_margin;

/* Size limits of this implementation (every limit has a parity test at its
 * boundary: B = 8192 on the 16-bit path, B = 4096 on the fp32 path). */
#define PFC_MAX_BATCH 8192
#define PFC_MAX_CLASSES (1LL << 30)

/*
 * Budget and capacity (Eq. local_sampling): the shard's activation budget is
 * b = r*C when r*C is an integer (within 1e-9 relative), else ceil(r*C); the
 * active set has |S| = max(b, |P|) <= max(b, min(B, C)) classes, which is the
 * `active_cap` every other call must be given.  Also reports the workspace
 * size needed by a step with these sizes and compute dtype; every call that
 * takes `ws` needs it at a 256-byte aligned device address (hipMalloc's are).
 *
 * 1 <= B <= PFC_MAX_BATCH; 1 <= C <= PFC_MAX_CLASSES; 0 < r <= 1;
 * 8 <= d <= 1024 with d a multiple of 8 (else PFC_ERR_INVALID_ARG); compute
 * one of pfc_dtype.  Implemented sizes (else PFC_ERR_UNSUPPORTED): the
 * bf16 / fp16 MFMA path takes d in {128, 256, 512}; the fp32 path, meant for
 * parity-scale problems, takes B <= 4096.  The same limits apply to every
 * entry point that takes d and a compute dtype.  bytes, active_cap are host
 * pointers.
 */
int pfc_workspace_bytes(int64_t B, int64_t d, int64_t C, double r,
                        int compute_dtype, size_t* bytes /*host*/,
                        int64_t* active_cap /*host*/);

/*
 * Stage 1 and 2: positive-preserving sampling and label remap (Sec. 3.3.1,
 * Sec. 3.3.2, Eq. local_sampling).
 *
 * labels         int64[B]  global class ids of the batch.
 * C, class_offset           the shard owns global ids [class_offset, class_offset + C).
 * r                         sampling rate, 0 < r <= 1.
 * seed                      sampler seed (a training step uses seed = step).
 * active         int32[active_cap] out: the active set S as sorted ascending
 *                local ids in [0, C); entries past n_active are unspecified.
 * n_active       int32[1]  out: |S|, left on the device.
 * labels_mapped  int32[B]  out: position of each row's local label in S
 *                (searchsorted), or -1 when the label is outside the shard.
 *
 * Selection rule: every owned label is kept; the remaining max(b - |P|, 0)
 * slots are the non-positive classes with the smallest 64-bit keys, ties
 * going to the lower class id.  The key of global class g is word (g mod 4)
 * of the Philox4x64-10 block (counter (g/4, 0, 0, 0), key (seed, 0))
 * (Salmon et al., SC'11), so it is independent of how classes are sharded.
 * Labels outside the shard are not an error: they map to -1.
 */
int pfc_sample(const int64_t* labels, int64_t B, int64_t C,
               int64_t class_offset, double r, uint64_t seed, int32_t* active,
               int64_t active_cap, int32_t* n_active, int32_t* labels_mapped,
               void* ws, size_t ws_bytes, void* stream);

/*
 * pfc_sample without a workspace, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc).  Same arguments, outputs and selection rule as
 * pfc_sample, minus ws / ws_bytes: the sampler's scratch is a file-scope
 * device array of the library, about 21 MiB on every device the library runs
 * on, held until the process ends.  Its address is looked up on the first
 * call on each device (that call must run with the device current).
 *
 * C above PFC_NOALLOC_MAX_CLASSES is PFC_ERR_SCRATCH (checked before any
 * launch; use pfc_sample with a workspace instead).  The call allocates
 * nothing and enqueues the same kernels as pfc_sample; the scratch keeps the
 * last call's contents and every call clears what must start at zero.  All
 * calls on one device share the one scratch: calls that overlap on a device
 * (concurrent streams, or host threads) race and give undefined results.
 */
#define PFC_NOALLOC_MAX_CLASSES (1LL << 21)
int pfc_sample_noalloc(const int64_t* labels, int64_t B, int64_t C,
                       int64_t class_offset, double r, uint64_t seed,
                       int32_t* active, int64_t active_cap, int32_t* n_active,
                       int32_t* labels_mapped, void* stream);

/*
 * Stages 3-5: normalise the rows of X and the active rows of W, the cosine
 * logits cos = x_hat . w_hat (a B x |S| contraction over d), the margin on the
 * target logit, and the row-wise log-sum-exp cross-entropy over S
 * (Sec. 3.1, Eq. sampled_probability, Sec. 3.2.1).
 *
 * X       [B x d] in x_dtype;  W [C x d] in w_dtype (the persistent shard).
 * active, n_active, labels_mapped: outputs of pfc_sample for this batch.
 *         The kernels rely on what pfc_sample guarantees and do not check
 *         it: n_active in [0, active_cap], active[0, n_active) ids in [0, C).
 *         A labels_mapped entry outside [0, n_active) counts as an unowned
 *         label (no target term, loss term 0).
 * compute must equal w_dtype and x_dtype (fp32, bf16 or fp16 operands; the
 *         contraction always accumulates in fp32).
 * s > 0 scale; margin m >= 0 (ArcFace: m < pi).
 * tau     PFC* conflict threshold (Sec. 3.3.4, Eq. noise_filtering): a
 *         non-target logit whose unmargined cosine exceeds tau is left out of
 *         the row's denominator, and so gets no gradient in the backward of
 *         this step; the target logit is never filtered.  tau >= 1 (or +inf)
 *         is plain PFC; NaN is PFC_ERR_INVALID_ARG.  Rows whose label is
 *         outside the shard have only negatives.
 * loss    float[1] out: (1/B) * sum over rows with an owned label of
 *         (lse_n - f_{n, y_n}); rows whose label is outside the shard add 0
 *         (their target term belongs to the owning shard).
 * row_lse float[B] out: lse_n = log sum_{j in S} exp(f_{n,j}), the per-row
 *         statistic a multi-shard caller would combine across shards.  A
 *         row whose label is outside the shard and whose every logit the
 *         PFC* filter drops has an empty denominator: lse_n = -inf, and the
 *         backward gives it no probability and no gradient.
 */
int pfc_forward_loss(const void* X, int x_dtype, int64_t B, int64_t d,
                     const void* W, int w_dtype, int64_t C,
                     const int32_t* active, const int32_t* n_active,
                     int64_t active_cap, const int32_t* labels_mapped,
                     int compute_dtype, float s, float m, int margin,
                     float tau, float* loss, float* row_lse, void* ws,
                     size_t ws_bytes, void* stream);

/*
 * Stage 6: backward through the margin softmax and both normalisations, then
 * lazy momentum SGD on the active rows only (Eq. proxy_update,
 * Eq. pfc_center_update, Sec. 3.2.1 matrix form).
 *
 * With G = (P - Y)/B (P the softmax over S, Y one-hot at labels_mapped) and
 * dcos = s * G (times sin(theta + m)/sin(theta) at an ArcFace target):
 *   dX  = d L / d X           (fp32 [B x d] out), through x_hat = x/||x||;
 *   g_j = d L / d W[S_j]      through w_hat = w/||w||, summed over all rows;
 *   M[S_j] <- mu * M[S_j] + g_j;   W'[S_j] <- W'[S_j] - lr * M[S_j]
 * where W' is W_master (fp32) when given, after which W[S_j] is its
 * round-to-nearest-even value in w_dtype; without a master the fp32 result is
 * rounded into W.  Rows not in S are not read or written.
 *
 * Same X, W, active, n_active, labels_mapped, dtypes, s, m, margin and ws as
 * the forward call of this step; W must not change between the two calls.
 * row_lse  float[B] in: the log-sum-exp the gradient is normalised with (the
 *          forward's output, or a cross-shard combination of it).
 * W        [C x d] in/out;  W_master fp32 [C x d] in/out or NULL;
 * momentum fp32 [C x d] in/out;  lr > 0, 0 <= mu < 1.
 */
int pfc_backward_update(const void* X, int x_dtype, int64_t B, int64_t d,
                        void* W, int w_dtype, float* W_master, float* momentum,
                        int64_t C, const int32_t* active,
                        const int32_t* n_active, int64_t active_cap,
                        const int32_t* labels_mapped, int compute_dtype,
                        float s, float m, int margin, const float* row_lse,
                        float lr, float mu, float* dX, void* ws,
                        size_t ws_bytes, void* stream);

/* Static description of a status code (never NULL). */
const char* pfc_status_string(int status);

/*
 * Measurement hook, outside the step itself.  Kernels (or kernel sequences)
 * of a step that can be timed on their own:
 */
typedef enum {
  PFC_K_SAMPLE = 0,     /* the whole sampling + remap sequence of pfc_sample */
  PFC_K_PREP = 1,       /* inverse norms of X rows and active W rows */
  PFC_K_FWD_GEMM = 2,   /* cosine contraction + margin + per-tile softmax statistics */
  PFC_K_LSE = 3,        /* per-row log-sum-exp and the loss */
  PFC_K_DX_GEMM = 4,    /* split-K contraction of the feature gradient */
  PFC_K_DX_FINAL = 5,   /* split reduction + normalisation backward of X */
  PFC_K_DW_UPDATE = 6,  /* class-gradient contraction + fused momentum update */
  PFC_K_COUNT = 7
} pfc_kernel;

/*
 * pfc_timing_begin: from now on, each launch of `kernel` (up to max_launches,
 * 1..65536) is bracketed by a pair of HIP events recorded on the stream it is
 * launched on.  The events are created here (host-side HIP objects; no device
 * memory is allocated).  Not thread-safe; one kernel at a time.
 * pfc_timing_end: waits for the recorded events, returns the summed duration
 * in milliseconds and the number of bracketed launches (host pointers), and
 * disarms the hook.  Returns PFC_ERR_INVALID_ARG when nothing is armed.
 */
int pfc_timing_begin(int kernel, int max_launches);
int pfc_timing_end(double* total_ms /*host*/, int* launches /*host*/);

/*
 * Tiered class storage (Sec. 3.3.3, the paragraph on asynchronous
 * hierarchical class storage, Fig. async_pipeline): the shard's class bank
 * (W, momentum, and the fp32 master if any) lives in pinned host memory, and
 * a step runs on a device SLOT holding only its active rows, slot row j being
 * bank row active[j].  The step itself is the three calls above with the slot
 * as W / momentum / W_master and an identity active list 0, 1, ..., cap - 1
 * (the sampler's list stays in active space for these copies; labels_mapped is
 * already a position in S).  With a ring of slots and side streams, the rows
 * of step t+1 are staged while step t runs:
 *   stage      cold rows - S(t+1) minus the previous sets still held in slots
 *              (prev: S(t), prev2: S(t-1) or NULL) - bank -> the next slot,
 *              any time after the write-back of the step that last used it
 *              and of every step whose rows it may read from the bank;
 *   patch      rows S(t+1) shares with an earlier set, that set's slot -> the
 *              next slot, after that step's update, older sets first (the
 *              newest copy wins); the next slot is ready after stage and patch;
 *   writeback  a slot -> bank, after its step, skipping the rows of the next
 *              step's set when it is given (next_active / next_n, or NULL):
 *              that step writes them back with newer values, and the next
 *              stages take them from its slot; the slot is free for reuse
 *              after the write-back.
 * Each call copies the rows of n_arrays arrays (1 to PFC_BANK_MAX_ARRAYS: W,
 * momentum and the master if any) at once: array a is a byte copy of
 * row_bytes[a] per row (a multiple of 16, at most 65536; d * 2 for 16-bit W,
 * d * 4 for momentum and the master) between banks[a] and slots[a] (or
 * prev_slots[a] and next_slots[a]); the three pointer / size arrays are host
 * arrays of n_arrays entries, each pointer non-NULL, a source never equal to
 * its destination.  active / next_active / prev_active are sorted ascending
 * id lists of active_cap entries (pfc_sample's output) with their device
 * counts n (a list and its count are given together or both NULL);
 * entries past the count are ignored, and counts are clamped to [0, cap].
 * Slots are [active_cap x row] device buffers.  Bank pointers (and
 * bank_version) must be host memory allocated pinned and mapped (hipHostMalloc,
 * or torch's pin_memory) or device memory; anything else - pageable host memory
 * in particular - is PFC_ERR_INVALID_ARG, checked before any launch.
 *
 * Versions (optional, pass both or neither):
 * bank_version int32[C] (host, pinned) holds the version of each bank row's
 * last write-back; row_version int32[C] (device) the version of each row's
 * last staging, starting from all zeros on both sides.  stage stamps
 * row_version[c] = version for every c in S(t+1), and a cold row whose
 * bank_version differs from its row_version (an update of it not yet written
 * back) adds 1 to stale[0]; writeback stamps bank_version[c] = version after
 * the row's data in every array has reached the bank.  Ids outside [0, C)
 * are not copied and also add 1 to stale.
 * stale (device int32[1]) may be NULL.  A caller uses version = t + 1 for the
 * rows of step t.
 */
#define PFC_BANK_MAX_ARRAYS 3
int pfc_bank_stage(int n_arrays, const void* const* banks /*host array*/,
                   void* const* slots /*host array*/,
                   const int64_t* row_bytes /*host array*/, int64_t C,
                   const int32_t* next_active, const int32_t* next_n,
                   const int32_t* prev_active /*or NULL*/,
                   const int32_t* prev_n /*or NULL*/,
                   const int32_t* prev2_active /*or NULL*/,
                   const int32_t* prev2_n /*or NULL*/, int64_t active_cap,
                   const int32_t* bank_version /*host, or NULL*/,
                   int32_t* row_version /*or NULL*/, int32_t version,
                   int32_t* stale /*or NULL*/, void* stream);
int pfc_bank_patch(int n_arrays, const void* const* prev_slots /*host array*/,
                   void* const* next_slots /*host array*/,
                   const int64_t* row_bytes /*host array*/,
                   const int32_t* prev_active, const int32_t* prev_n,
                   const int32_t* next_active, const int32_t* next_n,
                   int64_t active_cap, void* stream);
int pfc_bank_writeback(int n_arrays, const void* const* slots /*host array*/,
                       void* const* banks /*host array*/,
                       const int64_t* row_bytes /*host array*/,
                       const int32_t* active, const int32_t* n_active,
                       const int32_t* next_active /*or NULL*/,
                       const int32_t* next_n /*or NULL*/, int64_t active_cap,
                       int64_t C, int32_t* bank_version /*host, or NULL*/,
                       int32_t version, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* PFC_H */
