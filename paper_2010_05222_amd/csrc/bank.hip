// Tiered class storage: the shard's class bank (W, momentum, master rows) in
// pinned host memory, with only the active rows S(t) staged in a device slot
// for the step (Sec. 3.3.3, the paragraph on asynchronous hierarchical class
// storage, and Fig. async_pipeline).
//
// Three row copies, each moving every array of the bank (W, momentum, the
// master if any) for its rows in one launch, 16 bytes per lane:
//  - stage:     cold rows of S(t+1) - those in neither of the (up to two)
//               previous active sets still held in slots - from the bank
//               into the next slot, with a check of the per-row versions
//               (the host copy of a row must carry the version of its last
//               update);
//  - patch:     rows S(t+1) shares with an earlier set, from that set's slot
//               into the next one, once its step has updated them;
//  - writeback: the slot's rows back into the bank, stamping their version,
//               except rows the next step also holds (its write-back carries
//               their newer values).
// The host side of each copy goes over the host link with ordinary vector
// loads and stores on the mapped pinned pages; the device side is HBM.  One
// launch per row set and direction, rather than one per array, keeps rows of
// every size on both directions of the link at once: a 1 KB-row write-back
// beside a 2 KB-row stage measured well below the two together.
// Membership in S(t) is a binary search over its sorted id list, one row per
// lane: a wave settles 64 rows in one search's worth of dependent loads, then
// copies them eight at a time (a row per lane, and a search per row, made
// each wave spend most of its time in dependent loads rather than on the
// link).  The two host-link copies run on a fixed grid of 2048 waves that
// walks the rows: they wait on the host link most of the time, and a grid of
// one wave per 64 rows would hold the CUs and starve the step's kernels
// running beside them on other streams.  The patch, a device-to-device copy,
// takes one wave per 64 rows.
#include "pfc_device.h"
#include "pfc.h"

namespace pfc {
namespace {

constexpr int kBankWaves = 4;     // waves per workgroup
constexpr int kBankGrid = 512;    // workgroups of a copy
constexpr int64_t kMaxRowBytes = 1 << 16;

// Index of v in the ascending a[0, n), or -1; each lane looks up its own v.
// The number of steps depends on n only (a branch-free lower bound), so the
// lanes of a wave run their searches side by side: a wave settles the rows
// of 64 lanes in one search's worth of dependent loads.
__device__ __forceinline__ int64_t find_sorted(const int32_t* __restrict__ a, int64_t n,
                                               int32_t v) {
  if (n <= 0) return -1;
  int64_t base = 0, len = n;
  while (len > 1) {
    const int64_t half = len >> 1;   // base + half < base + len <= n
    base = a[base + half] < v ? base + half : base;
    len -= half;
  }
  const int64_t i = base + (a[base] < v ? 1 : 0);
  return (i < n && a[i] == v) ? i : -1;
}

__device__ __forceinline__ int64_t rows_of(const int32_t* n_p, int64_t cap) {
  const int64_t n = *n_p;
  return n < 0 ? 0 : (n > cap ? cap : n);
}

__device__ __forceinline__ int64_t wave_index() {
  return (int64_t)blockIdx.x * kBankWaves + (threadIdx.x >> 6);
}
__device__ __forceinline__ int64_t wave_count() { return (int64_t)gridDim.x * kBankWaves; }

// A wave settles the rows of its 64 lanes (lane l: row j0 + l of the list
// it walks) and then copies them kGroup at a time, array after array: all
// loads of a pass over kGroup rows are issued before the first store, so a
// wave keeps kGroup x 1 KB in flight on the host link.
constexpr int kGroup = 8;

// The arrays a call copies (W, momentum, master: up to kMaxArrays), each with
// rows of row16[a] 16-byte pieces.  One launch moves every array of a row
// set, so both directions of the host link carry all row sizes at once.
constexpr int kMaxArrays = PFC_BANK_MAX_ARRAYS;
struct Arrays {
  const uint4* src[kMaxArrays];
  uint4* dst[kMaxArrays];
  int row16[kMaxArrays];
  int n;
};

__device__ __forceinline__ int64_t lane_value(int64_t v, int l) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, l);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)v >> 32), l);
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// Copies the rows the lanes hold: lane l's row, when bit l of ok is set, goes
// from source row srow to destination row drow (both held by lane l).
__device__ __forceinline__ void copy_rows(const Arrays& ar, uint64_t ok, int64_t srow,
                                          int64_t drow, int lane) {
#pragma unroll 1
  for (int s0 = 0; s0 < 64; s0 += kGroup) {
    const uint32_t m = (uint32_t)(ok >> s0) & ((1u << kGroup) - 1);
    if (m == 0) continue;
    int64_t sr[kGroup], dr[kGroup];
#pragma unroll
    for (int k = 0; k < kGroup; ++k) {
      sr[k] = lane_value(srow, s0 + k);
      dr[k] = lane_value(drow, s0 + k);
    }
    for (int a = 0; a < ar.n; ++a) {
      const int row16 = ar.row16[a];
      const uint4* __restrict__ src = ar.src[a];
      uint4* __restrict__ dst = ar.dst[a];
      for (int i = lane; i < row16; i += 64) {
        uint4 v[kGroup];
#pragma unroll
        for (int k = 0; k < kGroup; ++k)
          if ((m >> k) & 1) v[k] = src[sr[k] * row16 + i];
#pragma unroll
        for (int k = 0; k < kGroup; ++k)
          if ((m >> k) & 1) dst[dr[k] * row16 + i] = v[k];
      }
    }
  }
}

__global__ void __launch_bounds__(64 * kBankWaves) k_bank_stage(
    Arrays ar, int64_t C, const int32_t* __restrict__ next_active,
    const int32_t* __restrict__ next_n, const int32_t* __restrict__ prev_active,
    const int32_t* __restrict__ prev_n, const int32_t* __restrict__ prev2_active,
    const int32_t* __restrict__ prev2_n, int64_t cap,
    const int32_t* __restrict__ bank_version, int32_t* __restrict__ row_version,
    int32_t version, int32_t* __restrict__ stale) {
  const int lane = threadIdx.x & 63;
  const int64_t n = rows_of(next_n, cap);
  const int64_t np = prev_active ? rows_of(prev_n, cap) : 0;
  const int64_t np2 = prev2_active ? rows_of(prev2_n, cap) : 0;
  for (int64_t j0 = wave_index() * 64; j0 < n; j0 += wave_count() * 64) {
    const int64_t j = j0 + lane;
    const int32_t c = j < n ? next_active[j] : -1;
    const bool in_bank = c >= 0 && c < C;
    const bool bad = j < n && !in_bank;   // not a row of the bank: nothing is copied
    const bool overlap = find_sorted(prev_active, np, c) >= 0 || find_sorted(prev2_active, np2, c) >= 0;
    const bool cold = in_bank && !overlap;
    bool behind = false;
    if (row_version && cold) behind = bank_version[c] != row_version[c];
    const uint64_t ok = __ballot(cold);
    const int n_stale = __popcll(__ballot(bad)) + __popcll(__ballot(behind));
    if (stale && lane == 0 && n_stale > 0) atomicAdd(stale, n_stale);
    copy_rows(ar, ok, cold ? c : 0, j, lane);
    if (row_version && in_bank) row_version[c] = version;
  }
}

__global__ void __launch_bounds__(64 * kBankWaves) k_bank_patch(
    Arrays ar, const int32_t* __restrict__ prev_active, const int32_t* __restrict__ prev_n,
    const int32_t* __restrict__ next_active, const int32_t* __restrict__ next_n, int64_t cap) {
  const int lane = threadIdx.x & 63;
  const int64_t n = rows_of(next_n, cap), np = rows_of(prev_n, cap);
  for (int64_t j0 = wave_index() * 64; j0 < n; j0 += wave_count() * 64) {
    const int64_t j = j0 + lane;
    const int64_t i = find_sorted(prev_active, np, j < n ? next_active[j] : -1);
    copy_rows(ar, __ballot(j < n && i >= 0), i >= 0 ? i : 0, j, lane);
  }
}

__global__ void __launch_bounds__(64 * kBankWaves) k_bank_writeback(
    Arrays ar, const int32_t* __restrict__ active, const int32_t* __restrict__ n_active,
    const int32_t* __restrict__ next_active, const int32_t* __restrict__ next_n, int64_t cap,
    int64_t C, int32_t* __restrict__ bank_version, int32_t version) {
  const int lane = threadIdx.x & 63;
  const int64_t n = rows_of(n_active, cap);
  const int64_t nn = next_active ? rows_of(next_n, cap) : 0;
  for (int64_t j0 = wave_index() * 64; j0 < n; j0 += wave_count() * 64) {
    const int64_t j = j0 + lane;
    const int32_t c = j < n ? active[j] : -1;
    const bool ok = c >= 0 && c < C && find_sorted(next_active, nn, c) < 0;
    copy_rows(ar, __ballot(ok), j, ok ? c : 0, lane);
    if (bank_version) {
      // Every array's row reaches system scope before the row's version does.
      __threadfence_system();
      if (ok) bank_version[c] = version;
    }
  }
}

// A pointer the kernels may dereference: device memory, or host memory
// allocated pinned and mapped (its device address equal to its host address).
bool device_accessible(const void* p) {
  hipPointerAttribute_t at;
  if (hipPointerGetAttributes(&at, p) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  if (at.type == hipMemoryTypeDevice || at.type == hipMemoryTypeManaged) return true;
  if (at.type == hipMemoryTypeHost) return at.devicePointer == p;
  return false;
}

int common_checks(int64_t active_cap) {
  if (active_cap < 1 || active_cap > PFC_MAX_CLASSES) return PFC_ERR_INVALID_ARG;
  return PFC_OK;
}

// The arrays of a call: n in [1, PFC_BANK_MAX_ARRAYS], every pointer given and
// reachable from the device, row sizes multiples of 16 up to kMaxRowBytes.
int take_arrays(int n, const void* const* src, void* const* dst, const int64_t* row_bytes,
                Arrays* ar) {
  if (n < 1 || n > kMaxArrays || !src || !dst || !row_bytes) return PFC_ERR_INVALID_ARG;
  *ar = Arrays{};
  ar->n = n;
  for (int a = 0; a < n; ++a) {
    const int64_t rb = row_bytes[a];
    if (!src[a] || !dst[a] || src[a] == dst[a]) return PFC_ERR_INVALID_ARG;
    if (rb < 16 || rb > kMaxRowBytes || rb % 16 != 0) return PFC_ERR_INVALID_ARG;
    ar->src[a] = (const uint4*)src[a];
    ar->dst[a] = (uint4*)dst[a];
    ar->row16[a] = (int)(rb / 16);
  }
  return PFC_OK;
}

int arrays_accessible(const Arrays& ar) {
  for (int a = 0; a < ar.n; ++a)
    if (!device_accessible(ar.src[a]) || !device_accessible(ar.dst[a])) return PFC_ERR_INVALID_ARG;
  return PFC_OK;
}

int device_present() {
  int n = 0;
  if (hipGetDeviceCount(&n) != hipSuccess || n < 1) {
    (void)hipGetLastError();
    return PFC_ERR_HIP;
  }
  return PFC_OK;
}

unsigned grid_of(int64_t cap) {
  const int64_t g = ceil_div(cap, 64 * kBankWaves);
  return (unsigned)(g < kBankGrid ? g : kBankGrid);
}

}  // namespace
}  // namespace pfc

using namespace pfc;

extern "C" {

int pfc_bank_stage(int n_arrays, const void* const* banks, void* const* slots,
                   const int64_t* row_bytes, int64_t C, const int32_t* next_active,
                   const int32_t* next_n, const int32_t* prev_active, const int32_t* prev_n,
                   const int32_t* prev2_active, const int32_t* prev2_n, int64_t active_cap,
                   const int32_t* bank_version, int32_t* row_version, int32_t version,
                   int32_t* stale, void* stream) {
  if (!next_active || !next_n) return PFC_ERR_INVALID_ARG;
  if (C < 1 || C > PFC_MAX_CLASSES) return PFC_ERR_INVALID_ARG;
  if ((prev_active == nullptr) != (prev_n == nullptr)) return PFC_ERR_INVALID_ARG;
  if ((prev2_active == nullptr) != (prev2_n == nullptr)) return PFC_ERR_INVALID_ARG;
  if ((bank_version == nullptr) != (row_version == nullptr)) return PFC_ERR_INVALID_ARG;
  Arrays ar;
  int st = take_arrays(n_arrays, banks, slots, row_bytes, &ar);
  if (st == PFC_OK) st = common_checks(active_cap);
  if (st != PFC_OK) return st;
  const int dv = device_present();
  if (dv != PFC_OK) return dv;
  if (arrays_accessible(ar) != PFC_OK) return PFC_ERR_INVALID_ARG;
  if (bank_version && !device_accessible(bank_version)) return PFC_ERR_INVALID_ARG;
  (void)hipGetLastError();
  hipLaunchKernelGGL(k_bank_stage, dim3(grid_of(active_cap)), dim3(64 * kBankWaves), 0,
                     (hipStream_t)stream, ar, C, next_active, next_n, prev_active, prev_n,
                     prev2_active, prev2_n, active_cap, bank_version, row_version, version,
                     stale);
  return hipGetLastError() == hipSuccess ? PFC_OK : PFC_ERR_HIP;
}

int pfc_bank_patch(int n_arrays, const void* const* prev_slots, void* const* next_slots,
                   const int64_t* row_bytes, const int32_t* prev_active, const int32_t* prev_n,
                   const int32_t* next_active, const int32_t* next_n, int64_t active_cap,
                   void* stream) {
  if (!prev_active || !prev_n || !next_active || !next_n) return PFC_ERR_INVALID_ARG;
  Arrays ar;
  int st = take_arrays(n_arrays, prev_slots, next_slots, row_bytes, &ar);
  if (st == PFC_OK) st = common_checks(active_cap);
  if (st != PFC_OK) return st;
  const int dv = device_present();
  if (dv != PFC_OK) return dv;
  if (arrays_accessible(ar) != PFC_OK) return PFC_ERR_INVALID_ARG;
  (void)hipGetLastError();
  // A device-to-device copy: enough waves for every group of rows at once.
  hipLaunchKernelGGL(k_bank_patch, dim3((unsigned)ceil_div(active_cap, 64 * kBankWaves)),
                     dim3(64 * kBankWaves), 0, (hipStream_t)stream, ar, prev_active, prev_n,
                     next_active, next_n, active_cap);
  return hipGetLastError() == hipSuccess ? PFC_OK : PFC_ERR_HIP;
}

int pfc_bank_writeback(int n_arrays, const void* const* slots, void* const* banks,
                       const int64_t* row_bytes, const int32_t* active, const int32_t* n_active,
                       const int32_t* next_active, const int32_t* next_n, int64_t active_cap,
                       int64_t C, int32_t* bank_version, int32_t version, void* stream) {
  if (!active || !n_active) return PFC_ERR_INVALID_ARG;
  if ((next_active == nullptr) != (next_n == nullptr)) return PFC_ERR_INVALID_ARG;
  if (C < 1 || C > PFC_MAX_CLASSES) return PFC_ERR_INVALID_ARG;
  Arrays ar;
  int st = take_arrays(n_arrays, slots, banks, row_bytes, &ar);
  if (st == PFC_OK) st = common_checks(active_cap);
  if (st != PFC_OK) return st;
  const int dv = device_present();
  if (dv != PFC_OK) return dv;
  if (arrays_accessible(ar) != PFC_OK) return PFC_ERR_INVALID_ARG;
  if (bank_version && !device_accessible(bank_version)) return PFC_ERR_INVALID_ARG;
  (void)hipGetLastError();
  hipLaunchKernelGGL(k_bank_writeback, dim3(grid_of(active_cap)), dim3(64 * kBankWaves), 0,
                     (hipStream_t)stream, ar, active, n_active, next_active, next_n, active_cap,
                     C, bank_version, version);
  return hipGetLastError() == hipSuccess ? PFC_OK : PFC_ERR_HIP;
}

}  // extern "C"
