// Tiered class storage: the shard's class bank (W, momentum, master rows) in
// pinned host memory, with only the active rows S(t) staged in a device slot
// for the step (Sec. 3.3.3, the paragraph on asynchronous hierarchical class
// storage, and Fig. async_pipeline).
//
// Three row copies, 16 bytes per lane, eight rows per wave at a time:
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
// loads and stores on the mapped pinned pages; the device side is HBM.
// Membership in S(t) is a binary search over its sorted id list.  The two
// host-link copies run on a fixed grid of 2048 waves that walks the rows, with
// all eight loads of a group issued before its stores: they wait on the host
// link most of the time, and a grid of one wave per row would hold the CUs
// and starve the step's kernels running beside them on other streams.  The
// patch, a device-to-device copy, takes one wave per group of rows.
#include "pfc_device.h"
#include "pfc.h"

namespace pfc {
namespace {

constexpr int kBankWaves = 4;     // waves per workgroup
constexpr int kBankGrid = 512;    // workgroups of a copy
constexpr int64_t kMaxRowBytes = 1 << 16;

// Index of v in the ascending a[0, n), or -1.
__device__ __forceinline__ int64_t find_sorted(const int32_t* __restrict__ a, int64_t n,
                                               int32_t v) {
  int64_t lo = 0, hi = n;
  while (lo < hi) {
    const int64_t mid = (lo + hi) >> 1;
    if (a[mid] < v) lo = mid + 1;
    else hi = mid;
  }
  return (lo < n && a[lo] == v) ? lo : -1;
}

__device__ __forceinline__ int64_t rows_of(const int32_t* n_p, int64_t cap) {
  const int64_t n = *n_p;
  return n < 0 ? 0 : (n > cap ? cap : n);
}

__device__ __forceinline__ int64_t wave_index() {
  return (int64_t)blockIdx.x * kBankWaves + (threadIdx.x >> 6);
}
__device__ __forceinline__ int64_t wave_count() { return (int64_t)gridDim.x * kBankWaves; }

// A wave copies kGroup rows at a time: all their loads are issued before the
// first store, so a wave keeps kGroup x 1 KB in flight on the host link.
constexpr int kGroup = 8;

struct RowGroup {
  const uint4* src[kGroup];
  uint4* dst[kGroup];
  bool ok[kGroup];
};

__device__ __forceinline__ void copy_group(const RowGroup& g, int row16, int lane) {
  for (int i = lane; i < row16; i += 64) {
    uint4 v[kGroup];
#pragma unroll
    for (int k = 0; k < kGroup; ++k)
      if (g.ok[k]) v[k] = g.src[k][i];
#pragma unroll
    for (int k = 0; k < kGroup; ++k)
      if (g.ok[k]) g.dst[k][i] = v[k];
  }
}

__global__ void __launch_bounds__(64 * kBankWaves) k_bank_stage(
    const uint4* __restrict__ bank, int64_t C, int row16, const int32_t* __restrict__ next_active,
    const int32_t* __restrict__ next_n, const int32_t* __restrict__ prev_active,
    const int32_t* __restrict__ prev_n, const int32_t* __restrict__ prev2_active,
    const int32_t* __restrict__ prev2_n, int64_t cap, uint4* __restrict__ slot,
    const int32_t* __restrict__ bank_version, int32_t* __restrict__ row_version,
    int32_t version, int32_t* __restrict__ stale) {
  const int lane = threadIdx.x & 63;
  const int64_t n = rows_of(next_n, cap);
  const int64_t np = prev_active ? rows_of(prev_n, cap) : 0;
  const int64_t np2 = prev2_active ? rows_of(prev2_n, cap) : 0;
  for (int64_t j0 = wave_index() * kGroup; j0 < n; j0 += wave_count() * kGroup) {
    RowGroup g;
    int32_t cls[kGroup];
#pragma unroll
    for (int k = 0; k < kGroup; ++k) {
      const int64_t j = j0 + k;
      cls[k] = -1;
      g.ok[k] = false;
      g.src[k] = bank;
      g.dst[k] = slot;
      if (j >= n) continue;
      const int32_t c = next_active[j];
      if (c < 0 || c >= C) {   // not a row of the bank: nothing is copied
        if (lane == 0 && stale) atomicAdd(stale, 1);
        continue;
      }
      cls[k] = c;
      const bool overlap = (np > 0 && find_sorted(prev_active, np, c) >= 0) ||
                           (np2 > 0 && find_sorted(prev2_active, np2, c) >= 0);
      if (overlap) continue;
      if (row_version && lane == 0 && bank_version[c] != row_version[c] && stale)
        atomicAdd(stale, 1);
      g.ok[k] = true;
      g.src[k] = bank + (int64_t)c * row16;
      g.dst[k] = slot + j * row16;
    }
    copy_group(g, row16, lane);
    if (row_version && lane == 0) {
#pragma unroll
      for (int k = 0; k < kGroup; ++k)
        if (cls[k] >= 0) row_version[cls[k]] = version;
    }
  }
}

__global__ void __launch_bounds__(64 * kBankWaves) k_bank_patch(
    const uint4* __restrict__ prev_slot, const int32_t* __restrict__ prev_active,
    const int32_t* __restrict__ prev_n, const int32_t* __restrict__ next_active,
    const int32_t* __restrict__ next_n, int64_t cap, int row16, uint4* __restrict__ next_slot) {
  const int lane = threadIdx.x & 63;
  const int64_t n = rows_of(next_n, cap), np = rows_of(prev_n, cap);
  for (int64_t j0 = wave_index() * kGroup; j0 < n; j0 += wave_count() * kGroup) {
    RowGroup g;
#pragma unroll
    for (int k = 0; k < kGroup; ++k) {
      const int64_t j = j0 + k;
      const int64_t i = j < n ? find_sorted(prev_active, np, next_active[j]) : -1;
      g.ok[k] = i >= 0;
      g.src[k] = i >= 0 ? prev_slot + i * row16 : prev_slot;
      g.dst[k] = i >= 0 ? next_slot + j * row16 : next_slot;
    }
    copy_group(g, row16, lane);
  }
}

__global__ void __launch_bounds__(64 * kBankWaves) k_bank_writeback(
    const uint4* __restrict__ slot, const int32_t* __restrict__ active,
    const int32_t* __restrict__ n_active, const int32_t* __restrict__ next_active,
    const int32_t* __restrict__ next_n, int64_t cap, int row16, int64_t C,
    uint4* __restrict__ bank, int32_t* __restrict__ bank_version, int32_t version) {
  const int lane = threadIdx.x & 63;
  const int64_t n = rows_of(n_active, cap);
  const int64_t nn = next_active ? rows_of(next_n, cap) : 0;
  for (int64_t j0 = wave_index() * kGroup; j0 < n; j0 += wave_count() * kGroup) {
    RowGroup g;
    int32_t cls[kGroup];
#pragma unroll
    for (int k = 0; k < kGroup; ++k) {
      const int64_t j = j0 + k;
      const int32_t c = j < n ? active[j] : -1;
      const bool ok = c >= 0 && c < C && !(nn > 0 && find_sorted(next_active, nn, c) >= 0);
      cls[k] = ok ? c : -1;
      g.ok[k] = ok;
      g.src[k] = ok ? slot + j * row16 : slot;
      g.dst[k] = ok ? bank + (int64_t)c * row16 : bank;
    }
    copy_group(g, row16, lane);
    if (bank_version) {
      // The rows' data reach system scope before their versions do.
      __threadfence_system();
      if (lane == 0) {
#pragma unroll
        for (int k = 0; k < kGroup; ++k)
          if (cls[k] >= 0) bank_version[cls[k]] = version;
      }
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

int common_checks(int64_t row_bytes, int64_t active_cap) {
  if (row_bytes < 16 || row_bytes > kMaxRowBytes || row_bytes % 16 != 0) return PFC_ERR_INVALID_ARG;
  if (active_cap < 1 || active_cap > PFC_MAX_CLASSES) return PFC_ERR_INVALID_ARG;
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
  const int64_t g = ceil_div(cap, kBankWaves);
  return (unsigned)(g < kBankGrid ? g : kBankGrid);
}

}  // namespace
}  // namespace pfc

using namespace pfc;

extern "C" {

int pfc_bank_stage(const void* bank, int64_t C, int64_t row_bytes, const int32_t* next_active,
                   const int32_t* next_n, const int32_t* prev_active, const int32_t* prev_n,
                   const int32_t* prev2_active, const int32_t* prev2_n, int64_t active_cap,
                   void* slot, const int32_t* bank_version, int32_t* row_version,
                   int32_t version, int32_t* stale, void* stream) {
  if (!bank || !next_active || !next_n || !slot) return PFC_ERR_INVALID_ARG;
  if (C < 1 || C > PFC_MAX_CLASSES) return PFC_ERR_INVALID_ARG;
  if ((prev_active == nullptr) != (prev_n == nullptr)) return PFC_ERR_INVALID_ARG;
  if ((prev2_active == nullptr) != (prev2_n == nullptr)) return PFC_ERR_INVALID_ARG;
  if ((bank_version == nullptr) != (row_version == nullptr)) return PFC_ERR_INVALID_ARG;
  const int st = common_checks(row_bytes, active_cap);
  if (st != PFC_OK) return st;
  const int dv = device_present();
  if (dv != PFC_OK) return dv;
  if (!device_accessible(bank) || !device_accessible(slot)) return PFC_ERR_INVALID_ARG;
  if (bank_version && !device_accessible(bank_version)) return PFC_ERR_INVALID_ARG;
  (void)hipGetLastError();
  hipLaunchKernelGGL(k_bank_stage, dim3(grid_of(active_cap)), dim3(64 * kBankWaves), 0,
                     (hipStream_t)stream, (const uint4*)bank, C, (int)(row_bytes / 16),
                     next_active, next_n, prev_active, prev_n, prev2_active, prev2_n,
                     active_cap, (uint4*)slot,
                     bank_version, row_version, version, stale);
  return hipGetLastError() == hipSuccess ? PFC_OK : PFC_ERR_HIP;
}

int pfc_bank_patch(const void* prev_slot, const int32_t* prev_active, const int32_t* prev_n,
                   const int32_t* next_active, const int32_t* next_n, int64_t active_cap,
                   int64_t row_bytes, void* next_slot, void* stream) {
  if (!prev_slot || !prev_active || !prev_n || !next_active || !next_n || !next_slot)
    return PFC_ERR_INVALID_ARG;
  if (prev_slot == next_slot) return PFC_ERR_INVALID_ARG;
  const int st = common_checks(row_bytes, active_cap);
  if (st != PFC_OK) return st;
  const int dv = device_present();
  if (dv != PFC_OK) return dv;
  if (!device_accessible(prev_slot) || !device_accessible(next_slot)) return PFC_ERR_INVALID_ARG;
  (void)hipGetLastError();
  // A device-to-device copy: enough waves for every group of rows at once.
  hipLaunchKernelGGL(k_bank_patch, dim3((unsigned)ceil_div(active_cap, kGroup * kBankWaves)),
                     dim3(64 * kBankWaves), 0,
                     (hipStream_t)stream, (const uint4*)prev_slot, prev_active, prev_n,
                     next_active, next_n, active_cap, (int)(row_bytes / 16), (uint4*)next_slot);
  return hipGetLastError() == hipSuccess ? PFC_OK : PFC_ERR_HIP;
}

int pfc_bank_writeback(const void* slot, const int32_t* active, const int32_t* n_active,
                       const int32_t* next_active, const int32_t* next_n, int64_t active_cap,
                       int64_t row_bytes, int64_t C, void* bank, int32_t* bank_version,
                       int32_t version, void* stream) {
  if (!slot || !active || !n_active || !bank) return PFC_ERR_INVALID_ARG;
  if ((next_active == nullptr) != (next_n == nullptr)) return PFC_ERR_INVALID_ARG;
  if (C < 1 || C > PFC_MAX_CLASSES) return PFC_ERR_INVALID_ARG;
  const int st = common_checks(row_bytes, active_cap);
  if (st != PFC_OK) return st;
  const int dv = device_present();
  if (dv != PFC_OK) return dv;
  if (!device_accessible(bank) || !device_accessible(slot)) return PFC_ERR_INVALID_ARG;
  if (bank_version && !device_accessible(bank_version)) return PFC_ERR_INVALID_ARG;
  (void)hipGetLastError();
  hipLaunchKernelGGL(k_bank_writeback, dim3(grid_of(active_cap)), dim3(64 * kBankWaves), 0,
                     (hipStream_t)stream, (const uint4*)slot, active, n_active, next_active,
                     next_n, active_cap,
                     (int)(row_bytes / 16), C, (uint4*)bank, bank_version, version);
  return hipGetLastError() == hipSuccess ? PFC_OK : PFC_ERR_HIP;
}

}  // extern "C"
