// pfc_sample_noalloc: pfc_sample for callers that cannot allocate device
// memory.  The sampler's scratch (positive bitmap, key-digit histogram and
// digits, threshold candidates and their keys, compaction counts) lives in a
// file-scope device array instead of a caller workspace.  Declaration and
// contract in include/pfc.h.
#include <math.h>

#include <mutex>

#include "pfc.h"
#include "pfc_internal.h"

namespace pfc {
namespace {

// Largest sampler prefix of the workspace layout (ws_layout) for
// C <= PFC_NOALLOC_MAX_CLASSES, rounded up: bitmap C/8 + histogram 16 KiB +
// state + digits 2C + candidate keys 8C + four group arrays (20.3 MiB at
// C = 2^21).
constexpr size_t kScratchBytes = (size_t)21 << 20;

// One copy per device; every call on a device shares it.
__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mutex;
void* g_ptr[kMaxDevices] = {};

// Device address of this device's copy of `scratch`, looked up on the first
// call on the device (with it current) and kept.  NULL on failure.
void* scratch_ptr(int dev) {
  std::lock_guard<std::mutex> lock(g_mutex);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
    g_ptr[dev] = p;
  }
  return g_ptr[dev];
}

}  // namespace
}  // namespace pfc

using namespace pfc;

extern "C" int pfc_sample_noalloc(const int64_t* labels, int64_t B, int64_t C,
                                  int64_t class_offset, double r, uint64_t seed, int32_t* active,
                                  int64_t active_cap, int32_t* n_active, int32_t* labels_mapped,
                                  void* stream) {
  if (!labels || !active || !n_active || !labels_mapped) return PFC_ERR_INVALID_ARG;
  if (B < 1 || B > PFC_MAX_BATCH || C < 1 || C > PFC_MAX_CLASSES) return PFC_ERR_INVALID_ARG;
  if (class_offset < 0 || class_offset > ((int64_t)1 << 62) - C) return PFC_ERR_INVALID_ARG;
  if (!(isfinite(r) && r > 0.0 && r <= 1.0)) return PFC_ERR_INVALID_ARG;
  if (C > PFC_NOALLOC_MAX_CLASSES) return PFC_ERR_SCRATCH;
  if (active_cap < cap_of(B, C, r)) return PFC_ERR_CAPACITY;
  const WsLayout L = ws_layout(B, 8, C, active_cap, PFC_F32);
  if (L.sample_bytes > kScratchBytes) return PFC_ERR_SCRATCH;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return PFC_ERR_HIP;
  void* base = scratch_ptr(dev);
  if (!base) return PFC_ERR_HIP;
  (void)hipGetLastError();
  const hipError_t e = launch_sample(labels, B, C, class_offset, budget_of(r, C), seed, L.top_bits,
                                     L.n_groups, sample_ws(base, L), active, active_cap, n_active,
                                     labels_mapped, (hipStream_t)stream);
  return e == hipSuccess ? PFC_OK : PFC_ERR_HIP;
}
