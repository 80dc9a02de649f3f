// Measurement hook of libpfc: HIP events around the launches of one kernel id.
#include <vector>

#include "pfc.h"
#include "pfc_internal.h"

namespace pfc {
namespace {

struct Timing {
  int kernel = -1;
  int max_launches = 0;
  int recorded = 0;
  bool open = false;  // a start event was recorded without its stop yet
  std::vector<hipEvent_t> start, stop;
};

Timing g_timing;

void release() {
  for (hipEvent_t e : g_timing.start) (void)hipEventDestroy(e);
  for (hipEvent_t e : g_timing.stop) (void)hipEventDestroy(e);
  g_timing = Timing{};
}

}  // namespace

void timing_start(int kernel, hipStream_t stream) {
  if (kernel != g_timing.kernel || g_timing.recorded >= g_timing.max_launches) return;
  if (hipEventRecord(g_timing.start[g_timing.recorded], stream) == hipSuccess) g_timing.open = true;
}

void timing_stop(int kernel, hipStream_t stream) {
  if (kernel != g_timing.kernel || !g_timing.open) return;
  if (hipEventRecord(g_timing.stop[g_timing.recorded], stream) == hipSuccess) ++g_timing.recorded;
  g_timing.open = false;
}

}  // namespace pfc

using namespace pfc;

extern "C" int pfc_timing_begin(int kernel, int max_launches) {
  if (kernel < 0 || kernel >= PFC_K_COUNT || max_launches < 1 || max_launches > 65536)
    return PFC_ERR_INVALID_ARG;
  release();
  for (int i = 0; i < max_launches; ++i) {
    hipEvent_t a, b;
    if (hipEventCreate(&a) != hipSuccess) {
      release();
      return PFC_ERR_HIP;
    }
    if (hipEventCreate(&b) != hipSuccess) {
      (void)hipEventDestroy(a);
      release();
      return PFC_ERR_HIP;
    }
    g_timing.start.push_back(a);
    g_timing.stop.push_back(b);
  }
  g_timing.kernel = kernel;
  g_timing.max_launches = max_launches;
  return PFC_OK;
}

extern "C" int pfc_timing_end(double* total_ms, int* launches) {
  if (!total_ms || !launches || g_timing.kernel < 0) return PFC_ERR_INVALID_ARG;
  double sum = 0.0;
  int st = PFC_OK;
  for (int i = 0; i < g_timing.recorded; ++i) {
    float ms = 0.0f;
    if (hipEventSynchronize(g_timing.stop[i]) != hipSuccess ||
        hipEventElapsedTime(&ms, g_timing.start[i], g_timing.stop[i]) != hipSuccess) {
      st = PFC_ERR_HIP;
      break;
    }
    sum += ms;
  }
  *total_ms = sum;
  *launches = g_timing.recorded;
  release();
  return st;
}
