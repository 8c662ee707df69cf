// Event timing of kernel launches (gradlev_timing_* in gradlev.h).
#include <vector>

#include "../../include/gradlev.h"
#include "internal.hpp"

namespace gradlev {
namespace {

constexpr size_t kMaxPairs = 65536;

struct Family {
  std::vector<hipEvent_t> start, stop;  // event pool, grows on demand
  size_t used = 0;                      // pairs recorded since the last reset
  bool open = false;
  double ms = 0.0;                      // folded-in time of read pairs
  int64_t launches = 0;
};

unsigned g_mask = 0;  // bit f: family f is timed
Family g_fam[GRADLEV_K_COUNT];

void fold(Family& f) {
  for (size_t i = 0; i < f.used; ++i) {
    float ms = 0.f;
    if (hipEventSynchronize(f.stop[i]) == hipSuccess &&
        hipEventElapsedTime(&ms, f.start[i], f.stop[i]) == hipSuccess) {
      f.ms += ms;
      f.launches += 1;
    }
  }
  f.used = 0;
}

}  // namespace

void timing_begin(int family, hipStream_t s) {
  if (family < 0 || family >= GRADLEV_K_COUNT || !(g_mask & (1u << family))) return;
  Family& f = g_fam[family];
  if (f.used == kMaxPairs) {
    // Under stream capture the recorded events are graph nodes that have not
    // run yet: waiting on them would never return (or invalidate the
    // capture), so recording stops at the cap instead of folding.
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(s, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone) return;
    fold(f);
  }
  if (f.used == f.start.size()) {
    hipEvent_t a, b;
    if (hipEventCreate(&a) != hipSuccess) return;
    if (hipEventCreate(&b) != hipSuccess) {
      (void)hipEventDestroy(a);
      return;
    }
    f.start.push_back(a);
    f.stop.push_back(b);
  }
  if (hipEventRecord(f.start[f.used], s) == hipSuccess) f.open = true;
}

void timing_end(int family, hipStream_t s) {
  if (family < 0 || family >= GRADLEV_K_COUNT || !(g_mask & (1u << family))) return;
  Family& f = g_fam[family];
  if (!f.open) return;
  f.open = false;
  if (hipEventRecord(f.stop[f.used], s) == hipSuccess) f.used += 1;
}

}  // namespace gradlev

using namespace gradlev;

extern "C" {

int gradlev_timing_enable(int mask) {
  const int prev = (int)g_mask;
  g_mask = (unsigned)mask & ((1u << GRADLEV_K_COUNT) - 1u);
  return prev;
}

int gradlev_timing_reset(void) {
  for (Family& f : g_fam) {
    for (size_t i = 0; i < f.used; ++i) (void)hipEventSynchronize(f.stop[i]);
    f.used = 0;
    f.open = false;
    f.ms = 0.0;
    f.launches = 0;
  }
  return GRADLEV_OK;
}

int gradlev_timing_read(int family, double* ms, int64_t* launches) {
  if (family < 0 || family >= GRADLEV_K_COUNT || !ms || !launches) return GRADLEV_ERR_INVALID;
  Family& f = g_fam[family];
  fold(f);
  *ms = f.ms;
  *launches = f.launches;
  return GRADLEV_OK;
}

}  // extern "C"
