// Internal, host only: choosing a GEMM / convolution tile plan (kernels.h,
// kTilePlans) for one call site of a forward by timing every plan once on
// the device.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <vector>

#include "kernels.h"

namespace elasto {

constexpr int kTuneReps = 5;         // timed launches per plan (the fastest counts)
constexpr int kTuneMinBatch = 32;    // elastic-CNN handles for fewer images are not tuned
constexpr float kTuneMargin = 0.99f; // another choice must beat the default by 1%

// Times `launch(plan)` for every tile plan: each once untimed, then
// kTuneReps rounds in which every plan is launched once between events on
// `s` (round-robin, so that clock drift does not favour one plan).  Stores
// in *plan the fastest, or 0 (the planner's own choice) unless another plan
// is faster by the margin.  launch returns hipErrorNotSupported for a plan
// that cannot run the site's arguments; any other error ends the tuning.
template <class F>
hipError_t time_plans(F&& launch, hipStream_t s, hipEvent_t e0, hipEvent_t e1, uint8_t* plan) {
  bool ok[kTilePlans];
  float t[kTilePlans];
  for (int c = 0; c < kTilePlans; ++c) {
    const hipError_t e = launch(c);
    if (e != hipSuccess && e != hipErrorNotSupported) return e;
    ok[c] = e == hipSuccess;
    t[c] = 0.0f;
  }
  for (int r = 0; r < kTuneReps; ++r)
    for (int c = 0; c < kTilePlans; ++c) {
      if (!ok[c]) continue;
      hipError_t e;
      if ((e = hipEventRecord(e0, s)) != hipSuccess || (e = launch(c)) != hipSuccess ||
          (e = hipEventRecord(e1, s)) != hipSuccess || (e = hipEventSynchronize(e1)) != hipSuccess)
        return e;
      float ms = 0.0f;
      if ((e = hipEventElapsedTime(&ms, e0, e1)) != hipSuccess) return e;
      t[c] = r == 0 ? ms : std::min(t[c], ms);
    }
  int best = 0;
  for (int c = 1; c < kTilePlans; ++c)
    if (ok[c] && t[c] < t[best]) best = c;
  *plan = (uint8_t)(best != 0 && t[best] < kTuneMargin * t[0] ? best : 0);
  return hipSuccess;
}

// What a handle's create-time tuning chose: a tile plan per (mode, GEMM
// site) for whole forwards and for half-batch parts, and per mode whether to
// split.  Choices are kept per process under a key made of everything that
// sets the shapes of the forward's GEMMs (model configuration, DN widths,
// max_batch, device), so that handles of the same shapes take the same
// choices (and, where plans differ in rounding, give the same bits) and
// only the first of them pays for the timing.
struct TunedPlans {
  std::vector<uint8_t> plans, plans_half, split;
};
bool tuned_lookup(const std::vector<int64_t>& key, TunedPlans* out);
void tuned_store(const std::vector<int64_t>& key, const TunedPlans& t);

}  // namespace elasto
