// Internal, host only: choosing a GEMM / convolution tile plan (kernels.h,
// kTilePlans) for one call site of a forward by timing every plan once on
// the device.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "kernels.h"

namespace elasto {

constexpr int kTuneReps = 3;         // timed launches per plan (the fastest counts)
constexpr int kTuneMinBatch = 32;    // handles for fewer images are not tuned
constexpr float kTuneMargin = 0.97f; // another plan must beat the planner's by 3%

// Times `launch(plan)` for every tile plan (each once untimed, then
// kTuneReps times between events on `s`) and stores in *plan the fastest,
// or 0 (the planner's own choice) unless another plan is faster by the
// margin.  launch returns hipErrorNotSupported for a plan that cannot run
// the site's arguments; any other error ends the tuning.
template <class F>
hipError_t time_plans(F&& launch, hipStream_t s, hipEvent_t e0, hipEvent_t e1, uint8_t* plan) {
  float t0 = 0.0f, best_t = 0.0f;
  int best = 0;
  for (int c = 0; c < kTilePlans; ++c) {
    hipError_t e = launch(c);
    if (e == hipErrorNotSupported) continue;
    if (e != hipSuccess) return e;
    float t = 0.0f;
    for (int r = 0; r < kTuneReps; ++r) {
      if ((e = hipEventRecord(e0, s)) != hipSuccess || (e = launch(c)) != hipSuccess ||
          (e = hipEventRecord(e1, s)) != hipSuccess || (e = hipEventSynchronize(e1)) != hipSuccess)
        return e;
      float ms = 0.0f;
      if ((e = hipEventElapsedTime(&ms, e0, e1)) != hipSuccess) return e;
      t = r == 0 ? ms : std::min(t, ms);
    }
    if (c == 0) {
      t0 = best_t = t;
    } else if (t < best_t) {
      best_t = t;
      best = c;
    }
  }
  *plan = (uint8_t)(best != 0 && best_t < kTuneMargin * t0 ? best : 0);
  return hipSuccess;
}

}  // namespace elasto
