// DN selection of Eq. 11 (Section 4.4, system monitoring and network
// selection): the cheapest DN, by its table cost, that meets the latency,
// memory, accuracy and power bounds.  Host only.
#include <math.h>

#include "../../include/elasto.h"
#include "layout.h"

using namespace elasto;

extern "C" elasto_status_t elasto_select_mode(const elasto_dn_lut_t* lut, double max_latency_ms,
                                              double max_memory_bytes, double min_accuracy,
                                              double max_power_w, int32_t* mode) {
  if (!lut || !mode) return fail(ELASTO_ERR_INVALID_ARG, "NULL argument");
  if (lut->num_modes < 1) return fail(ELASTO_ERR_INVALID_ARG, "num_modes must be >= 1");
  if (!lut->flops || !lut->latency_ms || !lut->memory_bytes)
    return fail(ELASTO_ERR_INVALID_ARG, "flops, latency_ms and memory_bytes are required");
  if (isnan(max_latency_ms) || isnan(max_memory_bytes) || isnan(min_accuracy) || isnan(max_power_w))
    return fail(ELASTO_ERR_INVALID_ARG, "NaN bound");
  if (!lut->accuracy && min_accuracy != -INFINITY)
    return fail(ELASTO_ERR_INVALID_ARG, "min_accuracy needs accuracy data in the table");
  const int n = lut->num_modes;
  for (int k = 0; k < n; ++k) {
    if (isnan(lut->flops[k]) || isnan(lut->latency_ms[k]) || isnan(lut->memory_bytes[k]) ||
        (lut->accuracy && isnan(lut->accuracy[k])) || (lut->power_w && isnan(lut->power_w[k])))
      return fail(ELASTO_ERR_INVALID_ARG, "NaN entry for mode %d", k);
  }
  int best = -1;
  for (int k = 0; k < n; ++k) {
    if (!(lut->latency_ms[k] <= max_latency_ms)) continue;
    if (!(lut->memory_bytes[k] <= max_memory_bytes)) continue;
    if (lut->accuracy && !(lut->accuracy[k] >= min_accuracy)) continue;
    if (lut->power_w && !(lut->power_w[k] <= max_power_w)) continue;
    if (best < 0 || lut->flops[k] < lut->flops[best]) best = k;
  }
  *mode = best;
  if (best < 0) return fail(ELASTO_ERR_INFEASIBLE, "no DN meets the bounds");
  clear_error();
  return ELASTO_OK;
}
