// Process-wide store of the tile plans and stream splits chosen by the
// handles' create-time tuning (plans.h).
#include "plans.h"

#include <map>
#include <mutex>

namespace elasto {
namespace {
std::mutex g_mu;
std::map<std::vector<int64_t>, TunedPlans>& store() {
  static std::map<std::vector<int64_t>, TunedPlans> m;
  return m;
}
}  // namespace

bool tuned_lookup(const std::vector<int64_t>& key, TunedPlans* out) {
  std::lock_guard<std::mutex> lock(g_mu);
  const auto it = store().find(key);
  if (it == store().end()) return false;
  *out = it->second;
  return true;
}

void tuned_store(const std::vector<int64_t>& key, const TunedPlans& t) {
  std::lock_guard<std::mutex> lock(g_mu);
  store()[key] = t;
}

}  // namespace elasto
