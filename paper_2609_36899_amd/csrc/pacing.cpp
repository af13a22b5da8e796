#include "pacing.h"

#include <algorithm>

namespace pdec {

void pacing_plan(int64_t headroom, int64_t h_min, int64_t delta,
                 const std::vector<PacingResident>& active,
                 const std::vector<PacingPending>& pending, std::vector<int32_t>* evicted,
                 std::vector<int32_t>* placed) {
  evicted->clear();
  placed->clear();
  int64_t h = headroom;
  // Phase 1: longest residents first while below the floor.
  std::vector<PacingResident> res(active);
  std::sort(res.begin(), res.end(), [](const PacingResident& a, const PacingResident& b) {
    return a.length != b.length ? a.length > b.length : a.id < b.id;
  });
  std::vector<PacingPending> wait(pending);
  size_t k = 0;
  while (h < h_min && k < res.size()) {
    h += res[k].held_tokens;
    evicted->push_back(res[k].id);
    wait.push_back({res[k].id, res[k].length});
    ++k;
  }
  int64_t n_active = (int64_t)(res.size() - k);
  // Phase 2: shortest pending first, under the placement threshold.
  std::sort(wait.begin(), wait.end(), [](const PacingPending& a, const PacingPending& b) {
    return a.length != b.length ? a.length < b.length : a.id < b.id;
  });
  for (const PacingPending& r : wait) {
    const int64_t foot = ((int64_t)r.length + 15) / 16 * 16;
    const int64_t after = h - foot;
    if (after >= h_min + (n_active + 1) * delta) {
      h = after;
      ++n_active;
      placed->push_back(r.id);
    }
  }
}

}  // namespace pdec
