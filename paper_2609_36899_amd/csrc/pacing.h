// Headroom pacing on one worker (host only): which residents to evict and
// which pending trajectories to place (Design, "Separating Departure from
// Placement", pacing thresholds; Alg. pacing, restricted to one worker).
#pragma once

#include <cstdint>
#include <vector>

namespace pdec {

struct PacingResident {
  int32_t id;
  int32_t length;       // tokens cached
  int64_t held_tokens;  // pages held (reserve included) x 16
};

struct PacingPending {
  int32_t id;
  int32_t length;
};

// Phase 1: while headroom < h_min and residents remain, evict the longest
// (ties: lower id).  Phase 2: pending in ascending length (ties: lower id);
// place r when headroom - footprint(r) >= h_min + (|A| + 1) * delta, with
// footprint(r) = ceil(length / 16) * 16.  Evicted residents join the pending
// set before Phase 2.
void pacing_plan(int64_t headroom, int64_t h_min, int64_t delta,
                 const std::vector<PacingResident>& active,
                 const std::vector<PacingPending>& pending, std::vector<int32_t>* evicted,
                 std::vector<int32_t>* placed);

}  // namespace pdec
