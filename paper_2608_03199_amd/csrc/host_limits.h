// host_limits.h -- pure host-side size rules of libsieve (no HIP), so that a
// plain C++ compiler can check them without a GPU.
#pragma once

#include <stdint.h>
#include <stdlib.h>

namespace sieve {

// The final merge groups the candidate pool by query with 64-bit per-query
// offsets (exclusive scan of the counts, scatter cursors, segment starts), so
// the limit on candidate slots is a sanity bound, 2^38, far more than device
// memory holds (the pool's allocation fails first).  knob: the value of an
// override (tests lower the limit to reach the error path without filling
// memory); null, empty or non-positive means no override.
inline int64_t pool_index_limit(const char* knob) {
  const int64_t hard = (int64_t)1 << 38;
  if (!knob || !*knob) return hard;
  const long long v = atoll(knob);
  return v > 0 && v < hard ? (int64_t)v : hard;
}

// Whether a search whose scans claimed `slots` pool slots can be merged.
inline bool pool_slots_fit(uint64_t slots, int64_t limit) {
  return limit >= 0 && slots <= (uint64_t)limit;
}

}  // namespace sieve
