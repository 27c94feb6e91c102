// wave_sort.h -- candidates in the result order (score descending, then id
// ascending) sorted and merged across the 64 lanes of a wave with bitonic
// networks over lane shuffles.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sieve {
namespace {

struct Cand {
  float s;
  long long id;
  int rank;  // carried only by the calibration variant of the top-k
};

__device__ __forceinline__ bool better(const Cand& a, const Cand& b) {
  return a.s > b.s || (a.s == b.s && a.id < b.id);
}

template <bool kRank>
__device__ __forceinline__ Cand shfl_xor_cand(const Cand& c, int m) {
  Cand o;
  o.s = __shfl_xor(c.s, m);
  const int lo = __shfl_xor((int)(c.id & 0xffffffffll), m);
  const int hi = __shfl_xor((int)(c.id >> 32), m);
  o.id = ((long long)hi << 32) | (unsigned int)lo;
  o.rank = kRank ? __shfl_xor(c.rank, m) : 0;
  return o;
}

template <bool kRank>
__device__ __forceinline__ Cand shfl_cand(const Cand& c, int src) {
  Cand o;
  o.s = __shfl(c.s, src);
  const int lo = __shfl((int)(c.id & 0xffffffffll), src);
  const int hi = __shfl((int)(c.id >> 32), src);
  o.id = ((long long)hi << 32) | (unsigned int)lo;
  o.rank = kRank ? __shfl(c.rank, src) : 0;
  return o;
}

// Sort 64 lane-held candidates, best first.
template <bool kRank>
__device__ __forceinline__ Cand wave_sort_desc(Cand v, int lane) {
#pragma unroll
  for (int k = 2; k <= 64; k <<= 1) {
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1) {
      const Cand o = shfl_xor_cand<kRank>(v, j);
      const bool lower = (lane & j) == 0;
      const bool desc = (lane & k) == 0;  // final stage: whole wave descending
      const bool keep_better = (lower == desc);
      const bool ob = better(o, v);
      if (keep_better ? ob : !ob) v = o;
    }
  }
  return v;
}

// Sort a bitonic 64-sequence, best first.
template <bool kRank>
__device__ __forceinline__ Cand wave_merge_desc(Cand v, int lane) {
#pragma unroll
  for (int j = 32; j > 0; j >>= 1) {
    const Cand o = shfl_xor_cand<kRank>(v, j);
    const bool lower = (lane & j) == 0;
    const bool ob = better(o, v);
    if (lower ? ob : !ob) v = o;
  }
  return v;
}

}  // namespace
}  // namespace sieve
