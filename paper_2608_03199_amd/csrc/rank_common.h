// rank_common.h -- pieces shared by the centroid-ranking kernels: the
// order-preserving integer image of fp32 scores, fp64 re-scoring of screen
// near-ties, and the per-wave finish that turns a candidate set into the
// exact order (Sec. 4.1's per-query partition order P_i).
//
// Exactness argument: the fp32 screen score s32[c] of centroid c is within
// delta = 2 (d + 2) 2^-24 |q| max_c |c| of its fp64 score s64[c] (the fp64
// sum of exact products in dimension order).  If v is the n-th largest
// screen score, every centroid of the fp64 top-n has s32 >= v - 2 delta, so
// any candidate set holding all centroids with s32 >= v - 2 delta holds the
// fp64 top-n.  Sorted by (s32 desc, c asc), candidates whose successive fp32
// gaps are all <= 2 delta form runs; a gap > 2 delta orders two centroids the
// same way in fp64, so only members of multi-element runs need fp64 scores,
// which then order each run by (s64 desc, c asc).
#pragma once

#include "sieve_internal.h"

namespace sieve {
namespace {

__device__ __forceinline__ uint32_t f2key(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float key2f(uint32_t k) {
  const uint32_t u = (k & 0x80000000u) ? (k & 0x7fffffffu) : ~k;
  return __uint_as_float(u);
}

template <int DT>
__device__ __forceinline__ double load_elem(const void* base, int64_t i) {
  if constexpr (DT == SIEVE_F32)
    return (double)((const float*)base)[i];
  else
    return (double)((const _Float16*)base)[i];
}

// fp64 inner product of query row q and centroid row c (global memory) by
// one wave: lane l sums dimensions l, l+64, ... in order, then the 64
// partial sums are added as a tree.  Its distance to the dimension-ordered
// sequential fp64 sum is at most (d + ceil(d/64) + 6) 2^-53 sum_t |q_t c_t|.
template <int DT>
__device__ __forceinline__ double wave_dot_fp64(const void* __restrict__ queries, int64_t q,
                                                const void* __restrict__ centroids, int c, int d) {
  const int lane = threadIdx.x & 63;
  double s = 0.0;
  for (int t0 = 0; t0 < d; t0 += 256) {
    double qv[4], cv[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int t = t0 + lane + 64 * k;
      const int tc = t < d ? t : d - 1;  // clamped: the loads issue together
      qv[k] = load_elem<DT>(queries, q * d + tc);
      cv[k] = load_elem<DT>(centroids, (int64_t)c * d + tc);
    }
#pragma unroll
    for (int k = 0; k < 4; ++k)
      if (t0 + lane + 64 * k < d) s += qv[k] * cv[k];
  }
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
  return s;
}

// The dimension-ordered sequential fp64 sum (what the order is defined by).
template <int DT>
__device__ __noinline__ double seq_dot_fp64(const void* __restrict__ queries, int64_t q,
                                            const void* __restrict__ centroids, int c, int d) {
  double s = 0.0;
  for (int t = 0; t < d; ++t)
    s += load_elem<DT>(queries, q * d + t) * load_elem<DT>(centroids, (int64_t)c * d + t);
  return s;
}

// Order candidates [0, m) already sorted by fp32 screen key: inside each run
// of near-ties (link[i]: the gap to i+1 is within the screen bound) sort by
// fp64 score desc, centroid asc.  Tier 1 scores come from wave_dot_fp64;
// a run whose tier-1 neighbours are within 2 * bound64 is re-scored with the
// exact sequential sum before its final sort.  NW waves of the calling block
// (waves w0..w0+NW-1) share the work; the caller synchronises between calls
// of the three steps.
template <int DT>
__device__ __forceinline__ void refine_members(unsigned long long* ck, double* cs,
                                               const uint8_t* link, int m,
                                               const void* queries, int64_t qg,
                                               const void* centroids, int d, int wave, int nwaves) {
  for (int i = wave; i < m; i += nwaves) {
    const bool member = link[i] || (i > 0 && link[i - 1]);  // wave-uniform
    if (member) {
      const double v = wave_dot_fp64<DT>(queries, qg, centroids, (int)(ck[i] & 0xffffffffu), d);
      if ((threadIdx.x & 63) == 0) cs[i] = v;
    }
  }
}

__device__ __forceinline__ void sort_run(unsigned long long* ck, double* cs, int i, int e) {
  for (int x = i + 1; x <= e; ++x) {
    const unsigned long long kv = ck[x];
    const double sx = cs[x];
    const unsigned cx = (unsigned)(kv & 0xffffffffu);
    int y = x - 1;
    while (y >= i) {
      const unsigned cy = (unsigned)(ck[y] & 0xffffffffu);
      const bool before = (sx > cs[y]) || (sx == cs[y] && cx < cy);
      if (!before) break;
      ck[y + 1] = ck[y];
      cs[y + 1] = cs[y];
      --y;
    }
    ck[y + 1] = kv;
    cs[y + 1] = sx;
  }
}

// One thread per run start: sort by tier-1 score; if two neighbours are
// within gap64, re-score the whole run exactly and sort again.
template <int DT>
__device__ __forceinline__ void order_runs(unsigned long long* ck, double* cs, const uint8_t* link,
                                           int m, const void* queries, int64_t qg,
                                           const void* centroids, int d, double gap64, int tid,
                                           int nthreads) {
  for (int i = tid; i < m; i += nthreads) {
    if (link[i] && (i == 0 || !link[i - 1])) {
      int e = i;
      while (link[e]) ++e;  // run is [i, e]
      sort_run(ck, cs, i, e);
      bool close = false;
      for (int x = i; x < e; ++x) close |= (cs[x] - cs[x + 1]) <= gap64;
      if (close) {
        for (int x = i; x <= e; ++x)
          cs[x] = seq_dot_fp64<DT>(queries, qg, centroids, (int)(ck[x] & 0xffffffffu), d);
        sort_run(ck, cs, i, e);
      }
    }
  }
}


// Wave-level fence: orders this wave's LDS writes before its later LDS reads
// (other lanes read what a lane wrote; no other wave shares the region).
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Bytes of one wave's LDS region in the wave-per-query kernel.
__host__ __device__ inline int wave_region_bytes(int capw) {
  return capw * 8 * 2 + capw * 8 + ((capw + 15) & ~15);
}

// Steps shared by the per-wave selectors: given this wave's m distinct
// candidate keys in ck[0, m) (key = ~f2key(s32) << 32 | centroid), sort them,
// link near-tie runs (gap <= 2 delta), re-score run members in fp64, order
// each run, and write the first n centroids to Prow.  LDS regions ck, out,
// cs, link belong to this wave alone.
template <int DT>
__device__ __forceinline__ void finish_candidates_wave(
    unsigned long long* ck, unsigned long long* out, double* cs, uint8_t* link, int m, int n,
    double gap, const void* __restrict__ queries, int64_t qg, const void* __restrict__ centroids,
    int d, double qn, double cmax, int32_t* __restrict__ Prow) {
  const int lane = threadIdx.x & 63;
  // 4a. rank by counting (keys are distinct): position = number of smaller keys
  for (int i = lane; i < m; i += 64) {
    const unsigned long long ki = ck[i];
    int pos = 0;
#pragma unroll 8
    for (int j = 0; j < m; ++j) pos += ck[j] < ki ? 1 : 0;
    out[pos] = ki;
  }
  wave_sync();
  // 4b. runs of near-ties
  for (int i = lane; i < m; i += 64) {
    bool l = false;
    if (i + 1 < m) {
      const double x = (double)key2f(~(uint32_t)(out[i] >> 32));
      const double y = (double)key2f(~(uint32_t)(out[i + 1] >> 32));
      l = (x - y) <= gap;
    }
    link[i] = l ? 1 : 0;
  }
  wave_sync();
  // Only positions [0, n) are written, and a run only reorders its own
  // members: runs that start at or past n cannot change them.  The candidates
  // that matter end with the run holding position n - 1.
  int me = n < m ? n : m;
  while (me < m && link[me - 1]) ++me;
  // 4c. fp64 scores of run members (this wave alone)
  refine_members<DT>(out, cs, link, me, queries, qg, centroids, d, 0, 1);
  wave_sync();
  // 4d. order inside each run (exact sequential sums where tier 1 is too close)
  {
    const double gap64 =
        2.0 * 2.0 * (double)(d + (d + 63) / 64 + 6) * 1.1102230246251565e-16 * qn * cmax + 1e-300;
    order_runs<DT>(out, cs, link, me, queries, qg, centroids, d, gap64, lane, 64);
  }
  wave_sync();
  for (int r = lane; r < n; r += 64) Prow[r] = (int32_t)(out[r] & 0xffffffffu);
}

}  // namespace
}  // namespace sieve
