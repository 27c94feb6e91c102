// topk.hip -- the final MergeTopK of Algorithm 1: every qualifying candidate
// a query met during the search is merged into its top-k, score descending
// then id ascending.  As in the paper, local results only accumulate during
// the search and are merged once at the end; the stop rule never looks at
// them.
//
// The candidate pool is unordered (appends from many tiles).  It is grouped
// by query with a counting sort (the per-query counts come from the scan's
// appends, then an exclusive scan and a scatter), and each query's segment is
// reduced by one wave64 that keeps its running top-64 in registers, one
// candidate per lane, merging 64 new candidates at a time with bitonic
// sorting networks over lane shuffles.  The total order makes the result
// independent of the pool's order.
#include "sieve_internal.h"
#include "wave_sort.h"

namespace sieve {
namespace {

constexpr int kScanBlock = 1024;
constexpr int kScanPer = 4;
constexpr int kScanTile = kScanBlock * kScanPer;

// In-block exclusive scan of kScanTile values starting at base, in 64-bit
// sums (a search may write more than 2^31 pool entries); returns the block
// total through *total.
template <typename TIn>
__device__ void block_scan_tile(const TIn* in, int64_t* out, int64_t* out2, int64_t n,
                                int64_t base, int64_t add, int64_t* total) {
  __shared__ int64_t s[kScanBlock];
  const int t = threadIdx.x;
  int64_t v[kScanPer];
  int64_t sum = 0;
  for (int e = 0; e < kScanPer; ++e) {
    const int64_t i = base + (int64_t)t * kScanPer + e;
    v[e] = i < n ? (int64_t)in[i] : 0;
    sum += v[e];
  }
  s[t] = sum;
  __syncthreads();
  for (int off = 1; off < kScanBlock; off <<= 1) {
    const int64_t x = t >= off ? s[t - off] : 0;
    __syncthreads();
    s[t] += x;
    __syncthreads();
  }
  int64_t run = s[t] - sum + add;
  if (out) {
    for (int e = 0; e < kScanPer; ++e) {
      const int64_t i = base + (int64_t)t * kScanPer + e;
      if (i < n) {
        out[i] = run;
        if (out2) out2[i] = run;
      }
      run += v[e];
    }
  }
  if (total && t == kScanBlock - 1) *total = s[t];
  __syncthreads();
}

__global__ __launch_bounds__(kScanBlock) void scan_partials_kernel(const int32_t* in, int64_t n,
                                                                  int64_t* partial) {
  block_scan_tile(in, nullptr, nullptr, n, (int64_t)blockIdx.x * kScanTile, 0,
                  &partial[blockIdx.x]);
}

__global__ __launch_bounds__(kScanBlock) void scan_partials_top_kernel(int64_t* partial,
                                                                      int32_t nparts) {
  // nparts <= kScanTile: exclusive scan in place
  __shared__ int64_t tot;
  block_scan_tile(partial, partial, nullptr, nparts, 0, 0, &tot);
}

__global__ __launch_bounds__(kScanBlock) void scan_apply_kernel(const int32_t* in, int64_t n,
                                                               const int64_t* partial,
                                                               int64_t* out, int64_t* out2) {
  block_scan_tile(in, out, out2, n, (int64_t)blockIdx.x * kScanTile, partial[blockIdx.x],
                  nullptr);
}

// Small inputs (a few tiles): one work-group scans the tiles in order with a
// running carry, in one launch instead of three.
constexpr int kScanSingleTiles = 16;

__global__ __launch_bounds__(kScanBlock) void scan_single_kernel(const int32_t* in, int64_t n,
                                                                int64_t* out, int64_t* out2) {
  __shared__ int64_t tot;
  int64_t carry = 0;
  for (int64_t base = 0; base < n; base += kScanTile) {
    block_scan_tile(in, out, out2, n, base, carry, &tot);  // ends with a barrier
    carry += tot;
    __syncthreads();  // every thread has read tot before the next tile writes it
  }
}

// The claims are aggregated per wave: one atomic per distinct query among the
// wave's 64 entries (a tile appends the candidates of a few queries row after
// row, so neighbouring entries mostly share queries, and one-address atomics
// serialise).  The order inside a query's segment is free: the top-k merge
// uses a total order.  Grid-stride over the pool in whole work-groups: a
// dispatch holds at most 2^32 work-items, fewer than a large pool's entries.
__global__ __launch_bounds__(256) void pool_scatter_kernel(const Hit* __restrict__ pool, int64_t n,
                                                           int64_t* __restrict__ cursor,
                                                           Hit* __restrict__ sorted,
                                                           int32_t qmask) {
  const int lane = threadIdx.x & 63;
  for (int64_t b0 = (int64_t)blockIdx.x * blockDim.x; b0 < n;
       b0 += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = b0 + threadIdx.x;
    Hit h = {-INFINITY, -1, -1};
    if (i < n) h = pool[i];
    const int q = h.q < 0 ? -1 : (h.q & qmask);  // -1: past the end
    // group the lanes by query (register work only), then every group's first
    // lane claims the group's slots, all groups at once
    unsigned long long todo = __ballot(q >= 0);
    int leader = lane, rank = 0, count = 0;
    while (todo) {  // wave-uniform
      const int first = __builtin_ctzll(todo);
      const int qf = __shfl(q, first);
      const unsigned long long same = __ballot(q == qf);
      if (q == qf) {
        leader = first;
        rank = __popcll(same & ((1ull << lane) - 1ull));
        count = __popcll(same);
      }
      todo &= ~same;
    }
    long long base = 0;
    if (q >= 0 && rank == 0)
      base = (long long)atomicAdd((unsigned long long*)&cursor[q], (unsigned long long)count);
    base = __shfl(base, leader);
    if (q >= 0) sorted[base + rank] = h;
  }
}

// One wave per query, grid-stride over the queries; each block adds its
// probe and candidate totals to the round counters once.  kRank: pool
// entries carry their rank (calibration search); out_rank receives it.
template <bool kRank>
__global__ __launch_bounds__(256) void topk_kernel(int64_t nq, int32_t k,
                                                   const Hit* __restrict__ sorted,
                                                   const int64_t* __restrict__ hoff,
                                                   const int32_t* __restrict__ hcount,
                                                   const int32_t* __restrict__ probes_src,
                                                   int32_t probes_const,
                                                   int64_t* __restrict__ out_ids,
                                                   float* __restrict__ out_scores,
                                                   int32_t* __restrict__ out_probes,
                                                   const int32_t* __restrict__ out_map,
                                                   int32_t* __restrict__ out_rank,
                                                   const int32_t* __restrict__ rank_limit,
                                                   RoundCounters* rc) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __shared__ unsigned long long s_probes[4], s_cands[4];
  unsigned long long probes = 0, cands = 0;
  const Cand none = {-INFINITY, 0x7fffffffffffffffll, -1};
  for (int64_t q = (int64_t)blockIdx.x * 4 + wave; q < nq; q += (int64_t)gridDim.x * 4) {
    const int m = hcount[q];
    const int64_t beg = m > 0 ? hoff[q] : 0;
    const int lim = rank_limit ? rank_limit[q] : 0x7fffffff;
    Cand top = none;
    for (int b = 0; b < m; b += 64) {
      Cand c = none;
      if (b + lane < m) {
        const Hit h = sorted[beg + b + lane];
        if (!rank_limit || (h.q >> kRankShift) < lim) {
          c.s = h.score;
          c.id = h.id;
          c.rank = kRank ? (h.q >> kRankShift) : 0;
        }
      }
      c = wave_sort_desc<kRank>(c, lane);
      if (b == 0) {
        top = c;
      } else {
        const Cand r = shfl_cand<kRank>(c, 63 - lane);  // reversed: top ++ reverse(c) is bitonic
        top = better(top, r) ? top : r;
        top = wave_merge_desc<kRank>(top, lane);
      }
    }
    const int64_t row = out_map ? (int64_t)out_map[q] : q;
    if (lane < k) {
      const bool real = top.id != none.id;
      out_ids[row * k + lane] = real ? (int64_t)top.id : -1;
      out_scores[row * k + lane] = real ? top.s : -INFINITY;
      if (kRank) out_rank[q * k + lane] = real ? top.rank : -1;
    }
    const int32_t p = probes_src ? probes_src[q] : probes_const;
    if (lane == 0) out_probes[row] = p;
    probes += (unsigned long long)p;
    cands += (unsigned long long)m;
  }
  if (lane == 0) {
    s_probes[wave] = probes;
    s_cands[wave] = cands;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    const int slot = blockIdx.x % kStatSlots;
    atomicAdd(&rc->probes[slot], s_probes[0] + s_probes[1] + s_probes[2] + s_probes[3]);
    atomicAdd(&rc->candidates[slot], s_cands[0] + s_cands[1] + s_cands[2] + s_cands[3]);
  }
}

// Multi-index merge: one wave per query takes the nshard per-index top-k
// lists (rows of sids / sscores, shard-major [nshard][nq][k], padded with
// id -1), keeps the best k in the same total order, and sums the per-index
// probe counts.
__global__ __launch_bounds__(256) void merge_shards_kernel(int64_t nq, int32_t k,
                                                           int32_t nshard,
                                                           const int64_t* __restrict__ sids,
                                                           const float* __restrict__ sscores,
                                                           const int32_t* __restrict__ sprobes,
                                                           int64_t* __restrict__ out_ids,
                                                           float* __restrict__ out_scores,
                                                           int32_t* __restrict__ out_probes) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const Cand none = {-INFINITY, 0x7fffffffffffffffll, -1};
  for (int64_t q = (int64_t)blockIdx.x * 4 + wave; q < nq; q += (int64_t)gridDim.x * 4) {
    const int m = nshard * k;  // candidates of this query, shard by shard
    Cand top = none;
    for (int b = 0; b < m; b += 64) {
      Cand c = none;
      const int j = b + lane;
      if (j < m) {
        const int sh = j / k, r = j - sh * k;
        const int64_t at = ((int64_t)sh * nq + q) * k + r;
        const int64_t id = sids[at];
        if (id >= 0) {
          c.s = sscores[at];
          c.id = id;
        }
      }
      c = wave_sort_desc<false>(c, lane);
      if (b == 0) {
        top = c;
      } else {
        const Cand rv = shfl_cand<false>(c, 63 - lane);
        top = better(top, rv) ? top : rv;
        top = wave_merge_desc<false>(top, lane);
      }
    }
    if (lane < k) {
      const bool real = top.id != none.id;
      out_ids[q * k + lane] = real ? (int64_t)top.id : -1;
      out_scores[q * k + lane] = real ? top.s : -INFINITY;
    }
    if (lane == 0) {
      int32_t p = 0;
      for (int sh = 0; sh < nshard; ++sh) p += sprobes[(int64_t)sh * nq + q];
      out_probes[q] = p;
    }
  }
}

}  // namespace

hipError_t launch_merge_shards(int64_t nq, int32_t k, int32_t nshard, const int64_t* sids,
                               const float* sscores, const int32_t* sprobes, int64_t* out_ids,
                               float* out_scores, int32_t* out_probes, hipStream_t s) {
  if (nq <= 0) return hipSuccess;
  const int64_t want = (nq + 3) / 4;
  const unsigned blocks = (unsigned)(want < 4096 ? want : 4096);
  hipLaunchKernelGGL(merge_shards_kernel, dim3(blocks), dim3(256), 0, s, nq, k, nshard, sids,
                     sscores, sprobes, out_ids, out_scores, out_probes);
  return hipGetLastError();
}

size_t exclusive_scan_tmp_elems(int64_t n) { return (size_t)((n + kScanTile - 1) / kScanTile) + 1; }

hipError_t launch_exclusive_scan(const int32_t* in, int64_t* out, int64_t* out_copy, int64_t n,
                                 int64_t* block_tmp, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t nb = (n + kScanTile - 1) / kScanTile;
  if (nb > kScanTile) return hipErrorInvalidValue;
  if (nb <= kScanSingleTiles) {
    hipLaunchKernelGGL(scan_single_kernel, dim3(1), dim3(kScanBlock), 0, s, in, n, out, out_copy);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(scan_partials_kernel, dim3((unsigned)nb), dim3(kScanBlock), 0, s, in, n,
                     block_tmp);
  hipLaunchKernelGGL(scan_partials_top_kernel, dim3(1), dim3(kScanBlock), 0, s, block_tmp,
                     (int32_t)nb);
  hipLaunchKernelGGL(scan_apply_kernel, dim3((unsigned)nb), dim3(kScanBlock), 0, s, in, n,
                     block_tmp, out, out_copy);
  return hipGetLastError();
}

hipError_t launch_pool_scatter(const Hit* pool, int64_t n, int64_t* cursor, Hit* sorted,
                               bool packed, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t want = (n + 255) / 256;
  const unsigned blocks = (unsigned)(want < (1 << 20) ? want : (1 << 20));
  hipLaunchKernelGGL(pool_scatter_kernel, dim3(blocks), dim3(256), 0, s, pool, n, cursor, sorted,
                     packed ? kQueryMask : (int32_t)0x7fffffff);
  return hipGetLastError();
}

hipError_t launch_topk(int64_t nq, int32_t k, const Hit* sorted, const int64_t* hoff,
                       const int32_t* hcount, const int32_t* probes_src, int32_t probes_const,
                       const int32_t* out_map, int64_t* out_ids, float* out_scores,
                       int32_t* out_probes, int32_t* out_rank, const int32_t* rank_limit,
                       RoundCounters* rc, hipStream_t s) {
  if (nq <= 0) return hipSuccess;
  const int64_t want = (nq + 3) / 4;
  const unsigned blocks = (unsigned)(want < 4096 ? want : 4096);
  if (out_rank)
    hipLaunchKernelGGL(topk_kernel<true>, dim3(blocks), dim3(256), 0, s, nq, k, sorted, hoff,
                       hcount, probes_src, probes_const, out_ids, out_scores, out_probes,
                       out_map, out_rank, rank_limit, rc);
  else
    hipLaunchKernelGGL(topk_kernel<false>, dim3(blocks), dim3(256), 0, s, nq, k, sorted, hoff,
                       hcount, probes_src, probes_const, out_ids, out_scores, out_probes,
                       out_map, nullptr, rank_limit, rc);
  return hipGetLastError();
}

}  // namespace sieve
