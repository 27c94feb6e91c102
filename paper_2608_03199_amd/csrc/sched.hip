// sched.hip -- device-side partition-major scheduling and the stop-rule
// update.
//
// Continuous batching (Sec. 4.2, Algorithm 1) regroups ready items (q_i, j)
// by partition p_{i,j}.  On the GPU this runs as bulk-synchronous rounds: all
// items ready at the start of a round are histogrammed by partition (the
// histogram is taken when the items are emitted), turned into partition-major
// buckets by an exclusive scan and a scatter, and cut into scan tiles.  The
// FIFO order and the 16K microbatch cap of the paper only decide timing, so
// a round simply dispatches every ready group at once.
//
// After a round's scan, the update applies the stop rule to every query:
//   lookahead (Sec. 4.3, Algorithm 2): a hit at rank j extends the stop line
//     s <- max(s, min(j + W, n)); the newly committed ranks are emitted at
//     once.  Only the largest hit rank of the round matters, because the
//     updates combine through max.
//   basic (Algorithm 1): one rank per round; stale resets on a hit and grows
//     on an empty probe; the next rank is emitted while stale < W and
//     next <= n.
// Ranks are ordered lazily: P holds the first have[q] ranks of query q.  An
// update that commits a rank at or beyond have[q] emits what it can, lists
// the query, and the host extends the listed queries' rank prefix before the
// next round (emit_pending then emits the rest).  Only the round in which an
// item is dispatched changes, which the result does not depend on (Sec. 4.3).
#include "sieve_internal.h"

namespace sieve {
namespace {

constexpr int kThreads = 256;
constexpr int kInitThreads = 1024;
constexpr int kInitBlocksMax = 512;

inline int blocks_for(int64_t n, int per = kThreads) {
  int64_t b = (n + per - 1) / per;
  return (int)(b < 1 ? 1 : b);
}

// Initial admission: ranks [0, s0) of every query of the chunk [q0, q0+nqc).
// mode 0: lookahead (stop line s0), 1: basic (next = 0, stale = 0), 2: fixed.
// The partition histogram of the items is taken in LDS (nlist bins) and
// added to the global one once per work-group: the first ranks of many
// queries fall on the same few partitions, and global atomics on one
// address serialise.
__global__ __launch_bounds__(kInitThreads) void emit_initial_kernel(
    const int32_t* __restrict__ P, int32_t n, int64_t nqc, int32_t q0, int32_t s0, int32_t mode,
    Item* __restrict__ items, int64_t item_cap, int32_t* __restrict__ cnt, int32_t nlist,
    int32_t* __restrict__ state_a, int32_t* __restrict__ state_b, int32_t* __restrict__ lmax) {
  extern __shared__ int32_t s_hist[];  // [nlist]
  for (int i = threadIdx.x; i < nlist; i += blockDim.x) s_hist[i] = 0;
  __syncthreads();
  for (int64_t ql = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; ql < nqc;
       ql += (int64_t)gridDim.x * blockDim.x) {
    const int32_t q = q0 + (int32_t)ql;
    for (int j = 0; j < s0; ++j) {
      Item it;
      it.q = q;
      it.rank = j;
      if (ql * s0 + j < item_cap) items[ql * s0 + j] = it;
      atomicAdd(&s_hist[P[ql * n + j]], 1);
    }
    if (mode == 0) {
      state_a[q] = s0;
      state_b[q] = s0;  // ranks issued (speculative issue)
      lmax[q] = 0;
    } else if (mode == 1) {
      state_a[q] = 0;  // next (0-based rank in flight)
      state_b[q] = 0;  // stale
      lmax[q] = 0;
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < nlist; i += blockDim.x)
    if (s_hist[i]) atomicAdd(&cnt[i], s_hist[i]);
}

// One work-group: exclusive scans over the lists of the item histogram and
// of the per-list tile counts; resets the round's counters.
constexpr int kOffThreads = 1024;
constexpr int kOffPer = (kMaxNlist + kOffThreads - 1) / kOffThreads;  // lists per thread, at most

// tiles non-null: also write the round's tiles and clear the histogram (the
// work of sched_tiles_kernel), for indexes with few lists per thread.
// Items per query tile when a list's c items split into ntq = ceil(c / tile_q)
// tiles: the same share for every tile, in whole 16-query blocks where
// tile_q allows (tiles of one list then take about the same time, which keeps
// their reads of the list's rows close together), at most tile_q.  Every
// tile is non-empty: (ntq - 1) * gs <= (ntq - 1) * tile_q < c.
__device__ __forceinline__ int group_size(int c, int ntq, int tile_q) {
  const int share = (c + ntq - 1) / ntq;
  const int gs = tile_q >= 16 ? (share + 15) / 16 * 16 : share;
  return min(gs, tile_q);
}

__global__ __launch_bounds__(kOffThreads) void sched_offsets_kernel(
    int32_t* cnt, const int64_t* __restrict__ list_offsets, int32_t nlist,
    int32_t row_chunk, int32_t tile_q, int32_t* __restrict__ item_off,
    int32_t* __restrict__ cursor, int32_t* __restrict__ tile_off, RoundCounters* rc,
    Tile* __restrict__ tiles, int64_t tile_cap) {
  __shared__ int64_t s_items[kOffThreads];
  __shared__ int64_t s_tiles[kOffThreads];
  __shared__ unsigned long long s_stat[3];
  // every list's item count and length (rows < 2^31, checked at load) in
  // LDS: the loads are coalesced and all in flight at once, and each thread
  // then reads its own contiguous range of lists from LDS
  extern __shared__ int32_t s_lists[];  // [nlist] counts, then [nlist] lengths
  int32_t* const s_c = s_lists;
  int32_t* const s_l = s_lists + nlist;
  const int t = threadIdx.x;
  {
    int32_t cv[kOffPer];
    int64_t a0[kOffPer], a1[kOffPer];
#pragma unroll
    for (int u = 0; u < kOffPer; ++u) {
      const int p = u * kOffThreads + t;
      cv[u] = 0;
      a0[u] = a1[u] = 0;
      if (p < nlist) {
        cv[u] = cnt[p];
        a0[u] = list_offsets[p];
        a1[u] = list_offsets[p + 1];
      }
    }
#pragma unroll
    for (int u = 0; u < kOffPer; ++u) {
      const int p = u * kOffThreads + t;
      if (p < nlist) {
        s_c[p] = cv[u];
        s_l[p] = (int32_t)(a1[u] - a0[u]);
      }
    }
  }
  __syncthreads();
  const int per = (nlist + kOffThreads - 1) / kOffThreads;
  const int b = t * per, e = min(nlist, b + per);
  int64_t si = 0, st = 0;
  unsigned long long list_rows = 0, item_rows = 0, loads = 0;
  for (int p = b; p < e; ++p) {
    const int64_t len = s_l[p];
    const int c = s_c[p];
    si += c;
    if (c > 0 && len > 0) {
      st += (int64_t)((c + tile_q - 1) / tile_q) * ((len + row_chunk - 1) / row_chunk);
      list_rows += (unsigned long long)len;
      item_rows += (unsigned long long)len * (unsigned long long)c;
      loads += 1;
    }
  }
  if (t < 3) s_stat[t] = 0;
  s_items[t] = si;
  s_tiles[t] = st;
  __syncthreads();
  // inclusive Hillis-Steele scan over the 1024 partial sums
  for (int off = 1; off < kOffThreads; off <<= 1) {
    int64_t vi = t >= off ? s_items[t - off] : 0;
    int64_t vt = t >= off ? s_tiles[t - off] : 0;
    __syncthreads();
    s_items[t] += vi;
    s_tiles[t] += vt;
    __syncthreads();
  }
  int64_t ri = s_items[t] - si, rt = s_tiles[t] - st;  // exclusive prefixes
  for (int p = b; p < e; ++p) {
    const int64_t len = s_l[p];
    const int c = s_c[p];
    item_off[p] = (int32_t)ri;
    cursor[p] = (int32_t)ri;
    tile_off[p] = (int32_t)rt;
    if (tiles) {
      // the tiles of the list, written here (few lists per thread), and the
      // list's histogram entry cleared for the next round
      cnt[p] = 0;
      if (c > 0 && len > 0) {
        const int ntq = (c + tile_q - 1) / tile_q;
        const int gs = group_size(c, ntq, tile_q);
        const int nch = (int)((len + row_chunk - 1) / row_chunk);
        int32_t o = (int32_t)rt;
        const int64_t lb = list_offsets[p];
        for (int ch = 0; ch < nch; ++ch) {
          for (int tq = 0; tq < ntq; ++tq) {
            Tile tl;
            tl.r0 = lb + (int64_t)ch * row_chunk;
            tl.nrows = (int32_t)min<int64_t>(row_chunk, len - (int64_t)ch * row_chunk);
            tl.item_begin = (int32_t)ri + tq * gs;
            tl.nq = min(gs, c - tq * gs);
            tl.list = p;
            if (o < tile_cap) tiles[o] = tl;  // past the buffer: reported below
            ++o;
          }
        }
      }
    }
    ri += c;
    if (c > 0 && len > 0)
      rt += (int64_t)((c + tile_q - 1) / tile_q) * ((len + row_chunk - 1) / row_chunk);
  }
  for (int o = 32; o > 0; o >>= 1) {
    list_rows += __shfl_xor(list_rows, o);
    item_rows += __shfl_xor(item_rows, o);
    loads += __shfl_xor(loads, o);
  }
  if ((t & 63) == 0) {
    atomicAdd(&s_stat[0], list_rows);
    atomicAdd(&s_stat[1], item_rows);
    atomicAdd(&s_stat[2], loads);
  }
  __syncthreads();
  if (t == 0) {
    // a tile count past the buffer (never, by the host's bound) runs no scan
    // and fails the search
    const int64_t nt = s_tiles[kOffThreads - 1];
    rc->ntiles = nt <= tile_cap ? (int32_t)nt : 0;
    if (nt > tile_cap) rc->sched_error = 1;
    rc->new_items = 0;
    rc->n_ext = 0;
    for (int x = 0; x < 8; ++x) rc->queue[x] = 0;
    rc->list_rows += s_stat[0];
    rc->item_rows += s_stat[1];
    rc->list_loads += s_stat[2];
  }
}

__global__ void sched_scatter_kernel(const Item* __restrict__ items, int32_t n_items,
                                     const int32_t* __restrict__ P, int32_t n, int32_t q0,
                                     const int64_t* __restrict__ exclude,
                                     int32_t* __restrict__ cursor, BItem* __restrict__ bucket) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n_items) return;
  const Item it = items[i];
  const int p = P[(int64_t)(it.q - q0) * n + it.rank];
  const int pos = atomicAdd(&cursor[p], 1);
  BItem b;
  b.q = it.q;
  b.rank = it.rank;
  b.ex = exclude ? exclude[it.q] : INT64_MIN;
  bucket[pos] = b;
}

// One thread per list: write its tiles (query tiles x row chunks), tiles that
// share a row chunk adjacent, and clear the list's histogram entry for the
// next round.
__global__ void sched_tiles_kernel(int32_t* __restrict__ cnt, const int32_t* __restrict__ item_off,
                                   const int32_t* __restrict__ tile_off,
                                   const int64_t* __restrict__ list_offsets, int32_t nlist,
                                   int32_t row_chunk, int32_t tile_q, Tile* __restrict__ tiles,
                                   int64_t tile_cap) {
  const int p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= nlist) return;
  const int c = cnt[p];
  cnt[p] = 0;
  const int64_t len = list_offsets[p + 1] - list_offsets[p];
  if (c == 0 || len == 0) return;
  const int ntq = (c + tile_q - 1) / tile_q;
  const int gs = group_size(c, ntq, tile_q);
  const int nch = (int)((len + row_chunk - 1) / row_chunk);
  int32_t o = tile_off[p];
  const int64_t lb = list_offsets[p];
  for (int ch = 0; ch < nch; ++ch) {
    for (int tq = 0; tq < ntq; ++tq) {
      Tile t;
      t.r0 = lb + (int64_t)ch * row_chunk;
      t.nrows = (int32_t)min<int64_t>(row_chunk, len - (int64_t)ch * row_chunk);
      t.item_begin = item_off[p] + tq * gs;
      t.nq = min(gs, c - tq * gs);
      t.list = p;
      if (o < tile_cap) tiles[o] = t;
      ++o;
    }
  }
}

// The round's summary for the host: one wave reads the counters (the
// update launch before it on the stream has finished) and writes them to
// coherent pinned host memory with system-scope stores.
__global__ void publish_round_kernel(const RoundCounters* __restrict__ rc,
                                     RoundSummary* __restrict__ out) {
  if (threadIdx.x != 0) return;
  __hip_atomic_store(&out->new_items, rc->new_items, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  __hip_atomic_store(&out->n_ext, rc->n_ext, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  __hip_atomic_store(&out->rank_error, rc->rank_error, __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_SYSTEM);
  __hip_atomic_store(&out->heavy, rc->heavy, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  __hip_atomic_store(&out->sched_error, rc->sched_error, __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_SYSTEM);
  __hip_atomic_store(&out->hits, rc->hits, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  __threadfence_system();
}

// The summary written by the update launch itself when it is one work-group:
// the counter updates the summary reads (new_items, n_ext) are atomics whose
// results their threads consumed before the barrier, so they are done.
__device__ __forceinline__ void publish_from_block(const RoundCounters* rc, RoundSummary* out) {
  __syncthreads();
  if (threadIdx.x != 0) return;
  const int32_t ni = __hip_atomic_load(&rc->new_items, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const int32_t ne = __hip_atomic_load(&rc->n_ext, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(&out->new_items, ni, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  __hip_atomic_store(&out->n_ext, ne, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  __hip_atomic_store(&out->rank_error, rc->rank_error, __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_SYSTEM);
  __hip_atomic_store(&out->heavy, rc->heavy, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  __hip_atomic_store(&out->sched_error, rc->sched_error, __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_SYSTEM);
  __hip_atomic_store(&out->hits, rc->hits, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  __threadfence_system();
}

__device__ __forceinline__ void lookahead_one(int64_t q, const int32_t* __restrict__ P, int32_t n,
                                              int32_t W, int32_t* __restrict__ stop,
                                              int32_t* __restrict__ lmax,
                                              const int32_t* __restrict__ have,
                                              int32_t* __restrict__ ext,
                                              Item* __restrict__ items, int64_t item_cap,
                                              int32_t* __restrict__ cnt, RoundCounters* rc,
                                              const uint32_t* __restrict__ hitbits,
                                              int32_t words, int32_t* __restrict__ issued,
                                              int32_t spec_max, int32_t spec_min, int* emit_from,
                                              int* emit_n) {
  const int L = lmax[q];  // 1-based highest hit rank of this round, 0 = none
  if (L == 0) return;
  lmax[q] = 0;
  const int s = stop[q];
  const int hv = have[q];
  if (!hitbits) {
    // committed ranks only (issued, when kept, stays equal to the emitted end)
    const int reach = (W > n - L) ? n : L + W;  // min(L + W, n) without overflow
    if (reach <= s) return;
    const int e0 = min(s, hv), e1 = min(reach, hv);  // emitted so far / after this update
    if (e1 > e0) {
      // ranks [e0, e1) are emitted by the caller, after one claim per wave
      *emit_from = e0;
      *emit_n = e1 - e0;
      if (issued) issued[q] = e1;
    }
    if (reach > hv) ext[atomicAdd(&rc->n_ext, 1)] = (int32_t)q;
    stop[q] = reach;
    return;
  }
  // Speculative issue.  Ranks [0, i) are scanned, some of them past the stop
  // line s.  Replay the stop rule over the hit ranks in order: a hit at rank
  // r counts only once the line has reached it (r < s'), and then moves the
  // line to min(r + 1 + W, n).  Hits below s - W were counted by earlier
  // updates (every line so far came from a hit at most W below it): counting
  // one again changes nothing, and so does a missing bit there (ranks scanned
  // before the bitmap was kept).  The bits of this round's ranks are all set.
  const int i = issued[q];
  const uint32_t* bits = hitbits + q * words;
  int reach = s;
  int bound = min(reach, i);
  for (int j = s > W ? s - W : 0; j < bound;) {
    const int w = j >> 5;
    uint32_t b = bits[w] & (~0u << (j & 31));
    while (b) {
      const int r = (w << 5) + __builtin_ctz(b);
      if (r >= bound) break;
      const int to = (W > n - (r + 1)) ? n : r + 1 + W;
      if (to > reach) {
        reach = to;
        bound = min(reach, i);
      }
      b &= b - 1;
    }
    j = (w + 1) << 5;
  }
  stop[q] = reach;
  if (reach <= i) return;  // the line ends inside the scanned ranks: stopped
  // The line passed the scanned ranks: issue up to it and, when it moved by
  // at least spec_min ranks in this update, as far again (at most spec_max)
  // past it.
  const int adv = reach - s >= spec_min ? min(reach - s, spec_max) : 0;
  const int tgt = (adv > n - reach) ? n : reach + adv;
  const int e1 = min(tgt, hv);
  if (e1 > i) {
    const int base = atomicAdd(&rc->new_items, e1 - i);
    for (int j = i; j < e1; ++j) {
      Item it;
      it.q = (int32_t)q;
      it.rank = j;
      if ((int64_t)(uint32_t)base + (j - i) < item_cap) items[base + (j - i)] = it;
      atomicAdd(&cnt[P[q * n + j]], 1);
    }
    issued[q] = e1;
  }
  if (reach > hv) ext[atomicAdd(&rc->n_ext, 1)] = (int32_t)q;
}

__global__ void update_lookahead_kernel(int64_t nq, const int32_t* __restrict__ P, int32_t n,
                                        int32_t W, int32_t* __restrict__ stop,
                                        int32_t* __restrict__ lmax,
                                        const int32_t* __restrict__ have,
                                        int32_t* __restrict__ ext, Item* __restrict__ items, int64_t item_cap,
                                        int32_t* __restrict__ cnt, RoundCounters* rc,
                                        const uint32_t* __restrict__ hitbits, int32_t words,
                                        int32_t* __restrict__ issued, int32_t spec_max,
                                        int32_t spec_min, RoundSummary* out) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int e0 = 0, ne = 0;
  if (q < nq)
    lookahead_one(q, P, n, W, stop, lmax, have, ext, items, item_cap, cnt, rc, hitbits, words, issued,
                  spec_max, spec_min, &e0, &ne);
  // The new items of the committed path: one claim on the item counter per
  // wave (a one-address atomic per query would serialise the first round's
  // updates), each lane's share at its prefix of the wave's claim.
  const int lane = threadIdx.x & 63;
  int inc = ne;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int t = __shfl_up(inc, o);
    if (lane >= o) inc += t;
  }
  const int total = __shfl(inc, 63);
  int wbase = 0;
  if (lane == 63 && total > 0) wbase = atomicAdd(&rc->new_items, total);
  wbase = __shfl(wbase, 63);
  if (ne > 0) {
    const int base = wbase + inc - ne;
    for (int j = 0; j < ne; ++j) {
      Item it;
      it.q = (int32_t)q;
      it.rank = e0 + j;
      if ((int64_t)(uint32_t)base + j < item_cap) items[base + j] = it;
      atomicAdd(&cnt[P[q * n + e0 + j]], 1);
    }
  }
  if (out) publish_from_block(rc, out);  // one work-group only
}

// next[q]: rank in flight (0-based) or -1 once stopped; on stopping,
// stale[q] is overwritten with the probe count.
__device__ __forceinline__ void basic_one(int64_t q, const int32_t* __restrict__ P, int32_t n,
                                          int32_t W, int32_t* __restrict__ next,
                                          int32_t* __restrict__ stale,
                                          int32_t* __restrict__ lmax,
                                          const int32_t* __restrict__ have,
                                          int32_t* __restrict__ ext, Item* __restrict__ items, int64_t item_cap,
                                          int32_t* __restrict__ cnt, RoundCounters* rc) {
  const int cur = next[q];
  if (cur < 0) return;
  const bool hit = lmax[q] == cur + 1;
  lmax[q] = 0;
  const int st = hit ? 0 : stale[q] + 1;
  const int nx = cur + 1;
  if (st < W && nx < n) {
    stale[q] = st;
    next[q] = nx;
    if (nx < have[q]) {
      const int pos = atomicAdd(&rc->new_items, 1);
      Item it;
      it.q = (int32_t)q;
      it.rank = nx;
      if ((int64_t)(uint32_t)pos < item_cap) items[pos] = it;
      atomicAdd(&cnt[P[q * n + nx]], 1);
    } else {
      ext[atomicAdd(&rc->n_ext, 1)] = (int32_t)q;
    }
  } else {
    next[q] = -1;
    stale[q] = nx;  // probes
  }
}

__global__ void update_basic_kernel(int64_t nq, const int32_t* __restrict__ P, int32_t n,
                                    int32_t W, int32_t* __restrict__ next,
                                    int32_t* __restrict__ stale, int32_t* __restrict__ lmax,
                                    const int32_t* __restrict__ have, int32_t* __restrict__ ext,
                                    Item* __restrict__ items, int64_t item_cap, int32_t* __restrict__ cnt,
                                    RoundCounters* rc, RoundSummary* out) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q < nq) basic_one(q, P, n, W, next, stale, lmax, have, ext, items, item_cap, cnt, rc);
  if (out) publish_from_block(rc, out);  // one work-group only
}

// Row copy in 16-byte units: dst row i <- src row ext[i].
__global__ void gather_rows_kernel(const int32_t* __restrict__ ext, int32_t n_ext,
                                   const uint4* __restrict__ src, int64_t row_u4,
                                   uint4* __restrict__ dst) {
  const int64_t total = (int64_t)n_ext * row_u4;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = e / row_u4, c = e - i * row_u4;
    dst[e] = src[(int64_t)ext[i] * row_u4 + c];
  }
}

__global__ void scatter_ranks_kernel(const int32_t* __restrict__ ext, int32_t n_ext,
                                     const int32_t* __restrict__ Pext, int32_t n,
                                     int32_t* __restrict__ P) {
  const int64_t total = (int64_t)n_ext * n;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = e / n, j = e - i * n;
    P[(int64_t)ext[i] * n + j] = Pext[e];
  }
}

// After the listed queries' prefixes grew to new_have: lookahead (mode 0)
// emits ranks [min(stop, have), min(stop, new_have)); basic (mode 1) emits
// the rank in flight.
__global__ void emit_pending_kernel(const int32_t* __restrict__ ext, int32_t n_ext, int32_t mode,
                                    const int32_t* __restrict__ P, int32_t n,
                                    const int32_t* __restrict__ state_a,
                                    int32_t* __restrict__ have, int32_t new_have,
                                    Item* __restrict__ items, int64_t item_cap, int32_t* __restrict__ cnt,
                                    RoundCounters* rc, int32_t* __restrict__ issued) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n_ext) return;
  const int64_t q = ext[i];
  const int hv = have[q];
  int e0, e1;
  if (mode == 0) {
    const int s = state_a[q];
    e0 = min(s, hv);
    e1 = min(s, new_have);
  } else {
    const int nx = state_a[q];
    e0 = nx >= hv ? nx : 0;
    e1 = nx >= hv && nx < new_have ? nx + 1 : 0;
  }
  if (e1 > e0) {
    const int base = atomicAdd(&rc->new_items, e1 - e0);
    for (int j = e0; j < e1; ++j) {
      Item it;
      it.q = (int32_t)q;
      it.rank = j;
      if ((int64_t)(uint32_t)base + (j - e0) < item_cap) items[base + (j - e0)] = it;
      atomicAdd(&cnt[P[q * n + j]], 1);
    }
    if (mode == 0 && issued) issued[q] = e1;  // e0 == issued[q]: the update stopped at have
  }
  have[q] = new_have > hv ? new_have : hv;
}

__global__ void snapshot_round_kernel(const RoundCounters* __restrict__ rc,
                                      RoundSnap* __restrict__ log, int32_t slot) {
  if (threadIdx.x != 0) return;
  RoundSnap r;
  r.list_rows = rc->list_rows;
  r.item_rows = rc->item_rows;
  r.list_loads = rc->list_loads;
  r.cands = rc->cands;
  log[slot] = r;
}

__global__ void fill_i32_kernel(int32_t* p, int64_t n, int32_t v) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

__global__ void fill_multi_kernel(FillSegs f) {
  const int64_t step = (int64_t)gridDim.x * blockDim.x;
#pragma unroll
  for (int k = 0; k < kFillSegs; ++k) {
    int32_t* __restrict__ p = f.seg[k].p;
    const int64_t n = f.seg[k].n;
    const int32_t v = f.seg[k].v;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += step) p[i] = v;
  }
}

__global__ void zero_bytes_kernel(uint8_t* p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0;
}

}  // namespace

hipError_t launch_emit_initial(const int32_t* P, int32_t n, int64_t nqc, int32_t q0, int32_t s0,
                               int32_t mode, Item* items, int64_t item_cap, int32_t* cnt,
                               int32_t nlist, int32_t* state_a, int32_t* state_b, int32_t* lmax, hipStream_t s) {
  if (nqc <= 0) return hipSuccess;
  if (nlist < 1 || nlist > kMaxNlist) return hipErrorInvalidValue;
  const int b = std::min(blocks_for(nqc, kInitThreads), kInitBlocksMax);
  hipLaunchKernelGGL(emit_initial_kernel, dim3(b), dim3(kInitThreads), (size_t)nlist * 4, s, P,
                     n, nqc, q0, s0, mode, items, item_cap, cnt, nlist, state_a, state_b, lmax);
  return hipGetLastError();
}

hipError_t launch_sched_offsets(int32_t* cnt, const int64_t* list_offsets, int32_t nlist,
                                int32_t row_chunk, int32_t tile_q, int32_t* item_off,
                                int32_t* cursor, int32_t* tile_off, RoundCounters* rc,
                                Tile* tiles, int64_t tile_cap, hipStream_t s) {
  if (tiles && nlist > kFuseTilesMaxLists) return hipErrorInvalidValue;
  static const hipError_t attr =
      hipFuncSetAttribute((const void*)sched_offsets_kernel,
                          hipFuncAttributeMaxDynamicSharedMemorySize, 8 * kMaxNlist);
  if (attr != hipSuccess) return attr;
  if (nlist > kMaxNlist) return hipErrorInvalidValue;
  hipLaunchKernelGGL(sched_offsets_kernel, dim3(1), dim3(kOffThreads), (size_t)8 * nlist, s, cnt,
                     list_offsets, nlist, row_chunk, tile_q, item_off, cursor, tile_off, rc, tiles,
                     tile_cap);
  return hipGetLastError();
}

hipError_t launch_sched_scatter(const Item* items, int32_t n_items, const int32_t* P, int32_t n,
                                int32_t q0, const int64_t* exclude, int32_t* cursor,
                                BItem* bucket, hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  hipLaunchKernelGGL(sched_scatter_kernel, dim3(blocks_for(n_items)), dim3(kThreads), 0, s, items,
                     n_items, P, n, q0, exclude, cursor, bucket);
  return hipGetLastError();
}

hipError_t launch_sched_tiles(int32_t* cnt, const int32_t* item_off, const int32_t* tile_off,
                              const int64_t* list_offsets, int32_t nlist, int32_t row_chunk,
                              int32_t tile_q, Tile* tiles, int64_t tile_cap, hipStream_t s) {
  hipLaunchKernelGGL(sched_tiles_kernel, dim3(blocks_for(nlist)), dim3(kThreads), 0, s, cnt,
                     item_off, tile_off, list_offsets, nlist, row_chunk, tile_q, tiles, tile_cap);
  return hipGetLastError();
}

hipError_t launch_update_lookahead(int64_t nq, const int32_t* P, int32_t n, int32_t W,
                                   int32_t* stop, int32_t* lmax, const int32_t* have,
                                   int32_t* ext, Item* items, int64_t item_cap, int32_t* cnt,
                                   RoundCounters* rc, const uint32_t* hitbits, int32_t words,
                                   int32_t* issued,
                                   int32_t spec_max, int32_t spec_min, RoundSummary* out,
                                   hipStream_t s) {
  if (hitbits && (!issued || words * 32 < n || spec_max < 0)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(update_lookahead_kernel, dim3(blocks_for(nq)), dim3(kThreads), 0, s, nq, P, n,
                     W, stop, lmax, have, ext, items, item_cap, cnt, rc, hitbits, words, issued,
                     spec_max,
                     spec_min, blocks_for(nq) == 1 ? out : nullptr);
  if (out && blocks_for(nq) > 1)
    hipLaunchKernelGGL(publish_round_kernel, dim3(1), dim3(64), 0, s, rc, out);
  return hipGetLastError();
}

hipError_t launch_update_basic(int64_t nq, const int32_t* P, int32_t n, int32_t W, int32_t* next,
                               int32_t* stale, int32_t* lmax, const int32_t* have, int32_t* ext,
                               Item* items, int64_t item_cap, int32_t* cnt, RoundCounters* rc,
                               RoundSummary* out, hipStream_t s) {
  hipLaunchKernelGGL(update_basic_kernel, dim3(blocks_for(nq)), dim3(kThreads), 0, s, nq, P, n, W,
                     next, stale, lmax, have, ext, items, item_cap, cnt, rc,
                     blocks_for(nq) == 1 ? out : nullptr);
  if (out && blocks_for(nq) > 1)
    hipLaunchKernelGGL(publish_round_kernel, dim3(1), dim3(64), 0, s, rc, out);
  return hipGetLastError();
}

hipError_t launch_gather_rows(const int32_t* ext, int32_t n_ext, const void* src,
                              int64_t row_bytes, void* dst, hipStream_t s) {
  if (n_ext <= 0) return hipSuccess;
  const int64_t row_u4 = row_bytes / 16;
  const int64_t total = (int64_t)n_ext * row_u4;
  const int64_t b = (total + kThreads - 1) / kThreads;
  hipLaunchKernelGGL(gather_rows_kernel, dim3((unsigned)(b < 8192 ? b : 8192)), dim3(kThreads), 0,
                     s, ext, n_ext, (const uint4*)src, row_u4, (uint4*)dst);
  return hipGetLastError();
}

hipError_t launch_scatter_ranks(const int32_t* ext, int32_t n_ext, const int32_t* Pext,
                                int32_t n, int32_t* P, hipStream_t s) {
  if (n_ext <= 0) return hipSuccess;
  const int64_t total = (int64_t)n_ext * n;
  const int64_t b = (total + kThreads - 1) / kThreads;
  hipLaunchKernelGGL(scatter_ranks_kernel, dim3((unsigned)(b < 8192 ? b : 8192)), dim3(kThreads),
                     0, s, ext, n_ext, Pext, n, P);
  return hipGetLastError();
}

hipError_t launch_emit_pending(const int32_t* ext, int32_t n_ext, int32_t mode, const int32_t* P,
                               int32_t n, const int32_t* state_a, int32_t* have,
                               int32_t new_have, Item* items, int64_t item_cap, int32_t* cnt,
                               RoundCounters* rc, int32_t* issued, hipStream_t s) {
  if (n_ext <= 0) return hipSuccess;
  hipLaunchKernelGGL(emit_pending_kernel, dim3(blocks_for(n_ext)), dim3(kThreads), 0, s, ext,
                     n_ext, mode, P, n, state_a, have, new_have, items, item_cap, cnt, rc, issued);
  return hipGetLastError();
}

hipError_t launch_snapshot_round(const RoundCounters* rc, RoundSnap* log, int32_t slot,
                                 hipStream_t s) {
  if (slot < 0 || slot >= kMaxLogRounds) return hipErrorInvalidValue;
  hipLaunchKernelGGL(snapshot_round_kernel, dim3(1), dim3(64), 0, s, rc, log, slot);
  return hipGetLastError();
}

hipError_t launch_fill_i32(int32_t* p, int64_t n, int32_t v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  int b = blocks_for(n);
  hipLaunchKernelGGL(fill_i32_kernel, dim3(b > 4096 ? 4096 : b), dim3(kThreads), 0, s, p, n, v);
  return hipGetLastError();
}

hipError_t launch_fill_multi(const FillSegs& f, hipStream_t s) {
  int64_t most = 0;
  for (int k = 0; k < kFillSegs; ++k) {
    if (f.seg[k].n < 0 || (f.seg[k].n > 0 && !f.seg[k].p)) return hipErrorInvalidValue;
    most = f.seg[k].n > most ? f.seg[k].n : most;
  }
  if (most == 0) return hipSuccess;
  const int b = std::min(blocks_for(most), 4096);
  hipLaunchKernelGGL(fill_multi_kernel, dim3(b), dim3(kThreads), 0, s, f);
  return hipGetLastError();
}

hipError_t launch_zero_bytes(void* p, int64_t bytes, hipStream_t s) {
  if (bytes <= 0) return hipSuccess;
  int b = blocks_for(bytes);
  hipLaunchKernelGGL(zero_bytes_kernel, dim3(b > 4096 ? 4096 : b), dim3(kThreads), 0, s,
                     (uint8_t*)p, bytes);
  return hipGetLastError();
}

}  // namespace sieve
