// api.hip -- the C ABI of libsieve: argument checks, the library-owned index
// layout, the workspace, and the host side of the round loop.
//
// A search is:
//   rank      fp32 MFMA centroid screen + exact fp64 order (rank.hip)
//   admit     initial ready items: ranks 1..min(W, n) with lookahead
//             (Algorithm 2), rank 1 without (Algorithm 1), 1..n for fixed
//   rounds    offsets -> scatter -> tiles -> scan -> update, then one
//             8-byte-class readback of the round counters decides whether
//             another round is needed (the only data-dependent host sync)
//   finalize  counting sort of the candidate pool by query, per-query top-k
// Fixed probing runs the same kernels with every rank admitted up front, in
// query chunks, without updates and without per-chunk syncs.
#include <math.h>
#include <stdlib.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <string>
#include <vector>

#include "host_limits.h"
#include "sieve_internal.h"

namespace sieve {
}

using namespace sieve;

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

#define HIP_TRY(expr)                                                                  \
  do {                                                                                 \
    hipError_t e_ = (expr);                                                            \
    if (e_ != hipSuccess)                                                              \
      return fail(e_ == hipErrorOutOfMemory ? SIEVE_ENOMEM : SIEVE_EDEVICE, "%s: %s (%s)", \
                  #expr, hipGetErrorString(e_), __func__);                             \
  } while (0)

struct Buf {
  void* p = nullptr;
  size_t bytes = 0;
};

// SIEVE_ALLOC_CAP (bytes) refuses any single workspace buffer above it with
// SIEVE_ENOMEM before hipMalloc is called (tests of the out-of-memory path;
// the buffer already held stays valid).
int ensure(Buf& b, size_t bytes) {
  if (bytes == 0) bytes = 16;
  if (b.bytes >= bytes) return SIEVE_OK;
  if (const char* cap = getenv("SIEVE_ALLOC_CAP")) {
    const unsigned long long c = strtoull(cap, nullptr, 10);
    if (c > 0 && bytes > c)
      return fail(SIEVE_ENOMEM, "workspace buffer of %zu bytes exceeds SIEVE_ALLOC_CAP = %llu",
                  bytes, c);
  }
  if (b.p) (void)hipFree(b.p);
  b.p = nullptr;
  b.bytes = 0;
  hipError_t e = hipMalloc(&b.p, bytes);
  if (e != hipSuccess) {
    b.p = nullptr;
    (void)hipGetLastError();
    return fail(SIEVE_ENOMEM, "hipMalloc of %zu bytes failed: %s", bytes, hipGetErrorString(e));
  }
  b.bytes = bytes;
  return SIEVE_OK;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

}  // namespace

struct sieve_index {
  int dtype = 0;
  int64_t n = 0;
  int d = 0;
  int nlist = 0;
  int device = 0;
  int cus = 256;
  void* vectors = nullptr;
  int64_t* offsets = nullptr;
  int64_t* ids = nullptr;
  void* centroids = nullptr;
  void* cfrag = nullptr;  // fragment-order centroids (ranking), or null
  void* vfrag = nullptr;  // fragment-order vectors (scan), or null
  int64_t* foff = nullptr;  // [nlist + 1] partition starts in vfrag (rows)
  std::vector<int64_t> h_offsets;
  int64_t max_list = 0;
  double cmax = 0.0;
  // workspace, grown on demand (every buffer is listed once, in SIEVE_WORKSPACE,
  // so that sieve_free_index releases all of them)
#define SIEVE_WORKSPACE(X)                                                                 \
  X(scores) X(P) X(items) X(bucket) X(tiles) X(cnt) X(item_off) X(cursor) X(tile_off) X(rc) \
  X(state_a) X(state_b) X(lmax) X(hcount) X(hoff) X(hcur) X(scan_tmp) X(pool)              \
  X(pool_sorted) X(heavy) X(spill) X(have) X(ext) X(qext) X(Pext) X(cand) X(ccount) X(cal_idx)      \
  X(cal_q) X(cal_x) X(cal_bits) X(cal_rank) X(cal_hist) X(mix_ids) X(mix_scores)            \
  X(mix_probes) X(spec_bits) X(rlog)
#define SIEVE_DECLARE_BUF(name) Buf name;
  SIEVE_WORKSPACE(SIEVE_DECLARE_BUF)
#undef SIEVE_DECLARE_BUF
  int64_t pool_cap = 0;
  int64_t heavy_cap = 0;  // HeavyRec records the heavy buffer holds
  RoundCounters* rc_host = nullptr;
  RoundSummary* rs_host = nullptr;  // coherent pinned memory the update launches write
  RoundSummary* rs_dev = nullptr;   // its device address
  // phase timing (only when stats are requested): events are recorded on the
  // stream as the search goes and read once after its final synchronisation
  std::vector<hipEvent_t> ev_pool;
  size_t ev_used = 0;
  std::vector<int> span_phase, span_a, span_b;
  // per-round log of the last timed search: items and the scan span of each
  // round as it runs, the finished records after the final synchronisation
  std::vector<int64_t> round_items;
  std::vector<int> round_span;
  std::vector<sieve_round> rounds_log;
  int32_t rounds_logged = 0;  // rounds of that search (records past kMaxLogRounds are dropped)
};

namespace {

int elem_bytes(int dtype) { return dtype == SIEVE_F32 ? 4 : 2; }

double host_elem(const void* base, int dtype, int64_t i) {
  if (dtype == SIEVE_F32) return (double)((const float*)base)[i];
  return (double)((const _Float16*)base)[i];
}

enum Phase { kRank = 0, kSched, kScan, kUpdate, kFinal, kTotal, kPhases };

// Record an event on the stream and return its slot; -1 when not timing.
int mark(sieve_index* ix, bool timed, hipStream_t s) {
  if (!timed) return -1;
  if (ix->ev_used == ix->ev_pool.size()) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) {
      (void)hipGetLastError();
      return -1;
    }
    ix->ev_pool.push_back(e);
  }
  const int slot = (int)ix->ev_used++;
  if (hipEventRecord(ix->ev_pool[slot], s) != hipSuccess) {
    (void)hipGetLastError();
    return -1;
  }
  return slot;
}

void span(sieve_index* ix, int phase, int a, int b) {
  if (a < 0 || b < 0) return;
  ix->span_phase.push_back(phase);
  ix->span_a.push_back(a);
  ix->span_b.push_back(b);
}

void reset_timeline(sieve_index* ix) {
  ix->ev_used = 0;
  ix->span_phase.clear();
  ix->span_a.clear();
  ix->span_b.clear();
  ix->round_items.clear();
  ix->round_span.clear();
}

// After the stream has drained: milliseconds per phase, and scan span count.
void read_timeline(sieve_index* ix, float* ms, int* scan_spans) {
  for (int p = 0; p < kPhases; ++p) ms[p] = 0.f;
  *scan_spans = 0;
  for (size_t i = 0; i < ix->span_phase.size(); ++i) {
    float t = 0.f;
    if (hipEventElapsedTime(&t, ix->ev_pool[ix->span_a[i]], ix->ev_pool[ix->span_b[i]]) !=
        hipSuccess) {
      (void)hipGetLastError();
      t = 0.f;
    }
    ms[ix->span_phase[i]] += t;
    if (ix->span_phase[i] == kScan) ++*scan_spans;
  }
}

// Tunables of the scan decomposition.  They never change results; the
// SIEVE_* environment variables override them for tuning sweeps.
int env_int(const char* name, int dflt) {
  const char* v = getenv(name);
  if (!v || !*v) return dflt;
  const int x = atoi(v);
  return x > 0 ? x : dflt;
}

// A count that may be zero.
int env_count(const char* name, int dflt) {
  const char* v = getenv(name);
  if (!v || !*v) return dflt;
  const int x = atoi(v);
  return x >= 0 ? x : dflt;
}

int row_chunk_for(const sieve_index* ix, const char* knob, int dflt) {
  // the scan addresses a tile's rows with 32-bit byte offsets
  const int64_t row_bytes = (int64_t)ix->d * elem_bytes(ix->dtype);
  const int64_t lim = ((int64_t)INT32_MAX / row_bytes) / 64 * 64;
  int64_t rc = env_int(knob, dflt);
  rc = ((rc + 63) / 64) * 64;
  return (int)std::max<int64_t>(64, std::min(rc, lim));
}

int scan_grid(const sieve_index* ix, int tile_q) {
  const size_t lds = scan_lds_bytes(ix->dtype, ix->d, tile_q) + 4096;
  int per_cu = (int)((160 * 1024) / lds);
  per_cu = per_cu < 1 ? 1 : (per_cu > 2 ? 2 : per_cu);
  if (scan_uses_rega(ix->dtype, ix->d)) per_cu = 1;  // the whole register file per wave
  per_cu = std::min(env_int("SIEVE_SCAN_BLOCKS_PER_CU", per_cu), 2);  // <= the spill grid
  return ((ix->cus * per_cu + 7) / 8) * 8;  // the scan's schedule needs a multiple of 8
}

// Rounds with many tiles per work-group balance better with the atomic
// queue, rounds with a few without it.  The round's tile count is estimated on
// the host from its size: every touched list gives at least one tile per row
// chunk, and a dense round about n_items / group more per chunk.
int scan_dynamic(const sieve_index* ix, int64_t n_items, bool dense, int chunk, int group,
                 int grid) {
  const int64_t avg_len = std::max<int64_t>(ix->n / std::max(ix->nlist, 1), 1);
  const int64_t chunks = (avg_len + chunk - 1) / chunk;
  const int64_t lists = std::min<int64_t>(n_items, ix->nlist);
  const int64_t groups = dense ? lists + n_items / std::max(group, 1) : lists;
  const int64_t min_tiles = (int64_t)env_int("SIEVE_DYNAMIC_MIN_TILES", 16) * grid;
  return groups * chunks >= min_tiles ? 1 : 0;
}

struct SearchPlan {
  int n;            // effective probes limit
  int mode;         // 0 lookahead, 1 basic, 2 fixed
  int W;
  int k;
  float tau;
  int64_t nq;
  int tile_q;           // query rows a tile stages (LDS sizing)
  int group_q;          // items of one list grouped into a tile (tile_q; 1 = serial)
  bool rega;            // register-A scan: dense and sparse rounds take different tiles
  int min_group;        // smallest tile grouping of any round (workspace bound)
  int row_chunk;        // rows per tile in sparse rounds
  int row_chunk_dense;  // rows per tile in dense rounds (long tiles amortise the tile start)
  int dense_q;          // a round is dense with at least this many items per list on average
  int64_t rank_chunk;  // queries per centroid-screen chunk
  int64_t fix_chunk;   // queries per fixed-probe chunk
  int64_t item_cap;
  int r0;              // ranks ordered up front (the rest on demand)
  bool wide;           // wide scan configuration (see tile_rows_wide)
  int scan_grid;       // scan work-groups (fixed for the whole search)
  bool wide_rank;      // rank with room for every boundary near-tie (retry path)
  int rank_div;        // register-query prefix ranking: first pass over 1/rank_div of the
                       // centroids (a looser bound; 1 after an overflow)
  bool spec;           // lookahead with speculative issue past the stop line
  int spec_round;      // first round whose update speculates
  int spec_max;        // ranks issued past the stop line, at most
  int spec_min;        // a line must move at least this far to speculate
  int hit_words;       // 32-bit words per query of the rank bitmap (spec)
};

int check_common(const sieve_index* ix, const void* queries, int64_t nq, int32_t k, float tau,
                 int64_t* out_ids, float* out_scores, int32_t* out_probes) {
  if (!ix) return fail(SIEVE_EINVAL, "index handle is NULL");
  if (nq < 0) return fail(SIEVE_EINVAL, "nq = %lld is negative", (long long)nq);
  if (k < 1 || k > SIEVE_K_MAX) return fail(SIEVE_EINVAL, "k = %d outside [1, %d]", k, SIEVE_K_MAX);
  if (isnan(tau)) return fail(SIEVE_EINVAL, "tau is NaN");
  if (nq > 0 && (!queries || !out_ids || !out_scores || !out_probes))
    return fail(SIEVE_EINVAL, "queries and every output pointer must be non-NULL when nq > 0");
  if (nq > 0 && !aligned16(queries)) return fail(SIEVE_EINVAL, "queries must be 16-byte aligned");
  if (nq > (int64_t)INT32_MAX / 2) return fail(SIEVE_EUNSUPPORTED, "nq = %lld too large", (long long)nq);
  return SIEVE_OK;
}

// Spill entries per scan work-group (rows past a query's LDS slots in one
// tile); 0 when a tile could hold more rows than the entries can address.
int spill_cap(const sieve_index* ix) {
  if (ix->max_list >= ((int64_t)1 << kSpillRowBits)) return 0;
  // SIEVE_SPILL_CAP lowers it (tests of the overflow path)
  return std::min(env_count("SIEVE_SPILL_CAP", 16384), 16384) & ~1;  // even: see SrtEnt
}
// The candidate arena packs a row offset in 24 bits; SIEVE_ARENA = 0 turns it
// off (every tile with candidates then takes the exact top-k pass; tests).
bool arena_on(const sieve_index* ix) {
  return ix->max_list < ((int64_t)1 << kSpillRowBits) && env_count("SIEVE_ARENA", 1) != 0;
}
int spill_grid(const sieve_index* ix) { return ((2 * ix->cus + 7) / 8) * 8; }

int grow_workspace(sieve_index* ix, const SearchPlan& pl) {
  const int64_t nq = pl.nq;
  const int n = pl.n;
  const int64_t rank_rows = pl.mode == 2 ? pl.fix_chunk : nq;
  int st;
  if ((st = ensure(ix->scores, (size_t)pl.rank_chunk * ix->nlist * sizeof(float)))) return st;
  if ((st = ensure(ix->P, (size_t)rank_rows * n * sizeof(int32_t)))) return st;
  if ((st = ensure(ix->items, (size_t)pl.item_cap * sizeof(Item)))) return st;
  if ((st = ensure(ix->bucket, (size_t)pl.item_cap * sizeof(BItem)))) return st;
  // tiles: sum_p ceil(c_p / tq) * ceil(len_p / rc) <= items * max_chunks / tq + lists + rows / rc
  const int64_t max_ch = (ix->max_list + pl.row_chunk - 1) / pl.row_chunk;
  const int64_t tile_cap = pl.item_cap / std::min(pl.group_q, pl.min_group) *
                               (max_ch > 0 ? max_ch : 1) +
                           ix->nlist + ix->n / pl.row_chunk + 16;
  if (tile_cap > INT32_MAX) return fail(SIEVE_EUNSUPPORTED, "tile count bound overflows int32");
  if ((st = ensure(ix->tiles, (size_t)tile_cap * sizeof(Tile)))) return st;
  const size_t nl = (size_t)ix->nlist;
  if ((st = ensure(ix->cnt, nl * 4)) || (st = ensure(ix->item_off, nl * 4)) ||
      (st = ensure(ix->cursor, nl * 4)) || (st = ensure(ix->tile_off, nl * 4)))
    return st;
  if ((st = ensure(ix->rc, sizeof(RoundCounters)))) return st;
  const size_t qn = (size_t)nq * 4;
  if ((st = ensure(ix->have, qn)) || (st = ensure(ix->ext, qn))) return st;
  if ((st = ensure(ix->state_a, qn)) || (st = ensure(ix->state_b, qn)) ||
      (st = ensure(ix->lmax, qn)) || (st = ensure(ix->hcount, qn)) ||
      (st = ensure(ix->hoff, (size_t)nq * 8)) || (st = ensure(ix->hcur, (size_t)nq * 8)))
    return st;
  if ((st = ensure(ix->scan_tmp, exclusive_scan_tmp_elems(nq) * 8))) return st;
  if (pl.spec && (st = ensure(ix->spec_bits, (size_t)nq * pl.hit_words * 4))) return st;
  if ((st = ensure(ix->rlog, (size_t)kMaxLogRounds * sizeof(RoundSnap)))) return st;
  // The pool holds at most k entries per (query, tile); most searches need far
  // fewer, so it starts small and grows (the search is then re-run) only when
  // a search needs more.
  if (ix->pool_cap < (1 << 20)) {
    int64_t cap = nq * 16;
    ix->pool_cap = cap < (1 << 20) ? (1 << 20) : cap;
  }
  // overflow records: a first size (SIEVE_HEAVY_CAP0 lowers it for tests of the
  // regrowth), then grown on demand
  if (ix->heavy_cap == 0)
    ix->heavy_cap = env_int("SIEVE_HEAVY_CAP0", (int)std::min<int64_t>(std::max<int64_t>(4096, nq / 8), 1 << 24));
  if ((st = ensure(ix->heavy, (size_t)ix->heavy_cap * sizeof(HeavyRec)))) return st;
  // per scan work-group: the candidate arena's global extension and the
  // tile's grouped arena (every grid of this search has at most spill_grid
  // work-groups)
  if ((st = ensure(ix->spill,
                   (size_t)spill_grid(ix) * arena_block_entries(spill_cap(ix)) * sizeof(TileSpill))))
    return st;
  if ((st = ensure(ix->pool, (size_t)ix->pool_cap * sizeof(Hit)))) return st;
  if ((st = ensure(ix->pool_sorted, (size_t)ix->pool_cap * sizeof(Hit)))) return st;
  if (!ix->rc_host) HIP_TRY(hipHostMalloc((void**)&ix->rc_host, sizeof(RoundCounters), 0));
  if (!ix->rs_host) {
    HIP_TRY(hipHostMalloc((void**)&ix->rs_host, sizeof(RoundSummary),
                          hipHostMallocCoherent | hipHostMallocMapped));
    HIP_TRY(hipHostGetDevicePointer((void**)&ix->rs_dev, ix->rs_host, 0));
  }
  return SIEVE_OK;
}

// Centroid order of queries [q0, q0 + cnt) into P (row-major [cnt][n]).
// Ranking path: 1 materialised screen scores + selection, 2 fused screen +
// selection (short prefixes only); SIEVE_RANK_PATH forces one for tests.
bool use_prefix_path(const sieve_index* ix, int nsel, bool wide) {
  if (wide || nsel > kRankPrefixMax || nsel > ix->nlist) return false;
  const int forced = env_int("SIEVE_RANK_PATH", 0);
  if (forced == 1) return false;
  if (forced == 2) return true;
  return ix->nlist > 1024;
}

// Order the first nsel centroids of queries [q0, q0 + cnt) into rows of P
// (row stride ldp), in chunks whose screen scores (or candidate lists) fit
// the given buffers: prefix path, chunks of chunk_prefix queries with
// cand[chunk * rank_prefix_cap] and ccount[chunk]; screen path, chunks of
// chunk_scores queries with scores[chunk * nlist].
int rank_queries_in(const sieve_index* ix, const void* queries, int64_t q0, int64_t cnt, int nsel,
                    int64_t ldp, const SearchPlan& pl, int32_t* P, RoundCounters* rc,
                    unsigned long long* cand, int32_t* ccount, int64_t chunk_prefix,
                    float* scores, int64_t chunk_scores, hipStream_t s) {
  if (use_prefix_path(ix, nsel, pl.wide_rank)) {
    for (int64_t a = 0; a < cnt; a += chunk_prefix) {
      const int32_t c = (int32_t)((cnt - a) < chunk_prefix ? (cnt - a) : chunk_prefix);
      HIP_TRY(launch_rank_prefix(ix->dtype, queries, q0 + a, c, ix->centroids, ix->cfrag,
                                 ix->nlist, ix->d, nsel, ix->cmax, cand, ccount, P + a * ldp, ldp,
                                 rc, pl.rank_div, s));
    }
    return SIEVE_OK;
  }
  for (int64_t a = 0; a < cnt; a += chunk_scores) {
    const int32_t c = (int32_t)((cnt - a) < chunk_scores ? (cnt - a) : chunk_scores);
    HIP_TRY(launch_rank_scores(ix->dtype, queries, q0 + a, c, ix->centroids, ix->nlist, ix->d,
                               scores, s));
    HIP_TRY(launch_rank_select(ix->dtype, queries, q0 + a, c, ix->centroids, ix->nlist, ix->d,
                               scores, nsel, ix->cmax, P + a * ldp, ldp, rc, pl.wide_rank, s));
  }
  return SIEVE_OK;
}

// rank_queries_in with the index's own workspace (grown as needed).
int rank_queries(sieve_index* ix, const void* queries, int64_t q0, int64_t cnt, int nsel,
                 int64_t ldp, const SearchPlan& pl, int32_t* P, hipStream_t s) {
  RoundCounters* rc = (RoundCounters*)ix->rc.p;
  int64_t chunk_prefix = 1;
  if (use_prefix_path(ix, nsel, pl.wide_rank)) {
    const int64_t cap = rank_prefix_cap(nsel, ix->nlist);
    chunk_prefix = cnt < (1 << 18) ? cnt : (1 << 18);
    int st;
    if ((st = ensure(ix->cand, (size_t)chunk_prefix * cap * sizeof(unsigned long long))) ||
        (st = ensure(ix->ccount, (size_t)chunk_prefix * sizeof(int32_t))))
      return st;
  }
  return rank_queries_in(ix, queries, q0, cnt, nsel, ldp, pl, P, rc,
                         (unsigned long long*)ix->cand.p, (int32_t*)ix->ccount.p, chunk_prefix,
                         (float*)ix->scores.p, pl.rank_chunk, s);
}

ScanArgs make_scan_args(sieve_index* ix, const void* queries, const int64_t* exclude,
                        const SearchPlan& pl) {
  ScanArgs a;
  RoundCounters* rc = (RoundCounters*)ix->rc.p;
  a.vectors = ix->vectors;
  a.vfrag = ix->vfrag;
  a.frag_offsets = ix->foff;
  a.list_offsets = ix->offsets;
  a.ids = ix->ids;
  a.queries = queries;
  a.exclude = exclude;
  a.bucket = (const BItem*)ix->bucket.p;
  a.tiles = (const Tile*)ix->tiles.p;
  a.rc = rc;
  a.lmax = (int32_t*)ix->lmax.p;
  a.hcount = (int32_t*)ix->hcount.p;
  a.pool = (Hit*)ix->pool.p;
  a.pool_count = &rc->hits;
  a.pool_cap = ix->pool_cap;
  a.heavy = (HeavyRec*)ix->heavy.p;
  a.heavy_count = &rc->heavy;
  a.heavy_cap = ix->heavy_cap;
  a.k = pl.k;
  a.spill = (TileSpill*)ix->spill.p;
  a.spill_cap = spill_cap(ix);
  a.arena_on = arena_on(ix) ? 1 : 0;
  a.d = ix->d;
  a.row_chunk = pl.row_chunk;
  a.tile_q = pl.tile_q;
  a.wide = pl.wide ? 1 : 0;
  a.tau = pl.tau;
  return a;
}

// One scheduling round over n_items ready items (already histogrammed).
// at: an event recorded at the stream's current position (-1: none), which
// then opens the schedule span; on return, the event that closes the scan.
int run_round(sieve_index* ix, const ScanArgs& sa, int n_items, int64_t q0, const int32_t* P,
              const SearchPlan& pl, hipStream_t s, bool timed, int* at) {
  RoundCounters* rc = (RoundCounters*)ix->rc.p;
  const bool dense = (int64_t)n_items >= (int64_t)pl.dense_q * ix->nlist;
  const int chunk = dense ? pl.row_chunk_dense : pl.row_chunk;
  int group = pl.group_q, tile_q = pl.tile_q, grid = pl.scan_grid;
  if (pl.rega) {
    // dense rounds: 128-query tiles of whole lists, one work-group per CU;
    // sparse rounds: 64-query tiles of 512 rows, two per CU
    // (SIEVE_REGA_DENSE = 0 gives dense rounds the sparse shape; tuning only)
    const bool big = dense && env_count("SIEVE_REGA_DENSE", 1) != 0;
    tile_q = scan_rega_tile_q(big);
    group = pl.group_q == 1 ? 1 : tile_q;
    grid = ((ix->cus * (big ? 1 : 2) + 7) / 8) * 8;
  }
  const int e0 = *at >= 0 ? *at : mark(ix, timed, s);
  // few lists: the offsets launch also writes the tiles
  const int64_t tile_cap = (int64_t)(ix->tiles.bytes / sizeof(Tile));
  const bool fuse = ix->nlist <= kFuseTilesMaxLists;
  HIP_TRY(launch_sched_offsets((int32_t*)ix->cnt.p, ix->offsets, ix->nlist, chunk, group,
                               (int32_t*)ix->item_off.p, (int32_t*)ix->cursor.p,
                               (int32_t*)ix->tile_off.p, rc, fuse ? (Tile*)ix->tiles.p : nullptr,
                               tile_cap, s));
  HIP_TRY(launch_sched_scatter((const Item*)ix->items.p, n_items, P, pl.n, (int32_t)q0, sa.exclude,
                               (int32_t*)ix->cursor.p, (BItem*)ix->bucket.p, s));
  if (!fuse)
    HIP_TRY(launch_sched_tiles((int32_t*)ix->cnt.p, (const int32_t*)ix->item_off.p,
                               (const int32_t*)ix->tile_off.p, ix->offsets, ix->nlist, chunk,
                               group, (Tile*)ix->tiles.p, tile_cap, s));
  const int e1 = mark(ix, timed, s);
  ScanArgs sr = sa;
  sr.dynamic = scan_dynamic(ix, n_items, dense, chunk, group, grid);
  sr.tile_q = tile_q;
  HIP_TRY(launch_scan(ix->dtype, sr, grid, s));
  const int e2 = mark(ix, timed, s);
  span(ix, kSched, e0, e1);
  span(ix, kScan, e1, e2);
  *at = e2;
  if (timed) {
    // the round's counters, for the per-round log (sieve_round_log)
    const int slot = (int)ix->round_items.size();
    ix->round_items.push_back(n_items);
    ix->round_span.push_back(e1 >= 0 && e2 >= 0 ? (int)ix->span_phase.size() - 1 : -1);
    if (slot < kMaxLogRounds)
      HIP_TRY(launch_snapshot_round(rc, (RoundSnap*)ix->rlog.p + slot, 0, s));
  }
  return SIEVE_OK;
}

// Turn the per-round counter snapshots of a timed search into its round log
// (differences of consecutive snapshots, scan time from the round's span).
int finish_round_log(sieve_index* ix, int32_t kind, hipStream_t s) {
  const int n = (int)std::min<size_t>(ix->round_items.size(), kMaxLogRounds);
  std::vector<RoundSnap> snap((size_t)n);
  if (n > 0) {
    HIP_TRY(hipMemcpyAsync(snap.data(), ix->rlog.p, (size_t)n * sizeof(RoundSnap),
                           hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
  }
  const double eb = (double)ix->d * elem_bytes(ix->dtype);
  ix->rounds_log.assign((size_t)n, sieve_round{});
  ix->rounds_logged = (int32_t)ix->round_items.size();
  RoundSnap prev = {0, 0, 0, 0};
  for (int r = 0; r < n; ++r) {
    sieve_round& o = ix->rounds_log[(size_t)r];
    o.items = ix->round_items[(size_t)r];
    o.list_rows = (int64_t)(snap[r].list_rows - prev.list_rows);
    o.item_rows = (int64_t)(snap[r].item_rows - prev.item_rows);
    o.list_loads = (int64_t)(snap[r].list_loads - prev.list_loads);
    o.candidates = (int64_t)(snap[r].cands - prev.cands);
    o.scan_bytes = (double)o.list_rows * eb + (double)o.items * (eb + sizeof(Item)) +
                   (double)o.candidates * sizeof(Hit);
    o.scan_flops = 2.0 * (double)ix->d * (double)o.item_rows;
    o.kind = kind;
    o.ms_scan = 0.f;
    const int sp = ix->round_span[(size_t)r];
    if (sp >= 0 && hipEventElapsedTime(&o.ms_scan, ix->ev_pool[ix->span_a[sp]],
                                       ix->ev_pool[ix->span_b[sp]]) != hipSuccess) {
      (void)hipGetLastError();
      o.ms_scan = 0.f;
    }
    prev = snap[r];
  }
  return SIEVE_OK;
}

// Extra outputs of the fixed-probe sample search of a calibrated call: per
// query a bitmap of the ranks whose probe had a candidate, and the rank each
// returned neighbour was found at.
struct CalibOut {
  uint32_t* hitbits;
  int32_t words;
  int32_t* frank;
};

// out_map: null, or [nq] output row of each query.  cal: null, or the
// calibration outputs (then nq < kCalibMaxSample).
int search_impl(sieve_index* ix, const void* queries, int64_t nq, const int64_t* exclude,
                SearchPlan pl, const int32_t* out_map, int64_t* out_ids, float* out_scores,
                int32_t* out_probes, sieve_stats* stats, hipStream_t s,
                const CalibOut* cal = nullptr) {
  int st;
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  if (dev != ix->device)
    return fail(SIEVE_EINVAL, "current device %d differs from the index's device %d", dev,
                ix->device);
  const bool timed = stats != nullptr;
  if ((st = grow_workspace(ix, pl))) return st;

  RoundCounters* rc = (RoundCounters*)ix->rc.p;
  const int e = elem_bytes(ix->dtype);
  const ScanArgs sa0 = make_scan_args(ix, queries, exclude, pl);

  int pool_retries = 0;
  for (;;) {
    reset_timeline(ix);
    int rounds = 0;
    int64_t items_total = 0;
    ScanArgs sa = sa0;
    sa.pool = (Hit*)ix->pool.p;
    sa.pool_cap = ix->pool_cap;
    sa.heavy = (HeavyRec*)ix->heavy.p;
    sa.heavy_cap = ix->heavy_cap;
    if (cal) {
      sa.hitbits = cal->hitbits;
      sa.hit_words = cal->words;
    }

    const int t_begin = mark(ix, timed, s);
    int at = -1;  // an event at the stream's current position, when one was just recorded
    {
      // every per-search reset in one launch: counters, partition histogram,
      // per-query candidate counts, the calibration bitmap, the ordered-prefix lengths
      static_assert(sizeof(RoundCounters) % 4 == 0, "word fills");
      FillSegs f = {};
      f.seg[0] = {(int32_t*)rc, (int64_t)(sizeof(RoundCounters) / 4), 0};
      f.seg[2] = {(int32_t*)ix->cnt.p, (int64_t)ix->nlist, 0};
      f.seg[3] = {(int32_t*)ix->hcount.p, nq, 0};
      if (cal) f.seg[4] = {(int32_t*)cal->hitbits, nq * (int64_t)cal->words, 0};
      if (pl.mode != 2) f.seg[5] = {(int32_t*)ix->have.p, nq, pl.r0};
      HIP_TRY(launch_fill_multi(f, s));
    }
    bool spec_used = false;  // a round kept the rank bitmap (its ranks may pass stop lines)
    RoundSummary sm = {0, 0, 0, 0, 0, 0, 0};  // the host's view of the last round
    int32_t* P = (int32_t*)ix->P.p;

    if (pl.mode != 2) {
      const int r0 = mark(ix, timed, s);
      if ((st = rank_queries(ix, queries, 0, nq, pl.r0, pl.n, pl, P, s))) return st;
      const int s0 = pl.mode == 0 ? (pl.W < pl.n ? pl.W : pl.n) : 1;
      HIP_TRY(launch_emit_initial(P, pl.n, nq, 0, s0, pl.mode, (Item*)ix->items.p, pl.item_cap,
                                  (int32_t*)ix->cnt.p, ix->nlist, (int32_t*)ix->state_a.p,
                                  (int32_t*)ix->state_b.p, (int32_t*)ix->lmax.p, s));
      // adjacent phases share the event between them (fewer records per round)
      at = mark(ix, timed, s);
      span(ix, kRank, r0, at);
      int64_t n_items = nq * s0;
      while (n_items > 0) {
        // speculative issue from round spec_round on: its scans keep the rank bitmap
        const bool spec_now = pl.spec && rounds >= pl.spec_round;
        if (spec_now && !spec_used) {
          HIP_TRY(launch_zero_bytes(ix->spec_bits.p, (size_t)nq * pl.hit_words * 4, s));
          sa.hitbits = (uint32_t*)ix->spec_bits.p;
          sa.hit_words = pl.hit_words;
          spec_used = true;
        }
        if ((st = run_round(ix, sa, (int)n_items, 0, P, pl, s, timed, &at))) return st;
        const int u0 = at;
        int32_t* have = (int32_t*)ix->have.p;
        int32_t* ext = (int32_t*)ix->ext.p;
        if (pl.mode == 0)
          HIP_TRY(launch_update_lookahead(
              nq, P, pl.n, pl.W, (int32_t*)ix->state_a.p, (int32_t*)ix->lmax.p, have, ext,
              (Item*)ix->items.p, pl.item_cap, (int32_t*)ix->cnt.p, rc, spec_now ? sa.hitbits : nullptr,
              sa.hit_words, pl.spec ? (int32_t*)ix->state_b.p : nullptr, pl.spec_max,
              pl.spec_min, ix->rs_dev, s));
        else
          HIP_TRY(launch_update_basic(nq, P, pl.n, pl.W, (int32_t*)ix->state_a.p,
                                      (int32_t*)ix->state_b.p, (int32_t*)ix->lmax.p, have, ext,
                                      (Item*)ix->items.p, pl.item_cap, (int32_t*)ix->cnt.p, rc, ix->rs_dev,
                                      s));
        at = mark(ix, timed, s);
        span(ix, kUpdate, u0, at);
        HIP_TRY(hipStreamSynchronize(s));
        const volatile RoundSummary* rs = ix->rs_host;
        sm.new_items = rs->new_items;
        sm.n_ext = rs->n_ext;
        sm.rank_error = rs->rank_error;
        sm.heavy = rs->heavy;
        sm.hits = rs->hits;
        if (rs->sched_error)
          return fail(SIEVE_EINTERNAL, "a round's tiles exceeded the tile buffer");
        items_total += n_items;
        ++rounds;
        if (sm.rank_error) break;  // handled below: re-rank wide or fail
        if (const int32_t n_ext = sm.n_ext) {
          // stop lines passed the ordered prefix: order every rank of those queries
          const int x0 = at;
          const int64_t rb = (int64_t)ix->d * e;
          if ((st = ensure(ix->qext, (size_t)n_ext * rb)) ||
              (st = ensure(ix->Pext, (size_t)n_ext * pl.n * sizeof(int32_t))))
            return st;
          HIP_TRY(launch_gather_rows(ext, n_ext, queries, rb, ix->qext.p, s));
          if ((st = rank_queries(ix, ix->qext.p, 0, n_ext, pl.n, pl.n, pl, (int32_t*)ix->Pext.p,
                                 s)))
            return st;
          HIP_TRY(launch_scatter_ranks(ext, n_ext, (const int32_t*)ix->Pext.p, pl.n, P, s));
          HIP_TRY(launch_emit_pending(ext, n_ext, pl.mode, P, pl.n, (const int32_t*)ix->state_a.p,
                                      have, pl.n, (Item*)ix->items.p, pl.item_cap, (int32_t*)ix->cnt.p, rc,
                                      pl.spec ? (int32_t*)ix->state_b.p : nullptr, s));
          at = mark(ix, timed, s);
          span(ix, kRank, x0, at);
          HIP_TRY(hipMemcpyAsync(ix->rc_host, rc, sizeof(RoundCounters), hipMemcpyDeviceToHost,
                                 s));
          HIP_TRY(hipStreamSynchronize(s));
          sm.new_items = ix->rc_host->new_items;
          sm.rank_error = ix->rc_host->rank_error;
          if (sm.rank_error) break;
        }
        n_items = sm.new_items;
        if (n_items > pl.item_cap)
          return fail(SIEVE_EINTERNAL, "round emitted %lld items, capacity %lld",
                      (long long)n_items, (long long)pl.item_cap);
      }
    } else {
      for (int64_t q0 = 0; q0 < nq; q0 += pl.fix_chunk) {
        const int64_t c = (nq - q0) < pl.fix_chunk ? (nq - q0) : pl.fix_chunk;
        const int r0 = mark(ix, timed, s);
        if ((st = rank_queries(ix, queries, q0, c, pl.n, pl.n, pl, P, s))) return st;
        HIP_TRY(launch_emit_initial(P, pl.n, c, (int32_t)q0, pl.n, 2, (Item*)ix->items.p,
                                    pl.item_cap, (int32_t*)ix->cnt.p, ix->nlist, nullptr, nullptr, nullptr,
                                    s));
        at = mark(ix, timed, s);
        span(ix, kRank, r0, at);
        if ((st = run_round(ix, sa, (int)(c * pl.n), q0, P, pl, s, timed, &at))) return st;
        items_total += c * pl.n;
        ++rounds;
      }
      HIP_TRY(hipMemcpyAsync(ix->rc_host, rc, sizeof(RoundCounters), hipMemcpyDeviceToHost, s));
      HIP_TRY(hipStreamSynchronize(s));
      at = -1;  // the copy ran after the last event
      if (ix->rc_host->sched_error)
        return fail(SIEVE_EINTERNAL, "a chunk's tiles exceeded the tile buffer");
      sm.rank_error = ix->rc_host->rank_error;
      sm.heavy = ix->rc_host->heavy;
      sm.hits = ix->rc_host->hits;
    }
    if (sm.rank_error) {
      // a query's rank candidates overflowed: first with the first pass over
      // every centroid (the tight bound), then with the wide buffers
      if (pl.rank_div > 1 && !pl.wide_rank) {
        pl.rank_div = 1;
        continue;
      }
      if (pl.wide_rank)
        return fail(SIEVE_EUNSUPPORTED,
                    "more than %d centroids tie within the fp32 screening bound at a rank "
                    "boundary", kMaxCand);
      pl.wide_rank = true;  // a rank boundary overflowed the narrow buffer: run again
      continue;
    }

    // Overflowed (tile, query) groups: the exact top-k pass appends their
    // candidates to the pool.  A record buffer too small for them grows, and
    // the search runs again (it is deterministic).
    const int64_t n_heavy = sm.heavy;
    if (n_heavy > ix->heavy_cap) {
      ix->heavy_cap = n_heavy + n_heavy / 4 + 1024;
      if ((st = ensure(ix->heavy, (size_t)ix->heavy_cap * sizeof(HeavyRec)))) return st;
      if (++pool_retries > 4) return fail(SIEVE_EINTERNAL, "overflow records kept overflowing");
      continue;
    }
    const int f0 = at >= 0 ? at : mark(ix, timed, s);
    unsigned long long pool_n = sm.hits;
    if (n_heavy > 0 && pool_n <= (unsigned long long)ix->pool_cap) {
      HeavyArgs ha;
      ha.vectors = ix->vectors;
      ha.vfrag = ix->vfrag;
      ha.ids = ix->ids;
      ha.queries = queries;
      ha.recs = (const HeavyRec*)ix->heavy.p;
      ha.nrec = (int32_t)n_heavy;
      ha.d = ix->d;
      ha.k = pl.k;
      ha.pack_rank = sa.hitbits != nullptr ? 1 : 0;
      ha.tau = pl.tau;
      ha.hcount = (int32_t*)ix->hcount.p;
      ha.pool = (Hit*)ix->pool.p;
      ha.pool_count = &rc->hits;
      ha.pool_cap = ix->pool_cap;
      const int grid = (int)std::min<int64_t>(n_heavy, (int64_t)ix->cus * 16);
      HIP_TRY(launch_scan_heavy(ix->dtype, ha, grid, s));
      HIP_TRY(hipMemcpyAsync(&ix->rc_host->hits, &rc->hits, sizeof(unsigned long long),
                             hipMemcpyDeviceToHost, s));
      HIP_TRY(hipStreamSynchronize(s));
      pool_n = ix->rc_host->hits;
    }
    const int64_t hits = (int64_t)pool_n;
    const int64_t limit = pool_index_limit(getenv("SIEVE_POOL_LIMIT"));
    if (!pool_slots_fit(pool_n, limit))
      return fail(SIEVE_EUNSUPPORTED,
                  "the search wrote %llu candidate-pool entries; the final merge takes at "
                  "most %lld", pool_n, (long long)limit);
    if (hits > ix->pool_cap) {
      // the pool overflowed: grow it and run again (the search is deterministic)
      ix->pool_cap = hits + hits / 8 + 4096;
      if ((st = ensure(ix->pool, (size_t)ix->pool_cap * sizeof(Hit)))) return st;
      if ((st = ensure(ix->pool_sorted, (size_t)ix->pool_cap * sizeof(Hit)))) return st;
      if (++pool_retries > 4) return fail(SIEVE_EINTERNAL, "candidate pool kept overflowing");
      continue;
    }

    // finalize: group the pool by query, then per-query top-k
    HIP_TRY(launch_exclusive_scan((const int32_t*)ix->hcount.p, (int64_t*)ix->hoff.p,
                                  (int64_t*)ix->hcur.p, nq, (int64_t*)ix->scan_tmp.p, s));
    HIP_TRY(launch_pool_scatter((const Hit*)ix->pool.p, hits, (int64_t*)ix->hcur.p,
                                (Hit*)ix->pool_sorted.p, cal != nullptr || spec_used, s));
    const int32_t* probes_src = pl.mode == 0   ? (const int32_t*)ix->state_a.p
                                : pl.mode == 1 ? (const int32_t*)ix->state_b.p
                                               : nullptr;
    HIP_TRY(launch_topk(nq, pl.k, (const Hit*)ix->pool_sorted.p, (const int64_t*)ix->hoff.p,
                        (const int32_t*)ix->hcount.p, probes_src, pl.n, out_map, out_ids,
                        out_scores, out_probes, cal ? cal->frank : nullptr,
                        spec_used ? (const int32_t*)ix->state_a.p : nullptr, rc, s));
    const int f1 = mark(ix, timed, s);
    span(ix, kFinal, f0, f1);
    span(ix, kTotal, t_begin, f1);
    // the statistics read the final counters; the outputs only need the stream drained
    if (timed)
      HIP_TRY(hipMemcpyAsync(ix->rc_host, rc, sizeof(RoundCounters), hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    if (timed) {
      float ms[kPhases];
      int scan_launches = 0;
      read_timeline(ix, ms, &scan_launches);
      if ((st = finish_round_log(ix, pl.mode == 2 ? 1 : 0, s))) return st;
      const RoundCounters& h = *ix->rc_host;
      unsigned long long probes_sum = 0, cand_sum = 0;
      for (int x = 0; x < kStatSlots; ++x) {
        probes_sum += h.probes[x];
        cand_sum += h.candidates[x];
      }
      const double eb = (double)ix->d * e;
      stats->rounds = rounds;
      stats->nprobe_eff = pl.n;
      stats->scan_launches = scan_launches;
      stats->pool_retries = pool_retries;
      stats->items = items_total;
      stats->probes_total = (int64_t)probes_sum;
      stats->vectors_scanned = (int64_t)h.item_rows;
      stats->list_loads = (int64_t)h.list_loads;
      stats->hits = (int64_t)h.cands;
      stats->pool_entries = (int64_t)cand_sum;
      stats->heavy_records = (int64_t)h.heavy;
      stats->scan_bytes = (double)h.list_rows * eb + (double)items_total * (eb + sizeof(Item)) +
                          (double)cand_sum * sizeof(Hit);
      stats->scan_flops = 2.0 * (double)ix->d * (double)h.item_rows;
      stats->rank_flops = 2.0 * (double)ix->d * (double)nq * (double)ix->nlist;
      stats->ms_rank = ms[kRank];
      stats->ms_sched = ms[kSched];
      stats->ms_scan = ms[kScan];
      stats->ms_update = ms[kUpdate];
      stats->ms_finalize = ms[kFinal];
      stats->ms_total = ms[kTotal];
    }
    return SIEVE_OK;
  }
}

// mode: 0 lookahead (Algorithm 2), 1 basic (Algorithm 1), 2 fixed probing.
// speculative: with mode 0, also issue ranks past the stop line (see
// launch_update_lookahead); outputs are the same either way.
int plan_search(const sieve_index* ix, int64_t nq, int32_t k, float tau, int32_t W,
                int32_t nprobe, int mode, bool speculative, SearchPlan* pl) {
  pl->n = nprobe < ix->nlist ? nprobe : ix->nlist;
  if (pl->n > kMaxRanks)
    return fail(SIEVE_EUNSUPPORTED, "min(nprobe, nlist) = %d exceeds %d", pl->n, kMaxRanks);
  pl->mode = mode;
  pl->W = W;
  pl->k = k;
  pl->tau = tau;
  pl->nq = nq;
  // default on where supported; SIEVE_SCAN_WIDE=2 turns it off (tuning only)
  pl->wide = scan_wide_supported(ix->dtype, ix->d) && env_int("SIEVE_SCAN_WIDE", 1) == 1;
  pl->rega = scan_uses_rega(ix->dtype, ix->d);
  pl->tile_q = pl->wide   ? tile_rows_wide(ix->dtype, ix->d)
               : pl->rega ? scan_rega_tile_q(true)
                          : tile_rows(ix->dtype, ix->d);
  pl->group_q = pl->tile_q;
  pl->min_group = pl->rega ? scan_rega_tile_q(false) : pl->tile_q;
  pl->wide_rank = false;
  // the register-query prefix ranking bounds the R-th score from the first
  // half of the centroids (any subset's R-th largest score is a valid lower
  // bound); a query whose candidates then overflow re-ranks with the full pass
  pl->rank_div = env_int("SIEVE_RANK_PASS1_DIV", 2);
  // sparse rounds: 1,024-row tiles for register-held queries (a tile's start
  // drains its row ring once), else 512
  pl->row_chunk = row_chunk_for(ix, "SIEVE_ROW_CHUNK", pl->rega ? 1024 : 512);
  // Dense rounds over short lists (at most 2048 rows on average) take whole
  // lists as one tile, which halves the tile starts of a 1,000-row list; with
  // long lists 1,024-row tiles measured fastest.
  const int64_t avg_len = ix->n / ix->nlist;
  // Register-held queries make a tile's start cheap, so dense rounds take
  // whole lists; otherwise the query staging favours 512-row tiles on long
  // lists.
  const int whole = (int)std::min<int64_t>(std::max<int64_t>(ix->max_list, 64), INT32_MAX / 2);
  pl->row_chunk_dense = row_chunk_for(
      ix, "SIEVE_ROW_CHUNK_DENSE",
      scan_uses_rega(ix->dtype, ix->d) ? whole : (avg_len <= 2048 ? 4096 : 1024));
  if (pl->row_chunk_dense < pl->row_chunk) pl->row_chunk_dense = pl->row_chunk;
  pl->dense_q = env_int("SIEVE_DENSE_Q", 64);
  // Speculative issue needs the rank packed beside the query in pool entries
  // (queries < 2^kRankShift) and a stop rule that can stop early (W < n).
  pl->spec = speculative && mode == 0 && W < pl->n && nq <= (int64_t)kQueryMask + 1;
  pl->spec_max =
      pl->spec ? (int)std::min<int64_t>(pl->n, (int64_t)env_int("SIEVE_SPEC_DEPTH", 3) * W) : 0;
  // Lines that move far keep moving (queries in large near-duplicate groups):
  // speculating for those merges their next ranks into the larger, earlier
  // rounds, where a list read serves more queries.  Short moves are common
  // and mostly final; speculating there reads extra lists for nothing.
  pl->spec_round = env_count("SIEVE_SPEC_ROUND", 0);
  pl->spec_min = env_int("SIEVE_SPEC_MIN", std::max(1, W / 2));
  pl->hit_words = (pl->n + 31) / 32;
  pl->scan_grid = pl->wide ? ((ix->cus + 7) / 8) * 8 : scan_grid(ix, pl->tile_q);
  // Lazy ranking: a stop line starts at min(W, n) and mostly stays near it,
  // so only the first r0 ranks are ordered up front (queries whose stop line
  // passes r0 get all n later).
  const int64_t r0 = env_int("SIEVE_RANK_PREFIX", 32);
  const int64_t w2 = 2 * (int64_t)W;
  pl->r0 = mode == 2 || (int64_t)W >= pl->n ? pl->n
                                           : (int)std::min<int64_t>(pl->n, std::max(r0, w2));
  int64_t rc = (int64_t)(256ll << 20) / ((int64_t)ix->nlist * 4);
  if (rc < 64) rc = 64;
  pl->rank_chunk = nq < rc ? nq : rc;
  if (pl->rank_chunk < 1) pl->rank_chunk = 1;
  if (mode == 2) {
    int64_t fc = (int64_t)(64ll << 20) / pl->n;  // <= 64M items per chunk
    if (fc < 1) fc = 1;
    pl->fix_chunk = nq < fc ? nq : fc;
    if (pl->fix_chunk < 1) pl->fix_chunk = 1;
    pl->item_cap = pl->fix_chunk * pl->n;
    if (pl->rank_chunk > pl->fix_chunk) pl->rank_chunk = pl->fix_chunk;
  } else {
    pl->fix_chunk = 0;
    const int s0 = mode == 0 ? (W < pl->n ? W : pl->n) : 1;
    // A lookahead update issues at most W ranks up to the new stop line
    // (every line comes from a hit below the old one) and, speculating, at
    // most spec_max more past it.
    pl->item_cap = nq * (int64_t)std::min<int64_t>(pl->n, (int64_t)s0 + pl->spec_max);
    if (pl->item_cap > INT32_MAX)
      return fail(SIEVE_EUNSUPPORTED, "nq * min(W, n) = %lld exceeds int32", (long long)pl->item_cap);
  }
  if (pl->item_cap < 1) pl->item_cap = 1;
  return SIEVE_OK;
}

// Round structure of a lookahead argument: 0 for Algorithm 2 (with or
// without speculative issue), 1 for Algorithm 1's one rank per round.
int lookahead_mode(int32_t lookahead) {
  return lookahead == SIEVE_LOOKAHEAD_COMMITTED || lookahead == SIEVE_LOOKAHEAD_SPECULATIVE ? 0
                                                                                            : 1;
}

void add_stats(sieve_stats* acc, const sieve_stats& x) {
  acc->rounds += x.rounds;
  acc->scan_launches += x.scan_launches;
  acc->pool_retries += x.pool_retries;
  acc->items += x.items;
  acc->probes_total += x.probes_total;
  acc->vectors_scanned += x.vectors_scanned;
  acc->list_loads += x.list_loads;
  acc->hits += x.hits;
  acc->pool_entries += x.pool_entries;
  acc->heavy_records += x.heavy_records;
  acc->scan_bytes += x.scan_bytes;
  acc->scan_flops += x.scan_flops;
  acc->rank_flops += x.rank_flops;
  acc->ms_rank += x.ms_rank;
  acc->ms_sched += x.ms_sched;
  acc->ms_scan += x.ms_scan;
  acc->ms_update += x.ms_update;
  acc->ms_finalize += x.ms_finalize;
  acc->ms_total += x.ms_total;
}

}  // namespace

extern "C" {

SIEVE_API const char* sieve_last_error(void) { return g_err.c_str(); }

SIEVE_API const char* sieve_version(void) { return "sieve-mi355x 0.1 (gfx950)"; }

SIEVE_API int sieve_load_index(const void* vectors, int32_t dtype, int64_t n, int32_t d,
                               const int64_t* list_offsets, int32_t nlist, const int64_t* ids,
                               const void* centroids, void* stream, sieve_index** out) {
  g_err.clear();
  if (!out) return fail(SIEVE_EINVAL, "out is NULL");
  if (dtype != SIEVE_F32 && dtype != SIEVE_F16) return fail(SIEVE_EINVAL, "bad dtype %d", dtype);
  if (n < 0) return fail(SIEVE_EINVAL, "n = %lld is negative", (long long)n);
  if (d < 1 || nlist < 1) return fail(SIEVE_EINVAL, "d and nlist must be >= 1");
  if (!list_offsets || !centroids || (n > 0 && (!vectors || !ids)))
    return fail(SIEVE_EINVAL, "a required pointer is NULL");
  if (d % 8 != 0 || d > kMaxD)
    return fail(SIEVE_EUNSUPPORTED, "d = %d: must be a multiple of 8 and <= %d", d, kMaxD);
  // a 16-query tile of fp32 rows must fit the scan's LDS
  if (dtype == SIEVE_F32 && d > kMaxD / 2)
    return fail(SIEVE_EUNSUPPORTED, "d = %d: fp32 rows must have at most %d dimensions", d,
                kMaxD / 2);
  if (nlist > kMaxNlist) return fail(SIEVE_EUNSUPPORTED, "nlist = %d exceeds %d", nlist, kMaxNlist);
  if ((n > 0 && !aligned16(vectors)) || !aligned16(centroids) || !aligned16(list_offsets) ||
      (n > 0 && !aligned16(ids)))
    return fail(SIEVE_EINVAL, "arrays must be 16-byte aligned");
  hipStream_t s = (hipStream_t)stream;
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  std::vector<int64_t> off(nlist + 1);
  HIP_TRY(hipMemcpyAsync(off.data(), list_offsets, sizeof(int64_t) * (nlist + 1),
                         hipMemcpyDeviceToHost, s));
  HIP_TRY(hipStreamSynchronize(s));
  if (off[0] != 0 || off[nlist] != n)
    return fail(SIEVE_EINVAL, "list_offsets must start at 0 and end at n");
  int64_t max_list = 0;
  for (int c = 0; c < nlist; ++c) {
    const int64_t len = off[c + 1] - off[c];
    if (len < 0) return fail(SIEVE_EINVAL, "list_offsets decrease at list %d", c);
    if (len > INT32_MAX / 2) return fail(SIEVE_EUNSUPPORTED, "list %d is too long", c);
    if (len > max_list) max_list = len;
  }
  const int e = elem_bytes(dtype);
  sieve_index* ix = new sieve_index();
  ix->dtype = dtype;
  ix->n = n;
  ix->d = d;
  ix->nlist = nlist;
  ix->device = dev;
  ix->h_offsets = off;
  ix->max_list = max_list;
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, dev) == hipSuccess && prop.multiProcessorCount > 0)
    ix->cus = prop.multiProcessorCount;
  auto bail = [&](int code) {
    sieve_free_index(ix);
    return code;
  };
  const size_t vbytes = (size_t)n * d * e, cbytes = (size_t)nlist * d * e;
  const size_t fbytes = centroid_frag_bytes(dtype, d, nlist);
  // partitions padded to whole 16-row blocks in the fragment-order copy
  std::vector<int64_t> hfoff(nlist + 1, 0);
  for (int l = 0; l < nlist; ++l) hfoff[l + 1] = hfoff[l] + (off[l + 1] - off[l] + 15) / 16 * 16;
  const size_t vfbytes = vector_frag_bytes(dtype, d, hfoff[nlist]);
  // the partition starts are read for every tile of a compile-time dimension,
  // also when the store is empty (then no row is)
  const bool vfixed = vector_frag_bytes(dtype, d, 16) > 0;
  hipError_t err;
  if ((err = hipMalloc(&ix->vectors, vbytes ? vbytes : 16)) != hipSuccess ||
      (err = hipMalloc((void**)&ix->offsets, sizeof(int64_t) * (nlist + 1))) != hipSuccess ||
      (err = hipMalloc((void**)&ix->ids, n > 0 ? sizeof(int64_t) * n : 16)) != hipSuccess ||
      (err = hipMalloc(&ix->centroids, cbytes)) != hipSuccess ||
      (fbytes && (err = hipMalloc(&ix->cfrag, fbytes)) != hipSuccess) ||
      (vfbytes && (err = hipMalloc(&ix->vfrag, vfbytes)) != hipSuccess) ||
      (vfixed && (err = hipMalloc((void**)&ix->foff, sizeof(int64_t) * (nlist + 1))) != hipSuccess)) {
    (void)hipGetLastError();
    return bail(fail(SIEVE_ENOMEM, "index allocation failed: %s", hipGetErrorString(err)));
  }
  if ((vbytes && (err = hipMemcpyAsync(ix->vectors, vectors, vbytes, hipMemcpyDeviceToDevice, s)) != hipSuccess) ||
      (err = hipMemcpyAsync(ix->offsets, list_offsets, sizeof(int64_t) * (nlist + 1), hipMemcpyDeviceToDevice, s)) != hipSuccess ||
      (n > 0 && (err = hipMemcpyAsync(ix->ids, ids, sizeof(int64_t) * n, hipMemcpyDeviceToDevice, s)) != hipSuccess) ||
      (err = hipMemcpyAsync(ix->centroids, centroids, cbytes, hipMemcpyDeviceToDevice, s)) != hipSuccess ||
      (fbytes && (err = launch_centroid_frag(dtype, d, ix->centroids, nlist, ix->cfrag, s)) != hipSuccess) ||
      (vfixed && (err = hipMemcpyAsync(ix->foff, hfoff.data(), sizeof(int64_t) * (nlist + 1),
                                        hipMemcpyHostToDevice, s)) != hipSuccess) ||
      (vfbytes && (err = launch_vector_frag(dtype, d, ix->vectors, ix->offsets, ix->foff, nlist,
                                            hfoff[nlist], ix->vfrag, s)) != hipSuccess))
    return bail(fail(SIEVE_EDEVICE, "index copy failed: %s", hipGetErrorString(err)));
  std::vector<uint8_t> hc(cbytes);
  if ((err = hipMemcpyAsync(hc.data(), centroids, cbytes, hipMemcpyDeviceToHost, s)) != hipSuccess ||
      (err = hipStreamSynchronize(s)) != hipSuccess)
    return bail(fail(SIEVE_EDEVICE, "index copy failed: %s", hipGetErrorString(err)));
  double cmax = 0.0;
  for (int c = 0; c < nlist; ++c) {
    double ss = 0.0;
    for (int t = 0; t < d; ++t) {
      const double v = host_elem(hc.data(), dtype, (int64_t)c * d + t);
      ss += v * v;
    }
    if (ss > cmax) cmax = ss;
  }
  ix->cmax = sqrt(cmax) * (1.0 + 1e-12);
  if (!isfinite(ix->cmax)) return bail(fail(SIEVE_EINVAL, "centroids contain inf or NaN"));
  *out = ix;
  return SIEVE_OK;
}

SIEVE_API void sieve_free_index(sieve_index* ix) {
  if (!ix) return;
#define SIEVE_FREE_BUF(name) \
  if (ix->name.p) (void)hipFree(ix->name.p);
  SIEVE_WORKSPACE(SIEVE_FREE_BUF)
#undef SIEVE_FREE_BUF
  if (ix->vectors) (void)hipFree(ix->vectors);
  if (ix->offsets) (void)hipFree(ix->offsets);
  if (ix->ids) (void)hipFree(ix->ids);
  if (ix->centroids) (void)hipFree(ix->centroids);
  if (ix->cfrag) (void)hipFree(ix->cfrag);
  if (ix->vfrag) (void)hipFree(ix->vfrag);
  if (ix->foff) (void)hipFree(ix->foff);
  if (ix->rc_host) (void)hipHostFree(ix->rc_host);
  if (ix->rs_host) (void)hipHostFree(ix->rs_host);
  for (hipEvent_t e : ix->ev_pool) (void)hipEventDestroy(e);
  delete ix;
}

SIEVE_API int sieve_search(const sieve_index* idx, const void* queries, int64_t nq,
                           const int64_t* exclude_ids, int32_t k, float tau, int32_t W,
                           int32_t nprobe_max, int32_t lookahead, int64_t* out_ids,
                           float* out_scores, int32_t* out_probes, sieve_stats* stats,
                           void* stream) {
  g_err.clear();
  int st = check_common(idx, queries, nq, k, tau, out_ids, out_scores, out_probes);
  if (st) return st;
  if (W < 1) return fail(SIEVE_EINVAL, "W = %d must be >= 1", W);
  if (nprobe_max < 1) return fail(SIEVE_EINVAL, "nprobe_max = %d must be >= 1", nprobe_max);
  if (lookahead < SIEVE_LOOKAHEAD_OFF || lookahead > SIEVE_LOOKAHEAD_SPECULATIVE)
    return fail(SIEVE_EINVAL, "lookahead = %d must be 0, 1, 2 or 3", lookahead);
  sieve_index* ix = const_cast<sieve_index*>(idx);
  SearchPlan pl;
  if ((st = plan_search(ix, nq, k, tau, W, nprobe_max, lookahead_mode(lookahead),
                        lookahead == SIEVE_LOOKAHEAD_SPECULATIVE, &pl)))
    return st;
  if (lookahead == SIEVE_LOOKAHEAD_SERIAL) pl.group_q = 1;  // no query shares a partition scan
  if (stats) memset(stats, 0, sizeof(*stats));
  if (nq == 0) {
    if (stats) stats->nprobe_eff = pl.n;
    return SIEVE_OK;
  }
  return search_impl(ix, queries, nq, exclude_ids, pl, nullptr, out_ids, out_scores, out_probes,
                     stats, (hipStream_t)stream);
}

SIEVE_API int sieve_round_log(const sieve_index* idx, sieve_round* out, int32_t max,
                              int32_t* n_rounds) {
  g_err.clear();
  if (!idx || !n_rounds) return fail(SIEVE_EINVAL, "idx and n_rounds must be non-NULL");
  if (max < 0 || (max > 0 && !out)) return fail(SIEVE_EINVAL, "bad output array");
  const int n = (int)idx->rounds_log.size();
  for (int r = 0; r < n && r < max; ++r) out[r] = idx->rounds_log[(size_t)r];
  *n_rounds = idx->rounds_logged;
  return SIEVE_OK;
}

SIEVE_API int sieve_rank(const sieve_index* idx, const void* queries, int64_t nq, int32_t nprobe,
                         int32_t* out_order, void* stream) {
  g_err.clear();
  if (!idx) return fail(SIEVE_EINVAL, "index handle is NULL");
  if (nq < 0) return fail(SIEVE_EINVAL, "nq is negative");
  if (nprobe < 1) return fail(SIEVE_EINVAL, "nprobe = %d must be >= 1", nprobe);
  if (nq > 0 && (!queries || !out_order))
    return fail(SIEVE_EINVAL, "queries and out_order must be non-NULL when nq > 0");
  if (nq > 0 && !aligned16(queries)) return fail(SIEVE_EINVAL, "queries must be 16-byte aligned");
  if (nq > (int64_t)INT32_MAX / 2) return fail(SIEVE_EUNSUPPORTED, "nq too large");
  sieve_index* ix = const_cast<sieve_index*>(idx);
  SearchPlan pl;
  int st;
  if ((st = plan_search(ix, nq, 1, 0.f, 1, nprobe, 1, false, &pl))) return st;
  if (nq == 0) return SIEVE_OK;
  if ((int64_t)nq * pl.n > (int64_t)INT32_MAX * 8)
    return fail(SIEVE_EUNSUPPORTED, "nq * nprobe too large");
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  if (dev != ix->device) return fail(SIEVE_EINVAL, "current device differs from the index's");
  hipStream_t s = (hipStream_t)stream;
  if ((st = ensure(ix->scores, (size_t)pl.rank_chunk * ix->nlist * sizeof(float)))) return st;
  if ((st = ensure(ix->rc, sizeof(RoundCounters)))) return st;
  if (!ix->rc_host) HIP_TRY(hipHostMalloc((void**)&ix->rc_host, sizeof(RoundCounters), 0));
  RoundCounters* rc = (RoundCounters*)ix->rc.p;
  const int div0 = pl.rank_div;
  for (int attempt = 0; attempt < 3; ++attempt) {
    // the first pass over a subset, then over every centroid, then wide buffers
    if (attempt == 1 && div0 <= 1) continue;
    pl.rank_div = attempt == 0 ? div0 : 1;
    pl.wide_rank = attempt == 2;
    HIP_TRY(launch_zero_bytes(rc, sizeof(RoundCounters), s));
    if ((st = rank_queries(ix, queries, 0, nq, pl.n, pl.n, pl, out_order, s))) return st;
    HIP_TRY(hipMemcpyAsync(ix->rc_host, rc, sizeof(RoundCounters), hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    if (!ix->rc_host->rank_error) return SIEVE_OK;
  }
  return fail(SIEVE_EUNSUPPORTED,
              "more than %d centroids tie within the fp32 screening bound at a rank boundary",
              kMaxCand);
}

// ---- allocation-free ranking ---------------------------------------------
// The workspace of sieve_rank_noalloc: a fixed device array, one copy per
// GPU the library runs on, held until the process ends.  Every call on a GPU
// uses that GPU's copy; calls that overlap in time on one GPU (other streams,
// other threads) race on it.  In host code `scratch` only names the symbol:
// kernels get its device address, looked up once per device.
constexpr size_t kScratchBytes = size_t(64) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices] = {};

// Device address of this device's scratch (dev must be current).
int scratch_address(int dev, unsigned char** out) {
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (dev < 0 || dev >= kMaxScratchDevices)
    return fail(SIEVE_EUNSUPPORTED, "device %d: the allocation-free entry point supports "
                "devices 0..%d", dev, kMaxScratchDevices - 1);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(SIEVE_EDEVICE, "no device address for the scratch array");
    g_scratch_ptr[dev] = p;
  }
  *out = (unsigned char*)g_scratch_ptr[dev];
  return SIEVE_OK;
}
}  // namespace

SIEVE_API int sieve_rank_noalloc(const sieve_index* idx, const void* queries, int64_t nq,
                                 int32_t nprobe, int32_t* out_order, void* stream) {
  g_err.clear();
  if (!idx) return fail(SIEVE_EINVAL, "index handle is NULL");
  if (nq < 0) return fail(SIEVE_EINVAL, "nq is negative");
  if (nprobe < 1) return fail(SIEVE_EINVAL, "nprobe = %d must be >= 1", nprobe);
  if (nq > 0 && (!queries || !out_order))
    return fail(SIEVE_EINVAL, "queries and out_order must be non-NULL when nq > 0");
  if (nq > 0 && !aligned16(queries)) return fail(SIEVE_EINVAL, "queries must be 16-byte aligned");
  if (nq > (int64_t)INT32_MAX / 2) return fail(SIEVE_EUNSUPPORTED, "nq too large");
  const sieve_index* ix = idx;
  SearchPlan pl;
  int st;
  if ((st = plan_search(ix, nq, 1, 0.f, 1, nprobe, 1, false, &pl))) return st;
  if (nq == 0) return SIEVE_OK;
  if ((int64_t)nq * pl.n > (int64_t)INT32_MAX * 8)
    return fail(SIEVE_EUNSUPPORTED, "nq * nprobe too large");
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  if (dev != ix->device) return fail(SIEVE_EINVAL, "current device differs from the index's");
  unsigned char* base = nullptr;
  if ((st = scratch_address(dev, &base))) return st;
  hipStream_t s = (hipStream_t)stream;
  // scratch layout: the round counters, then the ranking workspace
  constexpr size_t kHead = (sizeof(RoundCounters) + 255) & ~size_t(255);
  RoundCounters* rc = (RoundCounters*)base;
  unsigned char* ws = base + kHead;
  const size_t ws_bytes = kScratchBytes - kHead;
  const int div0 = pl.rank_div;
  for (int attempt = 0; attempt < 3; ++attempt) {
    // the first pass over a subset, then over every centroid, then wide buffers
    if (attempt == 1 && div0 <= 1) continue;
    pl.rank_div = attempt == 0 ? div0 : 1;
    pl.wide_rank = attempt == 2;
    // queries per chunk that fit the workspace
    unsigned long long* cand = nullptr;
    int32_t* ccount = nullptr;
    float* scores = nullptr;
    int64_t chunk_prefix = 1, chunk_scores = 1;
    if (use_prefix_path(ix, pl.n, pl.wide_rank)) {
      const size_t per = (size_t)rank_prefix_cap(pl.n, ix->nlist) * sizeof(unsigned long long) +
                         sizeof(int32_t);
      const int64_t fit = (int64_t)((ws_bytes - 256) / per);
      if (fit < 1)
        return fail(SIEVE_EUNSUPPORTED, "one query's ranking workspace (%zu bytes) exceeds the "
                    "%zu-byte scratch of the allocation-free entry point", per, ws_bytes - 256);
      chunk_prefix = std::min<int64_t>({fit, nq, int64_t(1) << 18});
      cand = (unsigned long long*)ws;
      ccount = (int32_t*)(ws + (((size_t)chunk_prefix * rank_prefix_cap(pl.n, ix->nlist) *
                                 sizeof(unsigned long long) + 255) & ~size_t(255)));
    } else {
      const size_t per = (size_t)ix->nlist * sizeof(float);
      const int64_t fit = (int64_t)(ws_bytes / per);
      if (fit < 1)
        return fail(SIEVE_EUNSUPPORTED, "one query's ranking workspace (%zu bytes) exceeds the "
                    "%zu-byte scratch of the allocation-free entry point", per, ws_bytes);
      chunk_scores = std::min<int64_t>({fit, nq, pl.rank_chunk});
      scores = (float*)ws;
    }
    HIP_TRY(launch_zero_bytes(rc, sizeof(RoundCounters), s));
    if ((st = rank_queries_in(ix, queries, 0, nq, pl.n, pl.n, pl, out_order, rc, cand, ccount,
                              chunk_prefix, scores, chunk_scores, s)))
      return st;
    int32_t rank_error = 0;  // pageable host memory: the copy allocates nothing here
    HIP_TRY(hipMemcpyAsync(&rank_error, &rc->rank_error, sizeof(rank_error),
                           hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    if (!rank_error) return SIEVE_OK;
  }
  return fail(SIEVE_EUNSUPPORTED,
              "more than %d centroids tie within the fp32 screening bound at a rank boundary",
              kMaxCand);
}

SIEVE_API int sieve_search_fixed(const sieve_index* idx, const void* queries, int64_t nq,
                                 const int64_t* exclude_ids, int32_t k, float tau, int32_t nprobe,
                                 int64_t* out_ids, float* out_scores, int32_t* out_probes,
                                 sieve_stats* stats, void* stream) {
  g_err.clear();
  int st = check_common(idx, queries, nq, k, tau, out_ids, out_scores, out_probes);
  if (st) return st;
  if (nprobe < 1) return fail(SIEVE_EINVAL, "nprobe = %d must be >= 1", nprobe);
  sieve_index* ix = const_cast<sieve_index*>(idx);
  SearchPlan pl;
  if ((st = plan_search(ix, nq, k, tau, SIEVE_W_INF, nprobe, 2, false, &pl))) return st;
  if (stats) memset(stats, 0, sizeof(*stats));
  if (nq == 0) {
    if (stats) stats->nprobe_eff = pl.n;
    return SIEVE_OK;
  }
  return search_impl(ix, queries, nq, exclude_ids, pl, nullptr, out_ids, out_scores, out_probes,
                     stats, (hipStream_t)stream);
}

}  // extern "C"

namespace {
// The calibrated search of one index (arguments checked by the caller):
// stats, if given, are added to (the caller zeroes them).
int calibrated_impl(sieve_index* ix, const void* queries, int64_t nq, const int64_t* exclude_ids,
                    int32_t k, float tau, int32_t nprobe_max, const int32_t* sample, int64_t ns,
                    float eps, int32_t W_fallback, int64_t* out_ids, float* out_scores,
                    int32_t* out_probes, int32_t* out_W, sieve_stats* stats, hipStream_t s) {
  int st;
  SearchPlan pf;
  if ((st = plan_search(ix, ns, k, tau, SIEVE_W_INF, nprobe_max, 2, false, &pf))) return st;
  if (stats) stats->nprobe_eff = pf.n;
  if (nq == 0) {
    *out_W = W_fallback;
    return SIEVE_OK;
  }
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  if (dev != ix->device)
    return fail(SIEVE_EINVAL, "current device %d differs from the index's device %d", dev,
                ix->device);
  const int64_t nr = nq - ns;
  const int64_t row_bytes = (int64_t)ix->d * elem_bytes(ix->dtype);

  // Output rows: the sample as given, then every other query in order.
  std::vector<int32_t> rows((size_t)nq);
  if (ns > 0) {
    HIP_TRY(hipMemcpyAsync(rows.data(), sample, (size_t)ns * 4, hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    std::vector<uint8_t> seen((size_t)nq, 0);
    for (int64_t i = 0; i < ns; ++i) {
      const int32_t q = rows[(size_t)i];
      if (q < 0 || q >= nq)
        return fail(SIEVE_EINVAL, "sample[%lld] = %d outside [0, nq)", (long long)i, q);
      if (seen[(size_t)q]) return fail(SIEVE_EINVAL, "sample index %d appears twice", q);
      seen[(size_t)q] = 1;
    }
    int64_t j = ns;
    for (int64_t q = 0; q < nq; ++q)
      if (!seen[(size_t)q]) rows[(size_t)j++] = (int32_t)q;
  }
  const int64_t gather_rows = ns > 0 ? std::max(ns, nr) : 0;
  if ((st = ensure(ix->cal_idx, (size_t)nq * 4)) ||
      (st = ensure(ix->cal_q, (size_t)gather_rows * row_bytes)) ||
      (exclude_ids && (st = ensure(ix->cal_x, (size_t)gather_rows * 8))))
    return st;
  if (ns > 0)
    HIP_TRY(hipMemcpyAsync(ix->cal_idx.p, rows.data(), (size_t)nq * 4, hipMemcpyHostToDevice, s));
  const int32_t* d_rows = (const int32_t*)ix->cal_idx.p;
  void* gq = ix->cal_q.p;
  int64_t* gx = exclude_ids ? (int64_t*)ix->cal_x.p : nullptr;

  // 1. Fixed-probe search of the sample, recording per-rank outcomes.
  int W = W_fallback;
  sieve_stats part;
  if (ns > 0) {
    const int32_t words = (pf.n + 31) / 32;
    if ((st = ensure(ix->cal_bits, (size_t)ns * words * 4)) ||
        (st = ensure(ix->cal_rank, (size_t)ns * k * 4)) ||
        (st = ensure(ix->cal_hist, (size_t)(pf.n + 3) * 8)))
      return st;
    HIP_TRY(launch_gather_rows(d_rows, (int32_t)ns, queries, row_bytes, gq, s));
    if (gx) HIP_TRY(launch_gather_i64(d_rows, ns, exclude_ids, gx, s));
    const CalibOut co = {(uint32_t*)ix->cal_bits.p, words, (int32_t*)ix->cal_rank.p};
    if ((st = search_impl(ix, gq, ns, gx, pf, d_rows, out_ids, out_scores, out_probes,
                          stats ? &part : nullptr, s, &co)))
      return st;
    if (stats) add_stats(stats, part);
    // 2. Replay the stop rule over the recorded outcomes; choose W.
    //    cal_hist: H[0..n], then the neighbour count Z, then the chosen W.
    unsigned long long* hist = (unsigned long long*)ix->cal_hist.p;
    unsigned long long* z = hist + pf.n + 1;
    int32_t* d_w = (int32_t*)(hist + pf.n + 2);
    HIP_TRY(launch_zero_bytes(hist, (int64_t)(pf.n + 3) * 8, s));
    HIP_TRY(launch_calib_replay(ns, pf.n, k, co.hitbits, words, co.frank, hist, z, s));
    HIP_TRY(launch_calib_choose(pf.n, eps, hist, z, d_w, s));
    int32_t w = 0;
    HIP_TRY(hipMemcpyAsync(&w, d_w, 4, hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    if (w > 0) W = w;
  }
  *out_W = W;

  // 3. Lookahead search of every other query with the chosen window.
  if (nr > 0) {
    SearchPlan pr;
    if ((st = plan_search(ix, nr, k, tau, W, nprobe_max, 0, false, &pr))) return st;
    if (ns == 0) {
      st = search_impl(ix, queries, nq, exclude_ids, pr, nullptr, out_ids, out_scores, out_probes,
                       stats ? &part : nullptr, s);
    } else {
      HIP_TRY(launch_gather_rows(d_rows + ns, (int32_t)nr, queries, row_bytes, gq, s));
      if (gx) HIP_TRY(launch_gather_i64(d_rows + ns, nr, exclude_ids, gx, s));
      st = search_impl(ix, gq, nr, gx, pr, d_rows + ns, out_ids, out_scores, out_probes,
                       stats ? &part : nullptr, s);
    }
    if (st) return st;
    if (stats) add_stats(stats, part);
  }
  return SIEVE_OK;
}

}  // namespace

extern "C" {

SIEVE_API int sieve_search_calibrated(const sieve_index* idx, const void* queries, int64_t nq,
                                      const int64_t* exclude_ids, int32_t k, float tau,
                                      int32_t nprobe_max, const int32_t* sample, int64_t ns,
                                      float eps, int32_t W_fallback, int64_t* out_ids,
                                      float* out_scores, int32_t* out_probes, int32_t* out_W,
                                      sieve_stats* stats, void* stream) {
  g_err.clear();
  int st = check_common(idx, queries, nq, k, tau, out_ids, out_scores, out_probes);
  if (st) return st;
  if (nprobe_max < 1) return fail(SIEVE_EINVAL, "nprobe_max = %d must be >= 1", nprobe_max);
  if (!(eps > 0.f && eps <= 1.f)) return fail(SIEVE_EINVAL, "eps = %g outside (0, 1]", (double)eps);
  if (W_fallback < 1) return fail(SIEVE_EINVAL, "W_fallback = %d must be >= 1", W_fallback);
  if (!out_W) return fail(SIEVE_EINVAL, "out_W is NULL");
  if (ns < 0 || ns > nq) return fail(SIEVE_EINVAL, "ns = %lld outside [0, nq]", (long long)ns);
  if (ns > kCalibMaxSample)
    return fail(SIEVE_EUNSUPPORTED, "ns = %lld exceeds %d", (long long)ns, kCalibMaxSample);
  if (ns > 0 && !sample) return fail(SIEVE_EINVAL, "sample is NULL with ns > 0");
  if (stats) memset(stats, 0, sizeof(*stats));
  return calibrated_impl(const_cast<sieve_index*>(idx), queries, nq, exclude_ids, k, tau,
                         nprobe_max, sample, ns, eps, W_fallback, out_ids, out_scores, out_probes,
                         out_W, stats, (hipStream_t)stream);
}

SIEVE_API int sieve_search_multi(const sieve_index* const* idxs, int32_t nidx,
                                 const void* queries, int64_t nq, const int64_t* exclude_ids,
                                 int32_t k, float tau, int32_t W, int32_t nprobe_max,
                                 int32_t lookahead, int64_t* out_ids, float* out_scores,
                                 int32_t* out_probes, sieve_stats* stats, void* stream) {
  g_err.clear();
  if (!idxs || nidx < 1 || nidx > SIEVE_MULTI_MAX)
    return fail(SIEVE_EINVAL, "idxs must hold 1 .. %d index handles", SIEVE_MULTI_MAX);
  for (int32_t i = 0; i < nidx; ++i) {
    if (!idxs[i]) return fail(SIEVE_EINVAL, "idxs[%d] is NULL", i);
    if (idxs[i]->dtype != idxs[0]->dtype || idxs[i]->d != idxs[0]->d ||
        idxs[i]->device != idxs[0]->device)
      return fail(SIEVE_EINVAL, "idxs[%d] differs from idxs[0] in dtype, d or device", i);
  }
  int st = check_common(idxs[0], queries, nq, k, tau, out_ids, out_scores, out_probes);
  if (st) return st;
  if (W < 1) return fail(SIEVE_EINVAL, "W = %d must be >= 1", W);
  if (nprobe_max < 1) return fail(SIEVE_EINVAL, "nprobe_max = %d must be >= 1", nprobe_max);
  if (lookahead < SIEVE_LOOKAHEAD_OFF || lookahead > SIEVE_LOOKAHEAD_SPECULATIVE)
    return fail(SIEVE_EINVAL, "lookahead = %d must be 0, 1, 2 or 3", lookahead);
  std::vector<SearchPlan> plans((size_t)nidx);
  for (int32_t i = 0; i < nidx; ++i) {
    sieve_index* ix = const_cast<sieve_index*>(idxs[i]);
    if ((st = plan_search(ix, nq, k, tau, W, nprobe_max, lookahead_mode(lookahead),
                          lookahead == SIEVE_LOOKAHEAD_SPECULATIVE, &plans[i])))
      return st;
    if (lookahead == SIEVE_LOOKAHEAD_SERIAL) plans[i].group_q = 1;
  }
  if (stats) memset(stats, 0, sizeof(*stats));
  if (nq == 0) return SIEVE_OK;
  hipStream_t s = (hipStream_t)stream;
  // per-index results, [nidx][nq][k], in the first index's workspace
  sieve_index* ws = const_cast<sieve_index*>(idxs[0]);
  const size_t rows = (size_t)nidx * (size_t)nq;
  if ((st = ensure(ws->mix_ids, rows * k * sizeof(int64_t))) ||
      (st = ensure(ws->mix_scores, rows * k * sizeof(float))) ||
      (st = ensure(ws->mix_probes, rows * sizeof(int32_t))))
    return st;
  int64_t* mids = (int64_t*)ws->mix_ids.p;
  float* msc = (float*)ws->mix_scores.p;
  int32_t* mpr = (int32_t*)ws->mix_probes.p;
  sieve_stats part;
  for (int32_t i = 0; i < nidx; ++i) {
    sieve_index* ix = const_cast<sieve_index*>(idxs[i]);
    const size_t r0 = (size_t)i * (size_t)nq;
    if ((st = search_impl(ix, queries, nq, exclude_ids, plans[i], nullptr, mids + r0 * k,
                          msc + r0 * k, mpr + r0, stats ? &part : nullptr, s)))
      return st;
    if (stats) add_stats(stats, part);
  }
  HIP_TRY(launch_merge_shards(nq, k, nidx, mids, msc, mpr, out_ids, out_scores, out_probes, s));
  HIP_TRY(hipStreamSynchronize(s));
  if (stats) stats->nprobe_eff = plans[0].n;
  return SIEVE_OK;
}

SIEVE_API int sieve_search_multi_calibrated(const sieve_index* const* idxs, int32_t nidx,
                                            const void* queries, int64_t nq,
                                            const int64_t* exclude_ids, int32_t k, float tau,
                                            int32_t nprobe_max, const int32_t* sample, int64_t ns,
                                            float eps, int32_t W_fallback, int64_t* out_ids,
                                            float* out_scores, int32_t* out_probes,
                                            int32_t* out_W, sieve_stats* stats, void* stream) {
  g_err.clear();
  if (!idxs || nidx < 1 || nidx > SIEVE_MULTI_MAX)
    return fail(SIEVE_EINVAL, "idxs must hold 1 .. %d index handles", SIEVE_MULTI_MAX);
  for (int32_t i = 0; i < nidx; ++i) {
    if (!idxs[i]) return fail(SIEVE_EINVAL, "idxs[%d] is NULL", i);
    if (idxs[i]->dtype != idxs[0]->dtype || idxs[i]->d != idxs[0]->d ||
        idxs[i]->device != idxs[0]->device)
      return fail(SIEVE_EINVAL, "idxs[%d] differs from idxs[0] in dtype, d or device", i);
  }
  int st = check_common(idxs[0], queries, nq, k, tau, out_ids, out_scores, out_probes);
  if (st) return st;
  if (nprobe_max < 1) return fail(SIEVE_EINVAL, "nprobe_max = %d must be >= 1", nprobe_max);
  if (!(eps > 0.f && eps <= 1.f)) return fail(SIEVE_EINVAL, "eps = %g outside (0, 1]", (double)eps);
  if (W_fallback < 1) return fail(SIEVE_EINVAL, "W_fallback = %d must be >= 1", W_fallback);
  if (!out_W) return fail(SIEVE_EINVAL, "out_W is NULL");
  if (ns < 0 || ns > nq) return fail(SIEVE_EINVAL, "ns = %lld outside [0, nq]", (long long)ns);
  if (ns > kCalibMaxSample)
    return fail(SIEVE_EUNSUPPORTED, "ns = %lld exceeds %d", (long long)ns, kCalibMaxSample);
  if (ns > 0 && !sample) return fail(SIEVE_EINVAL, "sample is NULL with ns > 0");
  if (stats) memset(stats, 0, sizeof(*stats));
  if (nq == 0) {
    for (int32_t i = 0; i < nidx; ++i) out_W[i] = W_fallback;
    return SIEVE_OK;
  }
  hipStream_t s = (hipStream_t)stream;
  // per-index results, [nidx][nq][k], in the first index's workspace
  sieve_index* ws = const_cast<sieve_index*>(idxs[0]);
  const size_t rows = (size_t)nidx * (size_t)nq;
  if ((st = ensure(ws->mix_ids, rows * k * sizeof(int64_t))) ||
      (st = ensure(ws->mix_scores, rows * k * sizeof(float))) ||
      (st = ensure(ws->mix_probes, rows * sizeof(int32_t))))
    return st;
  int64_t* mids = (int64_t*)ws->mix_ids.p;
  float* msc = (float*)ws->mix_scores.p;
  int32_t* mpr = (int32_t*)ws->mix_probes.p;
  // each index calibrates its own window on the same sampled queries
  for (int32_t i = 0; i < nidx; ++i) {
    sieve_index* ix = const_cast<sieve_index*>(idxs[i]);
    const size_t r0 = (size_t)i * (size_t)nq;
    sieve_stats part;
    memset(&part, 0, sizeof(part));
    if ((st = calibrated_impl(ix, queries, nq, exclude_ids, k, tau, nprobe_max, sample, ns, eps,
                              W_fallback, mids + r0 * k, msc + r0 * k, mpr + r0, out_W + i,
                              stats ? &part : nullptr, s)))
      return st;
    if (stats) {
      add_stats(stats, part);
      stats->nprobe_eff = part.nprobe_eff;
    }
  }
  HIP_TRY(launch_merge_shards(nq, k, nidx, mids, msc, mpr, out_ids, out_scores, out_probes, s));
  HIP_TRY(hipStreamSynchronize(s));
  return SIEVE_OK;
}

}  // extern "C"
