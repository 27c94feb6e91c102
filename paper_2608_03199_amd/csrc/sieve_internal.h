// sieve_internal.h -- device data layout and kernel launchers of the gfx950
// threshold-aware IVF search.  Everything here is internal to libsieve.so.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/sieve.h"

namespace sieve {

// One ready item (q_i, j) of Sec. 4.2: query index and 0-based probe rank.
struct Item {
  int32_t q;
  int32_t rank;
};

// One unit of partition-scan work: up to kTileQ items of one list, scored
// against one chunk of that list's rows.
struct Tile {
  int64_t r0;         // first stored row of the tile's row chunk
  int32_t nrows;      // rows in the chunk (1..row_chunk)
  int32_t item_begin; // first item of the tile in the partition-major bucket
  int32_t nq;         // items in the tile (1..kTileQ)
  int32_t list;       // partition id
};

// A bucketed item carries its query's exclusion id, so that the scan reads
// everything about its next tile's items with one load per item.
struct BItem {
  int32_t q;
  int32_t rank;
  int64_t ex;  // exclude_ids[q], or INT64_MIN
};

// One qualifying candidate found by the scan (score >= tau, not excluded).
struct Hit {
  float score;
  int32_t q;
  int64_t id;
};

// Query-tile width of the scan, in blocks of 16 queries (MFMA M = 16): at
// most 8 for tiles whose query rows stay in LDS and for the dense-round tiles
// whose query fragments are held in registers (12-block register tiles read
// the lists less often but leave too few registers for the row ring).
constexpr int kQB = 8;
constexpr int kRegAQB = 8;
constexpr int kTileQ = 16 * (kQB > kRegAQB ? kQB : kRegAQB);
constexpr int kScanThreads = 256;  // 4 wave64
constexpr int kMaxRanks = 2048;    // largest n = min(nprobe_max, nlist)
constexpr int kMaxNlist = 16384;   // centroid scores of one query fit in LDS
constexpr int kMaxCand = 4096;     // rank-boundary candidates kept for the exact sort
constexpr int kMaxD = 4096;

// Per-round scheduling counters (device).
constexpr int kStatSlots = 32;

struct RoundCounters {
  int32_t ntiles;          // tiles built this round
  int32_t new_items;       // items emitted by the update for the next round
  int32_t queue[8];        // per-XCD tile cursors of the scan's work queue
  int32_t rank_error;      // set when a rank boundary has more than kMaxCand candidates
  int32_t n_ext;           // queries whose stop line passed their ranked prefix (this round)
  unsigned long long list_rows;   // sum over active lists of their length (this round)
  unsigned long long item_rows;   // sum over items of their list's length (this round)
  unsigned long long list_loads;  // active non-empty lists (this round)
  unsigned long long hits;        // candidate-pool entries written (whole search)
  unsigned long long cands;       // qualifying (query, row) pairs the scans found (whole search)
  int32_t heavy;                  // HeavyRec records claimed (whole search)
  int32_t sched_error;            // set when a round's tiles exceed the tile buffer
  // Sums of out_probes and of the qualifying candidates merged by the final
  // top-k, spread over kStatSlots counters (work-group b adds to slot
  // b % kStatSlots): thousands of adds to one address would serialise.
  unsigned long long probes[kStatSlots];
  unsigned long long candidates[kStatSlots];
};

// What the host needs after each round, written by a one-wave kernel after
// the update straight into coherent pinned host memory (no copy command).
struct RoundSummary {
  int32_t new_items;
  int32_t n_ext;
  int32_t rank_error;
  int32_t heavy;             // HeavyRec records claimed so far
  int32_t sched_error;       // a round's tiles exceeded the tile buffer
  int32_t pad_;
  unsigned long long hits;  // pool entries written so far
};

// Cumulative scan counters after one round (the per-round log of a timed
// search takes differences of consecutive snapshots).
constexpr int kMaxLogRounds = 256;
struct RoundSnap {
  unsigned long long list_rows, item_rows, list_loads, cands;
};

// The qualifying rows a tile finds go to a candidate arena: the work-group's
// LDS first, then a per-work-group extension in global memory.  At the end of
// the tile the arena is grouped by staged query (counting sort into the
// work-group's sorted area) and each query writes its candidates to the pool
// when it has at most k of them, else its exact top k (score descending, id
// ascending): a (query, tile) pair writes at most k pool entries, so the pool
// is bounded by (items x row chunks per list x k).  A tile whose arena
// overflows hands its queries with candidates to the exact top-k pass
// (scan_heavy) in HeavyRec records instead.
struct TileSpill {
  float score;
  uint32_t rowq;  // row offset inside the tile (low 24 bits) | staged query << 24
};
constexpr int kSpillRowBits = 24;
// TileCand: a candidate of the exact top-k pass's LDS buffers.
struct TileCand {
  float score;
  uint32_t row;  // row offset inside the tile
};

// Up to kHeavyQ overflowed queries of one tile, with the tile's rows (used
// when the work-group's spill area overflows).
constexpr int kHeavyQ = 16;
struct HeavyRec {
  int64_t r0;     // first stored row
  int64_t fd;     // its row in the fragment-order copy, less r0
  int32_t nrows;  // rows
  int32_t nq;     // queries in the record (1..kHeavyQ)
  int32_t q[kHeavyQ];
  int32_t rank[kHeavyQ];
  int64_t ex[kHeavyQ];
};

// LDS arena entries at most.  A work-group's global area holds the arena's
// extension (spill_cap entries) and the grouped copy of the pairs of the
// queries with more than k of them (at most kArenaLdsMax + spill_cap
// entries, each with its row id: two TileSpill units).  spill_cap is even, so
// the grouped copy is 16-byte aligned.
constexpr int kArenaLdsMax = 12288;
struct SrtEnt {
  float score;
  int32_t pad;
  int64_t id;
};
static_assert(sizeof(SrtEnt) == 2 * sizeof(TileSpill), "grouped entries take two arena units");
__host__ __device__ inline size_t arena_block_entries(int spill_cap) {
  return (size_t)spill_cap + 2 * ((size_t)spill_cap + kArenaLdsMax);
}

struct ScanArgs {
  const void* vectors;         // [n, d] partition-major
  const void* vfrag;           // its fragment-order copy (compile-time dimensions)
  const int64_t* frag_offsets; // [nlist + 1] first row of each partition in the copy
  const int64_t* list_offsets; // [nlist + 1]
  const int64_t* ids;          // [n]
  const void* queries;         // [nq, d]
  const int64_t* exclude;      // [nq] or null
  const BItem* bucket;         // partition-major items of this round
  const Tile* tiles;
  RoundCounters* rc;
  int32_t* lmax;               // [nq] max 1-based hit rank this round (0 = none)
  int32_t* hcount;             // [nq] pool entries per query
  Hit* pool;
  unsigned long long* pool_count;
  int64_t pool_cap;
  HeavyRec* heavy;             // overflowed (tile, query) groups for the exact top-k pass
  int32_t* heavy_count;
  int64_t heavy_cap;
  int32_t k;
  TileSpill* spill;            // [grid][arena_block_entries(spill_cap)]: per work-group
                               // arena extension, then the grouped arena
  int32_t spill_cap;           // arena entries in global memory per work-group (0: none)
  int32_t arena_on;            // 0: no arena (tiles of 2^24 rows or more); every tile with
                               // candidates takes the exact top-k pass
  int32_t d;
  int32_t row_chunk;
  int32_t tile_q;              // query rows per tile (multiple of 16, <= kTileQ)
  int32_t dynamic;             // 1: atomic work queue, 0: static strided schedule
  int32_t stage_u4;            // 16-byte slots per query staging buffer (set by the launcher)
  int32_t cand_u4;             // 16-byte offset of the LDS arena in dynamic LDS (launcher)
  int32_t arena_lds;           // LDS arena entries (launcher)
  int32_t wide;                // 1: wide configuration (one big work-group per CU)
  // calibration outputs (Algorithm 3), null / 0 otherwise: per query a bitmap
  // of the ranks whose probe had a candidate, and pool entries that carry
  // the rank they were found at (Hit.q = query | rank << kRankShift)
  uint32_t* hitbits = nullptr;
  int32_t hit_words = 0;       // 32-bit words per query in hitbits
  float tau;
};

// Query rows per tile for a dtype and dimension: as many 16-row blocks (<= 8)
// as fit an 80 KB LDS budget, so that two work-groups share a CU.
int tile_rows(int dtype, int d);
// Wide scan configuration: one work-group of kScanThreadsWide threads per CU
// with a tile of up to 150 KB of staged queries (large rows: fewer re-reads
// of each list by its query tiles).
constexpr int kScanThreadsWide = 512;
int tile_rows_wide(int dtype, int d);
bool scan_wide_supported(int dtype, int d);
// Whether the scan keeps the tile's query fragments in registers (short rows;
// one work-group per CU, whole lists per tile in dense rounds).
bool scan_uses_rega(int dtype, int d);
// Query rows per register-A tile: dense rounds (one work-group per CU) and
// sparse rounds (two per CU); the launch picks the kernel from tile_q.
int scan_rega_tile_q(bool dense);

// ---- launchers (each returns the hipError_t of its launch) ----
hipError_t launch_rank_scores(int dtype, const void* queries, int64_t q0, int32_t nqc,
                              const void* centroids, int32_t nlist, int32_t d, float* scores,
                              hipStream_t s);
size_t scan_lds_bytes(int dtype, int d, int rows);
// Fused screen + selection of the first R (<= kRankPrefixMax) ranks of
// queries [q0, q0 + nqc) into P (row stride ldp); cand holds
// nqc * rank_prefix_cap(R, nlist) keys and ccount nqc counts.
constexpr int kRankPrefixMax = 64;
int rank_prefix_cap(int32_t R, int32_t nlist);
// Centroids in MFMA fragment order, for the ranking kernels of compile-time
// dimensions: 16-row block b, 64-byte chunk c of a row and lane l hold the 16
// bytes at slot (b nch + c) 64 + l, taken from row 16 b + l % 16, segment
// 4 c + l / 16 (zeros past the last row), so that a wave's fragment load
// reads 1 KB of consecutive bytes (nch = 64-byte chunks per row; the layout
// FragStream reads).  centroid_frag_bytes is 0 where no kernel reads a copy.
size_t centroid_frag_bytes(int dtype, int d, int32_t nlist);
hipError_t launch_centroid_frag(int dtype, int d, const void* centroids, int32_t nlist, void* frag,
                                hipStream_t s);
// Fragment-order copy of the stored vectors, read by the scan kernels of
// compile-time dimensions: each partition padded to whole 16-row blocks
// (frag_offsets: its first copy row, a multiple of 16), and for each 16-row
// block and 64-byte chunk of a row the 64 16-byte segments one MFMA fragment
// load takes, in lane order (the layout is given with the reader,
// FragStream).  frag_rows = frag_offsets[nlist].  vector_frag_bytes is 0 for
// dimensions the scan handles at run time (no copy).
size_t vector_frag_bytes(int dtype, int d, int64_t frag_rows);
hipError_t launch_vector_frag(int dtype, int d, const void* vectors, const int64_t* offsets,
                              const int64_t* frag_offsets, int32_t nlist, int64_t frag_rows,
                              void* frag, hipStream_t s);
// cfrag: the index's fragment-order centroids (centroid_frag_bytes > 0), or
// null where it has none.
hipError_t launch_rank_prefix(int dtype, const void* queries, int64_t q0, int32_t nqc,
                              const void* centroids, const void* cfrag, int32_t nlist, int32_t d,
                              int32_t R, double cmax, unsigned long long* cand, int32_t* ccount,
                              int32_t* P, int64_t ldp, RoundCounters* rc, int32_t pass1_div,
                              hipStream_t s);
hipError_t launch_rank_select(int dtype, const void* queries, int64_t q0, int32_t nqc,
                              const void* centroids, int32_t nlist, int32_t d, const float* scores,
                              int32_t n, double cmax, int32_t* P, int64_t ldp, RoundCounters* rc,
                              bool wide, hipStream_t s);

hipError_t launch_emit_initial(const int32_t* P, int32_t n, int64_t nqc, int32_t q0, int32_t s0,
                               int32_t mode, Item* items, int64_t item_cap, int32_t* cnt,
                               int32_t nlist,
                               int32_t* state_a, int32_t* state_b, int32_t* lmax, hipStream_t s);
// tiles: non-null (at most kFuseTilesMaxLists lists) to write the round's
// tiles and clear the histogram in the same launch (no sched_tiles launch).
constexpr int kFuseTilesMaxLists = 1024;
hipError_t launch_sched_offsets(int32_t* cnt, const int64_t* list_offsets, int32_t nlist,
                                int32_t row_chunk, int32_t tile_q, int32_t* item_off,
                                int32_t* cursor, int32_t* tile_off, RoundCounters* rc,
                                Tile* tiles, int64_t tile_cap, hipStream_t s);
hipError_t launch_sched_scatter(const Item* items, int32_t n_items, const int32_t* P, int32_t n,
                                int32_t q0, const int64_t* exclude, int32_t* cursor,
                                BItem* bucket, hipStream_t s);
hipError_t launch_sched_tiles(int32_t* cnt, const int32_t* item_off, const int32_t* tile_off,
                              const int64_t* list_offsets, int32_t nlist, int32_t row_chunk,
                              int32_t tile_q, Tile* tiles, int64_t tile_cap, hipStream_t s);
hipError_t launch_scan(int dtype, const ScanArgs& a, int32_t grid, hipStream_t s);
// The updates emit ranks below have[q] (ranks already ordered in P) and
// list the queries that need more in ext[] (count in rc->n_ext).
// issued: null, or [nq] end of the issued ranks of each query (kept by every
// update once given).  Speculative issue (hitbits non-null, issued required):
// ranks past the stop line may already be scanned; hitbits ([nq][words], bit
// r = the probe at rank r had a candidate, set for every rank scanned in the
// round just finished) replays the stop rule over them.  A line that moved by
// at least spec_min ranks gets as many more issued past it, at most spec_max.
hipError_t launch_update_lookahead(int64_t nq, const int32_t* P, int32_t n, int32_t W,
                                   int32_t* stop, int32_t* lmax, const int32_t* have,
                                   int32_t* ext, Item* items, int64_t item_cap, int32_t* cnt,
                                   RoundCounters* rc, const uint32_t* hitbits, int32_t words,
                                   int32_t* issued,
                                   int32_t spec_max, int32_t spec_min, RoundSummary* out,
                                   hipStream_t s);
hipError_t launch_update_basic(int64_t nq, const int32_t* P, int32_t n, int32_t W, int32_t* next,
                               int32_t* stale, int32_t* lmax, const int32_t* have, int32_t* ext,
                               Item* items, int64_t item_cap, int32_t* cnt, RoundCounters* rc,
                               RoundSummary* out, hipStream_t s);
// Lazy ranking: copy the listed queries' rows together, copy their new rank
// rows into P, and emit the items the extension unblocked.
hipError_t launch_gather_rows(const int32_t* ext, int32_t n_ext, const void* src,
                              int64_t row_bytes, void* dst, hipStream_t s);
hipError_t launch_scatter_ranks(const int32_t* ext, int32_t n_ext, const int32_t* Pext,
                                int32_t n, int32_t* P, hipStream_t s);
hipError_t launch_emit_pending(const int32_t* ext, int32_t n_ext, int32_t mode, const int32_t* P,
                               int32_t n, const int32_t* state_a, int32_t* have,
                               int32_t new_have, Item* items, int64_t item_cap, int32_t* cnt,
                               RoundCounters* rc, int32_t* issued, hipStream_t s);

hipError_t launch_snapshot_round(const RoundCounters* rc, RoundSnap* log, int32_t slot,
                                 hipStream_t s);
hipError_t launch_fill_i32(int32_t* p, int64_t n, int32_t v, hipStream_t s);
// Several 32-bit fills in one launch (segments with n = 0 are skipped).
constexpr int kFillSegs = 6;
struct FillSeg {
  int32_t* p;
  int64_t n;  // 32-bit words
  int32_t v;
};
struct FillSegs {
  FillSeg seg[kFillSegs];
};
hipError_t launch_fill_multi(const FillSegs& f, hipStream_t s);
hipError_t launch_zero_bytes(void* p, int64_t bytes, hipStream_t s);
hipError_t launch_exclusive_scan(const int32_t* in, int64_t* out, int64_t* out_copy, int64_t n,
                                 int64_t* block_tmp, hipStream_t s);
size_t exclusive_scan_tmp_elems(int64_t n);
// Exact top-k pass over the overflowed (tile, query) groups: one wave per
// HeavyRec selects each query's top k (score desc, id asc) among the tile's
// qualifying rows and appends them to the pool.
struct HeavyArgs {
  const void* vectors;
  const void* vfrag;  // fragment-order copy of vectors (compile-time dimensions)
  const int64_t* ids;
  const void* queries;
  const HeavyRec* recs;
  int32_t nrec;
  int32_t d;
  int32_t k;
  int32_t pack_rank;  // pool entries carry their rank (q | rank << kRankShift)
  float tau;
  int32_t* hcount;
  Hit* pool;
  unsigned long long* pool_count;
  int64_t pool_cap;
};
hipError_t launch_scan_heavy(int dtype, const HeavyArgs& a, int32_t grid, hipStream_t s);
// Pool entries of a calibration search pack the rank into Hit.q.
constexpr int kRankShift = 20;  // queries < 2^20, ranks < 2^11 (kMaxRanks)
constexpr int32_t kQueryMask = (1 << kRankShift) - 1;
hipError_t launch_pool_scatter(const Hit* pool, int64_t n, int64_t* cursor, Hit* sorted,
                               bool packed, hipStream_t s);
// out_map: null, or [nq] output row of each query (results of query q go to
// row out_map[q] of out_ids / out_scores / out_probes).  out_rank: null, or
// [nq * k] int32 (indexed by q, not mapped) receiving the 0-based rank each
// returned candidate was found at (-1 for padding); needs packed pool entries.
// rank_limit: null, or [nq] -- pool entries (packed) found at a rank >= the
// query's limit are left out (speculatively scanned ranks past the stop line).
hipError_t launch_topk(int64_t nq, int32_t k, const Hit* sorted, const int64_t* hoff,
                       const int32_t* hcount, const int32_t* probes_src, int32_t probes_const,
                       const int32_t* out_map, int64_t* out_ids, float* out_scores,
                       int32_t* out_probes, int32_t* out_rank, const int32_t* rank_limit,
                       RoundCounters* rc, hipStream_t s);
// Best k of nshard per-index top-k lists per query ([nshard][nq][k], id -1
// padding) and the sum of the per-index probe counts ([nshard][nq]).
hipError_t launch_merge_shards(int64_t nq, int32_t k, int32_t nshard, const int64_t* sids,
                               const float* sscores, const int32_t* sprobes, int64_t* out_ids,
                               float* out_scores, int32_t* out_probes, hipStream_t s);
// ---- in-call window calibration (Algorithm 3) ----
hipError_t launch_gather_i64(const int32_t* idx, int64_t n, const int64_t* src, int64_t* dst,
                             hipStream_t s);
// Required-window histogram hist[0..n] (hist[W]: neighbours whose required
// window is W) and their total z, from ns sampled queries' rank bitmaps and
// found ranks; then the chosen window into *w_out (0 when z = 0).
hipError_t launch_calib_replay(int64_t ns, int32_t n, int32_t k, const uint32_t* hitbits,
                               int32_t words, const int32_t* frank, unsigned long long* hist,
                               unsigned long long* z, hipStream_t s);
constexpr int kCalibMaxSample = 1 << kRankShift;
hipError_t launch_calib_choose(int32_t n, float eps, const unsigned long long* hist,
                               const unsigned long long* z, int32_t* w_out, hipStream_t s);

}  // namespace sieve
