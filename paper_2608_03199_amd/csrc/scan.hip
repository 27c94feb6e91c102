// scan.hip -- partition scan (within-partition search, Sec. 2.3 and Sec. 5)
// fused with the tau test, the exact top-k pass for tiles whose candidates
// overflow, and the centroid-screen GEMM of the ranking step (Sec. 4.1).  All
// use the MFMA tile engine of mfma_tile.h.
//
// Partition scan: each tile holds up to 16*QB ready items (q_i, j) of one
// partition (Sec. 4.2's partition group) and a range of that partition's rows
// (the whole list in dense rounds).  The tile's query rows are staged in LDS;
// every wave streams 16 rows at a time from HBM into registers and scores
// them against all the tile's queries.  For short rows (at most 4 MFMA
// chunks, e.g. 128-dim fp16) each wave first copies its query fragments from
// LDS into registers and keeps them for the whole tile (the staging buffer is
// then refilled with the next tile's queries while this one streams); longer
// rows read the fragments from LDS per row block.  A score that reaches tau
// (inclusive, Sec. 2.2) for a row whose id is not the query's exclusion id
// makes the probe a hit (Sec. 4.1): the query's highest hit rank of the round
// is raised with an atomic max.  The hit test depends only on the pair's own
// score, never on other candidates, so it is the same whatever the dispatch
// order (the property the lookahead equivalence of Sec. 4.3 needs).
//
// Local results (Algorithm 1 keeps each partition's filtered top-k for the
// final MergeTopK): a qualifying pair goes to the work-group's candidate
// arena (LDS, then a global extension); at the end of the tile each query
// writes its candidates, or its exact top k when it has more, to the pool.
// A (query, tile) pair thus writes at most k pool entries.  A tile whose
// arena overflows records its queries, with the tile's rows, for the exact
// top-k pass instead.
//
// Work distribution: a persistent grid pulls tiles from a per-XCD work queue
// (see the kernel); every block exits after its claims run dry, at most
// tiles + 8 claims per block.
#include "mfma_tile.h"
#include "wave_sort.h"

namespace sieve {
namespace {

// Query staging: with kAsync the tile's query rows are copied global -> LDS
// by the DMA path of the load unit (no registers) into one of two buffers
// while the previous tile is still being multiplied; otherwise they are
// staged through registers at the start of their tile.
template <int DT, int D>
constexpr bool async_stage_ok() {
  if (D <= 0 || D % DTraits<DT>::kChunkDims != 0) return false;  // no partial chunk to zero
  // two full-size buffers must fit the two-work-groups-per-CU budget
  const int row = (4 * (D / DTraits<DT>::kChunkDims) + 1) * 16;
  return 2 * 16 * qb_cap<DT, D>() * row <= 76 * 1024;
}

// Copy the query rows of a tile into a staging buffer with LDS-DMA loads:
// 64 consecutive 16-byte slots of the buffer per wave instruction, slot
// (row, seg) <- segment seg of the row's query.  Padding rows (past nq) and
// the pad segment copy real data (a padding row repeats row 0): their scores
// are never tested, and each buffer is padded to whole 64-slot chunks.
template <int DT>
__device__ __forceinline__ void dma_stage(u32x4* buf, const RowGeom<DT>& g,
                                          const char* __restrict__ qbase, size_t row_bytes,
                                          const int32_t* sq, int nq) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nwaves = blockDim.x >> 6;
  const int total = ((nq + 15) >> 4) * 16 * g.segs;
  const int nchunk = (total + 63) >> 6;
  for (int c = wave; c < nchunk; c += nwaves) {
    const int sidx = c * 64 + lane;
    const int row = sidx / g.segs, seg = sidx - row * g.segs;
    const int qrow = sq[row < nq ? row : 0];
    const int segc = (seg < g.dsegs && sidx < total) ? seg : 0;
    const char* src = qbase + (size_t)qrow * row_bytes + (size_t)segc * 16;
    __builtin_amdgcn_global_load_lds((const void*)src,
                                     (__attribute__((address_space(3))) void*)(buf + c * 64), 16,
                                     0, 0);
  }
}

// f(std::integral_constant<int, QB>) for the tile's number of 16-query
// blocks qb_n (uniform per tile), QB = 1 .. kMax.
template <int QB, int kMax, typename F>
__device__ __forceinline__ void with_qb(int qb_n, F&& f) {
  if constexpr (QB >= kMax) {
    f(std::integral_constant<int, kMax>{});
  } else {
    if (qb_n <= QB)
      f(std::integral_constant<int, QB>{});
    else
      with_qb<QB + 1, kMax>(qb_n, f);
  }
}

// Register-A tiles come in two shapes.  Dense rounds (many items per list):
// tiles of up to 8 query blocks, whose fragments take 128 registers at
// 128-dim fp16, so the kernel runs one work-group per CU and takes the whole
// register file (512 per lane).  Sparse rounds: tiles of up to 4 query
// blocks at two work-groups per CU (256 registers each), twice the waves to
// keep row loads in flight.
template <int kOcc>
constexpr int rega_max_qb() {
  return kOcc == 1 ? kRegAQB : 4;
}

// Unsigned key whose order is the float order of finite and infinite scores
// (sign flipped for positive values, all bits flipped for negative ones; -0
// takes +0's key, as the two compare equal).
__device__ __forceinline__ uint32_t order_key(float x) {
  const uint32_t u = __float_as_uint(x == 0.0f ? 0.0f : x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Top-k selection at the end of a tile: score keys per lane held in
// registers, and the LDS arena entries (8 bytes) each wave borrows to compact
// 64 segment positions.
constexpr int kSelR = 8;
constexpr int kSelSlots = 64 * (int)sizeof(int32_t) / (int)sizeof(TileSpill);

// Largest of one query block's four accumulator elements (the same tree in
// the vote and in the candidate test, so the two share it).
__device__ __forceinline__ float block_max(const f32x4& v) {
  return fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3]));
}

// Element x = 4 qb + r of a row block's accumulators, x uniform: a chain of
// selects on a scalar condition (no indexed register access).
template <int QB>
__device__ __forceinline__ float pick_score(const f32x4 (&acc)[QB], int x) {
  float v = acc[0][0];
#pragma unroll
  for (int y = 1; y < 4 * QB; ++y) v = x == y ? acc[y >> 2][y & 3] : v;
  return v;
}

// Staging modes of the scan kernel.
constexpr int kStageSync = 0;   // staged through registers at the start of each tile
constexpr int kStageAsync = 1;  // LDS-DMA into the other of two buffers, one tile ahead
constexpr int kStageRegA = 2;   // LDS-DMA into one buffer; fragments kept in registers

// Largest tile (staged queries) of a scan kernel configuration: its
// per-query LDS arrays are sized for it.
template <int kMode, int kOcc>
constexpr int scan_tile_max() {
  return kMode == kStageRegA ? 16 * rega_max_qb<kOcc>() : 16 * kQB;
}

template <int DT, int D, int kMode, int kNT, int kOcc>
__global__ __launch_bounds__(kNT, kOcc) void scan_kernel(ScanArgs a) {
  constexpr int kTQ = scan_tile_max<kMode, kOcc>();  // staged queries, at most
  extern __shared__ u32x4 lds[];
  __shared__ int32_t s_q[2][kTQ];     // item sets: the running tile and the next
  __shared__ int32_t s_rank[2][kTQ];
  __shared__ int64_t s_ex[2][kTQ];
  __shared__ int32_t s_hits[kTQ];  // qualifying rows per staged query in this tile
  __shared__ int32_t s_over[kTQ];  // staged queries whose candidates overflowed
  __shared__ int32_t s_lost[kTQ];  // their qualifying rows the full arena did not take
  __shared__ int32_t s_sel[kTQ];   // staged queries selected from slots + spill
  __shared__ int32_t s_soff[kTQ];  // their segment in the sorted spill
  __shared__ int32_t s_scur[kTQ];
  __shared__ int32_t s_poff[kTQ];  // their first pool entry (after the tile's base)
  __shared__ int32_t s_pool_n, s_over_n, s_sel_n, s_rbase;
  __shared__ int32_t s_wcnt[kNT / 64];  // pairs each wave appended in this tile
  __shared__ unsigned long long s_pbase;
  // per work-group: the arena's global extension (spill_cap entries), then
  // the tile's whole arena grouped by query (LDS part and extension)
  TileSpill* const arena_g = a.spill + (size_t)blockIdx.x * arena_block_entries(a.spill_cap);
  SrtEnt* const arena_srt = (SrtEnt*)(arena_g + a.spill_cap);
  TileSpill* s_arena = (TileSpill*)(lds + a.cand_u4);  // [arena_lds]
  const int arena_lds = a.arena_lds;
  // Each wave appends to a private part of the arena (no atomics): wcap
  // entries in LDS, then gcap in the global extension.
  const int nwv = (int)(blockDim.x >> 6);
  const int wv = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int wcap = arena_lds / nwv, gcap = a.spill_cap / nwv;
  int wcnt = 0;  // this wave's pairs in the running tile (uniform)

  const int d = D > 0 ? D : a.d;
  const RowGeom<DT> g = RowGeom<DT>::make(d);
  const int lane = threadIdx.x & 63;
  const int h = lane >> 4;
  const size_t row_bytes = (size_t)d * DTraits<DT>::kElem;
  const int ntiles = a.rc->ntiles;
  const char* qbase = (const char*)a.queries;
  __shared__ int s_claim;
  __shared__ int s_next;  // one-ahead claims: the tile claimed at this tile's start
  constexpr bool kShallow = (kMode == kStageRegA && kOcc == 1) ||
                            (kMode == kStageSync && kNT == kScanThreadsWide);

  // Tile schedule: the round's tiles are split into 8 contiguous ranges, one
  // per XCD (block b runs on XCD b % 8, so tiles of one list share that XCD's
  // L2).  Static: the blocks of an XCD take its range's tiles in a fixed
  // stride (no atomics; best for small rounds).  Dynamic: thread 0 claims
  // tiles from its XCD's range with an atomic counter and moves on to the
  // other ranges once it is drained (balances large rounds).  While tile t
  // runs, the block holds tile t+1 (items in LDS, queries staging) and the
  // descriptor and items of tile t+2 (loads issued under t's MFMAs).
  const int home = blockIdx.x & 7;
  int xq = 0;    // thread 0, dynamic schedule: ranges already drained
  int kseq = 0;  // thread 0, static schedule: tiles taken so far
  auto claim = [&]() -> int {
    if (!a.dynamic) {
      // static: block (home, slot) takes every (grid/8)-th tile of its range
      const int b = (int)(((int64_t)ntiles * home) / 8);
      const int e = (int)(((int64_t)ntiles * (home + 1)) / 8);
      const int tt = b + (blockIdx.x >> 3) + kseq * (int)(gridDim.x >> 3);
      ++kseq;
      return tt < e ? tt : -1;
    }
    while (xq < 8) {
      const int x = (home + xq) & 7;
      const int b = (int)(((int64_t)ntiles * x) / 8), e = (int)(((int64_t)ntiles * (x + 1)) / 8);
      const int i = atomicAdd(&a.rc->queue[x], 1);
      if (b + i < e) return b + i;
      ++xq;
    }
    return -1;
  };

  // Tile records and items flow through registers one tile ahead of use:
  // each is loaded a whole tile before it is needed and never behind another
  // load of the same tile (no dependent loads on the tile path).
  auto load_rec = [&](int tt) -> Tile {
    Tile r = {0, 0, 0, 0, 0};
    tt = __builtin_amdgcn_readfirstlane(tt);  // uniform: scalar loads
    if (tt >= 0) r = a.tiles[tt];
    return r;
  };
  auto load_items = [&](const Tile& r) -> BItem {
    // always a valid address: item 0 of the round stands in for no tile
    const int64_t idx = r.nq > 0 ? r.item_begin + min((int)threadIdx.x, r.nq - 1) : 0;
    return a.bucket[idx];
  };
  auto put_items = [&](int set, const Tile& r, const BItem& it) {
    if ((int)threadIdx.x < r.nq) {
      s_q[set][threadIdx.x] = it.q;
      s_rank[set][threadIdx.x] = it.rank;
      s_ex[set][threadIdx.x] = it.ex;
    }
  };

  // four claims ahead: t (runs), tn (stages), ta (items load), tb (record
  // loads); thread 0 claims the next one under each tile's MFMAs.  The dense
  // register-query kernel and the wide 768-dimension kernel (kShallow) claim
  // one tile ahead instead: tile t+1 is claimed at the start of tile t, its
  // record and items load under t's row stream, and its queries are staged
  // under t's end (register-query kernel) or at its own start (wide kernel).
  // Their tiles are long, so the chain fits in one tile, and a list's query
  // tiles, claimed one after another, then start within about one tile
  // duration of each other instead of four: they read the list's rows closer
  // together, and more of those reads hit L2.
  __shared__ int s_first[4];
  if (threadIdx.x == 0) {
    s_first[0] = claim();
    s_first[1] = kShallow ? -1 : claim();
    s_first[2] = kShallow ? -1 : claim();
    s_first[3] = kShallow ? -1 : claim();
    s_pool_n = 0;
    s_over_n = 0;
    s_sel_n = 0;
  }
  if (threadIdx.x < kTQ) {
    s_hits[threadIdx.x] = 0;
    s_lost[threadIdx.x] = 0;
  }
  __syncthreads();
  int t = s_first[0], tn = s_first[1], ta = s_first[2], tb = s_first[3];
  Tile recT = load_rec(t), recN = load_rec(tn), recA = load_rec(ta);
  BItem itN = load_items(recN);
  put_items(0, recT, load_items(recT));
  int set = 0;
  __syncthreads();
  if constexpr (kMode != kStageSync) {
    if (t >= 0) dma_stage<DT>(lds, g, qbase, row_bytes, s_q[0], recT.nq);
    __builtin_amdgcn_s_waitcnt(0);
  }
  __syncthreads();

  for (; t >= 0;) {
    const int nset = set ^ 1;
    const int32_t* sq = s_q[set];
    const int32_t* srank = s_rank[set];
    const int64_t* sex = s_ex[set];
    const int nq = recT.nq;
    const int qb_n = (nq + 15) >> 4;
    const int64_t r0 = recT.r0, r1 = recT.r0 + recT.nrows;
    // copy row minus store row of the tile's partition (fragment-order copy)
    const int64_t fd =
        D > 0 ? a.frag_offsets[recT.list] - a.list_offsets[recT.list] : (int64_t)0;
    // the next tile's items go to the other set
    if constexpr (!kShallow) put_items(nset, recN, itN);
    BItem itA;
    Tile recB;
    int t_claim = -1;

    // Only the tile's last 16-query block can hold padding rows (qb_n =
    // ceil(nq / 16)); its four rows of this lane get threshold +inf when they
    // are padding, so the test below needs no per-row index compares.
    const float tau = a.tau;
    float thr_last[4];
#pragma unroll
    for (int r = 0; r < 4; ++r)
      thr_last[r] = ((qb_n - 1) * 16 + 4 * h + r) < nq ? tau : INFINITY;
    // tau test of a row block, true (wave-uniform) when some lane's row
    // scores at least tau against some staged query: full query blocks
    // through a max tree, the last one (which may hold padding queries, with
    // threshold +inf) element by element.  Rows past r1 get threshold +inf.
    auto vote = [&](const auto& acc, int64_t row) -> bool {
      constexpr int QB = sizeof(acc) / sizeof(acc[0]);
      const float tr = row < r1 ? tau : INFINITY;
      float mx = -INFINITY;
#pragma unroll
      for (int qb = 0; qb + 1 < QB; ++qb) mx = fmaxf(mx, block_max(acc[qb]));
      bool any = mx >= tr;
#pragma unroll
      for (int r = 0; r < 4; ++r) any |= acc[QB - 1][r] >= fmaxf(tr, thr_last[r]);
      return __ballot(any) != 0ull;
    };
    // Qualifying pairs of the row block go to the wave's part of the arena as
    // (score, row offset, staged query), in (query block, element, lane)
    // order.  A query block whose maximum misses tau is skipped with one
    // compare; otherwise each of its elements is one vector compare into a
    // lane mask, a scalar branch skips it when no lane qualifies, else the
    // lanes of the mask take consecutive slots (LDS stores only).  The cost
    // follows the qualifying (block, element) pairs, not the lanes.  When the run could
    // reach past the LDS part, a slower path also covers the global part and,
    // past that, counts per query the pairs the arena cannot take (own row
    // excluded) for the heavy pass; its global accesses complete before it
    // returns (a store left pending would make the compiler wait for every
    // load of the row stream, not just the oldest).  The self-exclusion is
    // otherwise left to the end of the tile.
    auto candidates = [&](const auto& acc, int64_t row) {
      constexpr int QB = sizeof(acc) / sizeof(acc[0]);
      const float tr = row < r1 ? tau : INFINITY;
      const uint32_t roff = (uint32_t)(row - r0);
      auto thr = [&](int qb, int r) { return qb + 1 < QB ? tr : fmaxf(tr, thr_last[r]); };
      if (wcnt + 64 * 4 * QB <= wcap) {
        TileSpill* const dst = s_arena + wv * wcap;
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
          // most query blocks of a passing row block hold no qualifying pair:
          // one compare of the block's maximum skips them
          bool okq = false;
          if (qb + 1 < QB) {
            okq = block_max(acc[qb]) >= tr;
          } else {
#pragma unroll
            for (int r = 0; r < 4; ++r) okq |= acc[qb][r] >= thr(qb, r);
          }
          if (__ballot(okq) == 0ull) continue;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const bool ok = acc[qb][r] >= thr(qb, r);
            const unsigned long long m = __ballot(ok);
            if (m == 0ull) continue;
            if (ok) {
              const int pos = wcnt + (int)__builtin_amdgcn_mbcnt_hi(
                                         (uint32_t)(m >> 32),
                                         __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
              dst[pos] = TileSpill{acc[qb][r],
                                   roff | ((uint32_t)(qb * 16 + 4 * h + r) << kSpillRowBits)};
            }
            wcnt += __popcll(m);
          }
        }
        return;
      }
      uint32_t lm = 0;
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
#pragma unroll
        for (int r = 0; r < 4; ++r) lm |= (acc[qb][r] >= thr(qb, r) ? 1u : 0u) << (qb * 4 + r);
      }
      int cnt = __popc(lm), pre = 0, tot = 0;  // cnt <= 32: six bit planes
#pragma unroll
      for (int b = 0; b < 6; ++b) {
        const unsigned long long m = __ballot((cnt >> b) & 1);
        pre += (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                              __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u)) << b;
        tot += __popcll(m) << b;
      }
      int pos = wcnt + pre;
      while (lm) {
        const int x = __builtin_ctz(lm);
        lm &= lm - 1;
        const int i = (x >> 2) * 16 + 4 * h + (x & 3);
        const TileSpill ent{pick_score(acc, x), roff | ((uint32_t)i << kSpillRowBits)};
        if (pos < wcap)
          s_arena[wv * wcap + pos] = ent;
        else if (pos - wcap < gcap)
          arena_g[wv * gcap + pos - wcap] = ent;
        else if (a.ids[row] != sex[i])
          atomicAdd(&s_lost[i], 1);
        ++pos;
      }
      __builtin_amdgcn_s_waitcnt(0);
      wcnt += tot;
    };
    // epilogue of the LDS-staged streams
    auto epi = [&](const auto& acc, int64_t row) {
      if (vote(acc, row)) candidates(acc, row);
    };

    if constexpr (kMode == kStageRegA) {
      with_qb<1, rega_max_qb<kOcc>()>(qb_n, [&](auto qbc) {
        constexpr int QB = decltype(qbc)::value;
        constexpr int kNC = D / DTraits<DT>::kChunkDims;
        u32x4 qf[kNC][QB];
        int nxt = -1;
        if constexpr (kShallow) {
          if (threadIdx.x == 0) nxt = claim();
        }
        load_afrags<DT, D, QB>(lds, g.segs, qf);
        __builtin_amdgcn_s_waitcnt(0);  // fragments in registers
        if constexpr (kShallow) {
          if (threadIdx.x == 0) s_next = nxt;
        }
        __syncthreads();  // every wave has its fragments: the staging buffer is free
        if constexpr (kShallow) {
          tn = s_next;
          recN = load_rec(tn);
          itN = load_items(recN);
        } else {
          if (threadIdx.x == 0) t_claim = claim();  // published at the end of this tile
          // pipeline loads, used one tile from now
          itA = load_items(recA);
          recB = load_rec(tb);
        }
        stream_rows_rega<DT, D, QB, kOcc == 1 ? 512 : 256, true>(qf, (const char*)a.vfrag,
                                                                  row_bytes, r0, r1, vote,
                                                                  candidates, fd);
        // The next tile's queries are staged after the stream, under the end
        // of this tile: an LDS-DMA load in flight during the stream makes the
        // compiler wait for every load there, not just the oldest ones.
        if constexpr (kShallow) {
          put_items(nset, recN, itN);  // staged after the barrier below
        } else {
          if (tn >= 0) dma_stage<DT>(lds, g, qbase, row_bytes, s_q[nset], recN.nq);
        }
      });
    } else {
      if constexpr (kShallow) {
        if (threadIdx.x == 0) s_next = claim();
      }
      __syncthreads();
      if constexpr (kShallow) {
        tn = s_next;
        recN = load_rec(tn);
        itN = load_items(recN);
      } else {
        if (threadIdx.x == 0) t_claim = claim();  // published at the end of this tile
      }
      u32x4* buf = lds;
      if constexpr (kMode == kStageAsync) {
        buf = lds + set * a.stage_u4;
        if (tn >= 0)
          dma_stage<DT>(lds + nset * a.stage_u4, g, qbase, row_bytes, s_q[nset], recN.nq);
      } else {
        stage_queries<DT>(lds, g, qb_n * 16, [&](int i) -> const u32x4* {
          return i < nq ? (const u32x4*)(qbase + (size_t)sq[i] * row_bytes) : nullptr;
        });
        __syncthreads();
      }
      if constexpr (!kShallow) {
        itA = load_items(recA);
        recB = load_rec(tb);
      }
      stream_rows<DT, D, 8, kNT == kScanThreads ? 80 : 150, (D > 0)>(
          buf, g, (const char*)(D > 0 ? a.vfrag : a.vectors), row_bytes, r0, r1, qb_n, epi, fd);
      if constexpr (kShallow) put_items(nset, recN, itN);  // staged at the next tile's start
    }
    if (lane == 0) s_wcnt[wv] = wcnt;
    wcnt = 0;
    // this wave's staging copies and arena stores are complete (in L2)
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();  // every wave is done with this tile's queries, items and candidates
    if constexpr (kShallow && kMode == kStageRegA) {
      if (tn >= 0) dma_stage<DT>(lds, g, qbase, row_bytes, s_q[nset], recN.nq);
    }
    // the arena's parts: pairs held per wave, their prefix; any global part?
    int wn[kNT / 64], wpre[kNT / 64 + 1];
    bool ext = false;
    wpre[0] = 0;
#pragma unroll
    for (int w = 0; w < kNT / 64; ++w) {
      const int cw = w < nwv ? s_wcnt[w] : 0;
      wn[w] = min(cw, wcap + gcap);
      ext |= cw > wcap;
      wpre[w + 1] = wpre[w] + wn[w];
    }
    // Candidates in the arena's global extension were stored by other waves of
    // the work-group: an acquire at agent scope invalidates the CU's vector L1,
    // whose lines of that area may be stale (read in an earlier tile).
    if (ext) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");

    // End of the tile.  The arena's pairs are counted per staged query, each
    // query's own row excluded (a pair whose row id is the query's excluded
    // id); four pairs per thread are in flight at once.
    const int na = wpre[kNT / 64];  // pairs the arena holds
    auto arena_at = [&](int e) -> TileSpill {
      int w = 0;
#pragma unroll
      for (int u = 1; u < kNT / 64; ++u) w += e >= wpre[u] ? 1 : 0;
      const int ew = e - wpre[w];
      return ew < wcap ? s_arena[w * wcap + ew] : arena_g[w * gcap + ew - wcap];
    };
    auto excluded = [&](const TileSpill& ts, int64_t id) {
      return id == sex[ts.rowq >> kSpillRowBits];
    };
    auto row_id = [&](const TileSpill& ts) -> int64_t {
      return a.ids[r0 + (ts.rowq & ((1u << kSpillRowBits) - 1u))];
    };
    for (int e0 = threadIdx.x; e0 < na; e0 += 4 * (int)blockDim.x) {
      TileSpill ts[4];
      int64_t id[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int e = e0 + u * (int)blockDim.x;
        ts[u] = arena_at(e < na ? e : e0);
        id[u] = row_id(ts[u]);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (e0 + u * (int)blockDim.x < na && !excluded(ts[u], id[u]))
          atomicAdd(&s_hits[ts[u].rowq >> kSpillRowBits], 1);
    }
    __syncthreads();

    // Per staged query: the hit flag; then its candidates to the pool (all of
    // them, or its exact top k when it has more), or, when the arena could not
    // take all of them, a heavy record for the exact top-k pass.
    int c = 0, keep = 0;
    if ((int)threadIdx.x < nq) {
      const int lost = s_lost[threadIdx.x];
      c = s_hits[threadIdx.x];
      if (c + lost > 0) {
        const int q = sq[threadIdx.x];
        const int rk = srank[threadIdx.x];
        atomicMax(&a.lmax[q], rk + 1);
        if (a.hitbits)
          atomicOr(&a.hitbits[(int64_t)q * a.hit_words + (rk >> 5)], 1u << (rk & 31));
        if (lost == 0) {
          keep = min(c, a.k);
          s_poff[threadIdx.x] = atomicAdd(&s_pool_n, keep);
          atomicAdd(&a.hcount[q], keep);
          if (c > a.k) s_sel[atomicAdd(&s_sel_n, 1)] = threadIdx.x;
        } else {
          s_over[atomicAdd(&s_over_n, 1)] = threadIdx.x;
        }
      }
      c += lost;
    }
    {
      // qualifying pairs of the tile, for the statistics: one add per wave
      unsigned long long cs = (unsigned long long)c;
      for (int o = 32; o > 0; o >>= 1) cs += __shfl_xor(cs, o);
      if (lane == 0 && cs) atomicAdd(&a.rc->cands, cs);
    }
    __syncthreads();
    const int pool_n = s_pool_n, over_n = s_over_n, sel_n = s_sel_n;  // block-uniform
    if (pool_n + over_n > 0) {
      if (threadIdx.x == 0) {
        s_pbase = pool_n ? atomicAdd(a.pool_count, (unsigned long long)pool_n) : 0ull;
        s_rbase = over_n ? atomicAdd(&a.rc->heavy, (over_n + kHeavyQ - 1) / kHeavyQ) : 0;
      }
      if ((int)threadIdx.x < nq) s_scur[threadIdx.x] = 0;
      // segments of the sorted area, for the queries with more than k pairs
      // only (wave 0: an exclusive prefix over s_sel, kPer consecutive
      // entries per lane)
      if (sel_n > 0 && threadIdx.x < 64) {
        constexpr int kPer = (kTQ + 63) / 64;
        int v[kPer];
        int tot = 0;
#pragma unroll
        for (int u = 0; u < kPer; ++u) {
          const int j = kPer * lane + u;
          v[u] = j < sel_n ? s_hits[s_sel[j]] : 0;
          tot += v[u];
        }
        int inc = tot;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const int t = __shfl_up(inc, o);
          if (lane >= o) inc += t;
        }
        int ex = inc - tot;
#pragma unroll
        for (int u = 0; u < kPer; ++u) {
          const int j = kPer * lane + u;
          if (j < sel_n) s_soff[s_sel[j]] = ex;
          ex += v[u];
        }
      }
      __syncthreads();
      if ((int)threadIdx.x < over_n) {
        const int gi = threadIdx.x / kHeavyQ, m = threadIdx.x % kHeavyQ;
        const int64_t rec = (int64_t)s_rbase + gi;
        if (rec < a.heavy_cap) {
          HeavyRec* hr = a.heavy + rec;
          const int i = s_over[threadIdx.x];
          hr->q[m] = sq[i];
          hr->rank[m] = srank[i];
          hr->ex[m] = sex[i];
          if (m == 0) {
            hr->r0 = r0;
            hr->fd = fd;
            hr->nrows = (int32_t)(r1 - r0);
            hr->nq = min(kHeavyQ, over_n - gi * kHeavyQ);
          }
        }
      }
      if (pool_n > 0) {
        // The arena's pairs, own rows and heavy queries left out: a query
        // with at most k of them writes them to its pool segment directly;
        // one with more groups them in the sorted area (counting sort) for
        // the exact top-k merge below.  Four pairs per thread in flight.
        const int k = a.k;
        for (int e0 = threadIdx.x; e0 < na; e0 += 4 * (int)blockDim.x) {
          TileSpill ts[4];
          int64_t id[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int e = e0 + u * (int)blockDim.x;
            ts[u] = arena_at(e < na ? e : e0);
            id[u] = row_id(ts[u]);
          }
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int qs = (int)(ts[u].rowq >> kSpillRowBits);
            if (e0 + u * (int)blockDim.x >= na || id[u] == sex[qs] || s_lost[qs] > 0) continue;
            const int ci = s_hits[qs];
            const int slot = atomicAdd(&s_scur[qs], 1);
            if (ci <= k) {
              const unsigned long long pi = s_pbase + (unsigned long long)(s_poff[qs] + slot);
              if ((int64_t)pi < a.pool_cap) {
                Hit hv;
                hv.score = ts[u].score;
                hv.q = a.hitbits ? (sq[qs] | (srank[qs] << kRankShift)) : sq[qs];
                hv.id = id[u];
                a.pool[pi] = hv;
              }
            } else {
              arena_srt[s_soff[qs] + slot] = SrtEnt{ts[u].score, 0, id[u]};
            }
          }
        }
        if (sel_n > 0) {
          // the grouped area is read by other waves: stores complete,
          // barrier, L1 invalidated (as above)
          __builtin_amdgcn_s_waitcnt(0);
          __syncthreads();
          __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
          // queries with more than k: one wave selects the query's top k from
          // its segment.  Up to kSelR * 64 pairs: their score keys sit in
          // registers, kSelR per lane; the k-th largest of the 64 lane maxima (a radix
          // select over order-preserving score keys, ballots only) is a lower
          // bound L on the k-th score, since k lanes hold a pair >= L.  When at
          // most 64 pairs reach L, their positions are compacted through the
          // wave's slice of the (now idle) LDS arena, and the pairs are loaded
          // and sorted once: every pair of the top k is among them, ties at L
          // included.  Otherwise (and for longer
          // segments) the segment is merged 64 pairs at a time: the next batch
          // loads under this one's sort, and a batch none of whose pairs
          // reaches the k-th score kept so far is not sorted.
          const Cand none = {-INFINITY, 0x7fffffffffffffffll, -1};
          const bool slots_ok = arena_lds >= nwv * kSelSlots;  // uniform
          int32_t* const wslot = (int32_t*)(s_arena + wv * kSelSlots);
          for (int j = threadIdx.x >> 6; j < sel_n; j += blockDim.x >> 6) {
            const int i = s_sel[j];
            const int ci = s_hits[i];
            const SrtEnt* seg = arena_srt + s_soff[i];
            auto fetch = [&](int b0) -> Cand {
              if (b0 + lane >= ci) return none;
              const SrtEnt se = seg[b0 + lane];
              return Cand{se.score, (long long)se.id, 0};
            };
            Cand top = none;
            bool picked = false;
            if (slots_ok && ci > 64 && ci <= kSelR * 64) {
              uint32_t key[kSelR];
              uint32_t kmax = 0;
#pragma unroll
              for (int r = 0; r < kSelR; ++r) {
                const int e = r * 64 + lane;
                key[r] = e < ci ? order_key(seg[e].score) : 0u;
                kmax = max(kmax, key[r]);
              }
              // k-th largest lane maximum (every lane holds a pair: ci > 64)
              uint32_t pre = 0, msk = 0;
              int need = k;
              for (int b = 31; b >= 0; --b) {
                const uint32_t bit = 1u << b;
                const int nhi = __popcll(__ballot((kmax & msk) == pre && (kmax & bit) != 0u));
                if (nhi >= need)
                  pre |= bit;
                else
                  need -= nhi;
                msk |= bit;
              }
              int cnt = 0;
#pragma unroll
              for (int r = 0; r < kSelR; ++r) cnt += __popcll(__ballot(key[r] >= pre));
              if (cnt <= 64) {
                // segment positions of the pairs that reach L, then one load each
                int pos = 0;
#pragma unroll
                for (int r = 0; r < kSelR; ++r) {
                  const bool take = key[r] >= pre;
                  const unsigned long long m = __ballot(take);
                  if (take)
                    wslot[pos + (int)__builtin_amdgcn_mbcnt_hi(
                                    (uint32_t)(m >> 32),
                                    __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u))] = r * 64 + lane;
                  pos += __popcll(m);
                }
                __builtin_amdgcn_wave_barrier();
                Cand c = none;
                if (lane < cnt) {
                  const SrtEnt se = seg[wslot[lane]];
                  c = Cand{se.score, (long long)se.id, 0};
                }
                __builtin_amdgcn_wave_barrier();  // slots read before the next query's
                top = wave_sort_desc<false>(c, lane);
                picked = true;
              }
            }
            if (!picked) {
              top = wave_sort_desc<false>(fetch(0), lane);
              Cand nxt = fetch(64);
              for (int b0 = 64; b0 < ci; b0 += 64) {
                Cand cnd = nxt;
                nxt = fetch(b0 + 64);
                const Cand kth = shfl_cand<false>(top, k - 1);
                if (__ballot(!better(kth, cnd)) == 0ull) continue;
                cnd = wave_sort_desc<false>(cnd, lane);
                const Cand rv = shfl_cand<false>(cnd, 63 - lane);  // top ++ reverse(cnd): bitonic
                top = better(top, rv) ? top : rv;
                top = wave_merge_desc<false>(top, lane);
              }
            }
            const int kk = min(ci, k);
            const unsigned long long base = s_pbase + (unsigned long long)s_poff[i];
            if (lane < kk && (int64_t)(base + lane) < a.pool_cap) {
              Hit hv;
              hv.score = top.s;
              hv.q = a.hitbits ? (sq[i] | (srank[i] << kRankShift)) : sq[i];
              hv.id = top.id;
              a.pool[base + lane] = hv;
            }
          }
        }
      }
    }
    __syncthreads();  // the counts and the spill are read; reset them for the next tile
    if ((int)threadIdx.x < nq) {
      s_hits[threadIdx.x] = 0;
      s_lost[threadIdx.x] = 0;
    }
    if (threadIdx.x == 0) {
      s_claim = t_claim;
      s_pool_n = 0;
      s_over_n = 0;
      s_sel_n = 0;
    }
    if constexpr (kShallow) __builtin_amdgcn_s_waitcnt(0);  // the next tile's staging
    __syncthreads();
    if constexpr (kShallow) {
      t = tn;
      recT = recN;
      set = nset;
      continue;
    }
    t = tn;
    tn = ta;
    ta = tb;
    tb = s_claim;
    recT = recN;
    recN = recA;
    recA = recB;
    itN = itA;
    set = nset;
  }
}

// Exact top-k of overflowed (tile, query) groups: one wave per HeavyRec
// scores its queries (a 16-query block, staged in LDS) against the tile's
// rows with the scan's MFMA sequence (the same bits) and keeps, per query, the
// qualifying rows in an LDS buffer.  Rows below the query's running k-th
// score are not kept; whenever a buffer fills up, the wave sorts it (score
// descending, id ascending) and keeps its first k, whose k-th score becomes
// the new admission threshold (the final k-th can only be higher).  At the
// end each query's first k go to the pool.
constexpr int kHeavyCap = 128;  // buffered candidates per query (two per lane when sorting)

template <int DT, int D>
__global__ __launch_bounds__(64) void scan_heavy_kernel(HeavyArgs a) {
  extern __shared__ u32x4 lds[];
  __shared__ TileCand s_buf[kHeavyQ][kHeavyCap];
  __shared__ int32_t s_cnt[kHeavyQ];
  __shared__ int32_t s_qv[kHeavyQ];  // pool entry query field (rank packed when asked)
  __shared__ int32_t s_qi[kHeavyQ];  // query index
  __shared__ int64_t s_ex[kHeavyQ];
  const int d = D > 0 ? D : a.d;
  const RowGeom<DT> g = RowGeom<DT>::make(d);
  const int lane = threadIdx.x & 63;
  const int h = lane >> 4, r16 = lane & 15;
  const size_t row_bytes = (size_t)d * DTraits<DT>::kElem;
  const char* qbase = (const char*)a.queries;
  const int k = a.k;
  const Cand none = {-INFINITY, 0x7fffffffffffffffll, -1};

  for (int rec = blockIdx.x; rec < a.nrec; rec += gridDim.x) {
    const HeavyRec* hr = a.recs + rec;
    const int nq = __builtin_amdgcn_readfirstlane(hr->nq);
    const int64_t r0 = hr->r0;
    const int64_t r1 = r0 + hr->nrows;
    if (lane < kHeavyQ) {
      const int i = lane < nq ? lane : 0;
      s_qv[lane] = a.pack_rank ? (hr->q[i] | (hr->rank[i] << kRankShift)) : hr->q[i];
      s_qi[lane] = hr->q[i];
      s_ex[lane] = hr->ex[i];
      s_cnt[lane] = 0;
    }
    // (nq >= 1: row 0 is always a real query, as stage_queries needs)
    stage_queries<DT>(lds, g, kHeavyQ, [&](int i) -> const u32x4* {
      return i < nq ? (const u32x4*)(qbase + (size_t)hr->q[i] * row_bytes) : nullptr;
    });
    __syncthreads();
    // admission threshold of this lane's four queries (4h + r)
    float thr[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) thr[r] = (4 * h + r) < nq ? a.tau : INFINITY;

    // keep the first k of query j's buffer (sorted), raise its threshold
    auto compact = [&](int j, bool final_pass, unsigned long long pbase) {
      const int n = s_cnt[j];
      Cand x = none, y = none;
      if (lane < n) {
        const TileCand tc = s_buf[j][lane];
        x = Cand{tc.score, (long long)a.ids[r0 + tc.row], (int)tc.row};
      }
      if (lane + 64 < n) {
        const TileCand tc = s_buf[j][lane + 64];
        y = Cand{tc.score, (long long)a.ids[r0 + tc.row], (int)tc.row};
      }
      x = wave_sort_desc<true>(x, lane);
      Cand top = x;
      if (n > 64) {
        y = wave_sort_desc<true>(y, lane);
        const Cand ry = shfl_cand<true>(y, 63 - lane);  // x ++ reverse(y) is bitonic
        top = better(x, ry) ? x : ry;
        top = wave_merge_desc<true>(top, lane);
      }
      const int kk = n < k ? n : k;
      if (final_pass) {
        if (lane < kk) {
          Hit hv;
          hv.score = top.s;
          hv.q = s_qv[j];
          hv.id = top.id;
          if ((int64_t)(pbase + lane) < a.pool_cap) a.pool[pbase + lane] = hv;
        }
        return;
      }
      __builtin_amdgcn_wave_barrier();
      if (lane < kk) s_buf[j][lane] = TileCand{top.s, (uint32_t)top.rank};
      if (lane == 0) s_cnt[j] = kk;
      if (kk == k) {
        const float tk = __shfl(top.s, k - 1);
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (h == (j >> 2) && r == (j & 3)) thr[r] = fmaxf(thr[r], tk);
      }
      __builtin_amdgcn_wave_barrier();
    };

    auto epi = [&](const auto& acc, int64_t row) {
      bool pass[4];
      bool any = false;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        pass[r] = row < r1 && acc[0][r] >= thr[r];
        any |= pass[r];
      }
      if (__ballot(any) == 0) return;
      const int64_t rid = a.ids[row < r1 ? row : r1 - 1];
      const uint32_t roff = (uint32_t)(row - r0);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int j = 4 * h + r;  // this lane group's query for element r
        const bool ok = pass[r] && rid != s_ex[j];
        const unsigned long long mask = __ballot(ok);
        if (mask == 0) continue;
        const uint32_t gm = (uint32_t)(mask >> (16 * h)) & 0xffffu;
        const int base = s_cnt[j];
        __builtin_amdgcn_wave_barrier();
        if (ok) s_buf[j][base + __popc(gm & ((1u << r16) - 1u))] = TileCand{acc[0][r], roff};
        if (r16 == 0 && gm) s_cnt[j] = base + __popc(gm);
        __builtin_amdgcn_wave_barrier();
      }
      // a buffer that could not take another full row block is compacted
      for (int j = 0; j < nq; ++j)
        if (s_cnt[j] > kHeavyCap - 16) compact(j, false, 0);
    };
    stream_rows_qb<DT, D, 1, decltype(epi), 0, (D > 0)>(
        lds, g, (const char*)(D > 0 ? a.vfrag : a.vectors), row_bytes, r0, r1, epi, hr->fd);

    // each query's first k to the pool: one claim for the record
    int tot = 0;
    for (int j = 0; j < nq; ++j) tot += min(s_cnt[j], k);
    unsigned long long pbase = 0;
    if (lane == 0 && tot) pbase = atomicAdd(a.pool_count, (unsigned long long)tot);
    pbase = ((unsigned long long)(uint32_t)__shfl((int)(pbase >> 32), 0) << 32) |
            (uint32_t)__shfl((int)(uint32_t)pbase, 0);
    for (int j = 0; j < nq; ++j) {
      const int kk = min(s_cnt[j], k);
      if (kk == 0) continue;
      compact(j, true, pbase);
      if (lane == 0) atomicAdd(&a.hcount[s_qi[j]], kk);
      pbase += kk;
    }
    __syncthreads();  // the staging buffer and the candidate buffers are reused
  }
}

// Centroid screen: scores[qi - q0][c] = fp32 <query qi, centroid c> for a
// chunk of queries.  Grid: (ceil(nqc / rows), ceil(nlist / kScreenCents)),
// rows <= 16 * kScreenQB queries per work-group.
constexpr int kScreenCents = 256;
constexpr int kScreenQB = 4;

template <int DT, int D>
__global__ __launch_bounds__(kScanThreads, 2) void rank_scores_kernel(
    const void* queries, int64_t q0, int32_t nqc, const void* centroids, int32_t nlist,
    int32_t dd, int32_t rows, float* scores) {
  extern __shared__ u32x4 lds[];
  const int d = D > 0 ? D : dd;
  const RowGeom<DT> g = RowGeom<DT>::make(d);
  const int lane = threadIdx.x & 63;
  const int h = lane >> 4;
  const size_t row_bytes = (size_t)d * DTraits<DT>::kElem;
  const int qt0 = blockIdx.x * rows;
  const int nq = min(rows, nqc - qt0);
  const int qb_n = (nq + 15) >> 4;
  const char* qbase = (const char*)queries + (size_t)(q0 + qt0) * row_bytes;
  stage_queries<DT>(lds, g, qb_n * 16, [&](int i) -> const u32x4* {
    return i < nq ? (const u32x4*)(qbase + (size_t)i * row_bytes) : nullptr;
  });
  __syncthreads();
  const int64_t c0 = (int64_t)blockIdx.y * kScreenCents;
  const int64_t c1 = min<int64_t>(nlist, c0 + kScreenCents);
  stream_rows<DT, D, kScreenQB>(lds, g, (const char*)centroids, row_bytes, c0, c1, qb_n,
                     [&](const auto& acc, int64_t c) {
                       constexpr int QB = sizeof(acc) / sizeof(acc[0]);
                       if (c >= c1) return;
#pragma unroll
                       for (int qb = 0; qb < QB; ++qb) {
#pragma unroll
                         for (int r = 0; r < 4; ++r) {
                           const int i = qb * 16 + 4 * h + r;
                           if (i < nq) scores[(size_t)(qt0 + i) * nlist + c] = acc[qb][r];
                         }
                       }
                     });
}

// Dynamic LDS above 64 KB must be opted into once per kernel.
constexpr int kMaxDynLds = 150 * 1024;

// LDS per staging buffer (whole 64-slot chunks) and whether two of them fit
// the budget that keeps two work-groups per CU.
template <int DT, int D>
size_t stage_bytes(int d, int tile_q) {
  const size_t b = (size_t)tile_q * lds_row_bytes<DT>(D > 0 ? D : d);
  return (b + 1023) & ~(size_t)1023;
}

template <int DT, int D>
bool use_async(int d, int tile_q) {
  if constexpr (!async_stage_ok<DT, D>()) {
    (void)d;
    (void)tile_q;
    return false;
  } else {
    return 2 * stage_bytes<DT, D>(d, tile_q) <= (size_t)76 * 1024;
  }
}

template <int DT, int D, int kMode, int kNT, int kOcc>
hipError_t launch_scan_k(ScanArgs a, int32_t grid, hipStream_t s) {
  // dynamic LDS: what the device's per-work-group LDS leaves beside the
  // kernel's static LDS, at most kMaxDynLds (the attribute is set to that)
  static const size_t dyn_max = [] {
    hipFuncAttributes fa{};
    int dev = 0, per_block = 0;
    if (hipFuncGetAttributes(&fa, (const void*)scan_kernel<DT, D, kMode, kNT, kOcc>) !=
            hipSuccess ||
        hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&per_block, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) !=
            hipSuccess)
      return (size_t)0;
    const size_t left =
        (size_t)per_block > fa.sharedSizeBytes ? (size_t)per_block - fa.sharedSizeBytes : 0;
    return std::min(left, (size_t)kMaxDynLds);
  }();
  if (dyn_max == 0) return hipErrorInvalidValue;
  static const hipError_t attr =
      hipFuncSetAttribute((const void*)scan_kernel<DT, D, kMode, kNT, kOcc>,
                          hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn_max);
  if (attr != hipSuccess) return attr;
  if (a.tile_q > scan_tile_max<kMode, kOcc>() || a.k < 1 || a.k > 64) return hipErrorInvalidValue;
  const size_t one = stage_bytes<DT, D>(a.d, a.tile_q);
  const size_t stage = kMode == kStageAsync ? 2 * one : one;
  // the LDS arena takes what the staging leaves of the work-group's share,
  // at most kArenaLdsMax entries
  const size_t share = kOcc == 1 ? dyn_max : std::min(dyn_max, (size_t)(72 * 1024));
  const size_t room = share > stage ? share - stage : 0;
  a.arena_lds = a.arena_on ? (int32_t)std::min<size_t>(room / sizeof(TileSpill), kArenaLdsMax) : 0;
  if (!a.arena_on) a.spill_cap = 0;
  const size_t lds = stage + (size_t)a.arena_lds * sizeof(TileSpill);
  if (lds > dyn_max) return hipErrorInvalidValue;
  a.stage_u4 = (int32_t)(one / 16);
  a.cand_u4 = (int32_t)(stage / 16);
  hipLaunchKernelGGL((scan_kernel<DT, D, kMode, kNT, kOcc>), dim3(grid), dim3(kNT), lds, s, a);
  return hipGetLastError();
}

template <int DT, int D>
hipError_t launch_scan_t(const ScanArgs& a, int32_t grid, hipStream_t s) {
  if constexpr (rega_ok<DT, D>()) {
    if (a.tile_q > 16 * rega_max_qb<2>())
      return launch_scan_k<DT, D, kStageRegA, kScanThreads, 1>(a, grid, s);
    return launch_scan_k<DT, D, kStageRegA, kScanThreads, 2>(a, grid, s);
  } else {
    if constexpr (D == 768) {
      if (a.wide) return launch_scan_k<DT, D, kStageSync, kScanThreadsWide, 1>(a, grid, s);
    }
    if constexpr (async_stage_ok<DT, D>()) {
      if (use_async<DT, D>(a.d, a.tile_q))
        return launch_scan_k<DT, D, kStageAsync, kScanThreads, 2>(a, grid, s);
    }
    return launch_scan_k<DT, D, kStageSync, kScanThreads, 2>(a, grid, s);
  }
}

// The heavy kernel's static LDS (its candidate buffers) leaves this much of
// the 160 KB for the staged queries.
constexpr int kMaxDynLdsHeavy = 136 * 1024;

template <int DT, int D>
hipError_t launch_heavy_t(const HeavyArgs& a, int32_t grid, hipStream_t s) {
  static const hipError_t attr =
      hipFuncSetAttribute((const void*)scan_heavy_kernel<DT, D>,
                          hipFuncAttributeMaxDynamicSharedMemorySize, kMaxDynLdsHeavy);
  if (attr != hipSuccess) return attr;
  const size_t lds = (size_t)kHeavyQ * lds_row_bytes<DT>(D > 0 ? D : a.d);
  if (lds > (size_t)kMaxDynLdsHeavy) return hipErrorInvalidValue;
  hipLaunchKernelGGL((scan_heavy_kernel<DT, D>), dim3(grid), dim3(64), lds, s, a);
  return hipGetLastError();
}

template <int DT, int D>
hipError_t launch_rank_scores_t(const void* queries, int64_t q0, int32_t nqc,
                                const void* centroids, int32_t nlist, int32_t d, float* scores,
                                hipStream_t s) {
  static const hipError_t attr =
      hipFuncSetAttribute((const void*)rank_scores_kernel<DT, D>,
                          hipFuncAttributeMaxDynamicSharedMemorySize, kMaxDynLds);
  if (attr != hipSuccess) return attr;
  const int rows = tile_rows(DT, d) < 16 * kScreenQB ? tile_rows(DT, d) : 16 * kScreenQB;
  const size_t lds = (size_t)rows * lds_row_bytes<DT>(d);
  if (lds > (size_t)kMaxDynLds) return hipErrorInvalidValue;
  dim3 grid((nqc + rows - 1) / rows, (nlist + kScreenCents - 1) / kScreenCents);
  hipLaunchKernelGGL((rank_scores_kernel<DT, D>), grid, dim3(kScanThreads), lds, s, queries, q0,
                     nqc, centroids, nlist, d, rows, scores);
  return hipGetLastError();
}

}  // namespace

size_t scan_lds_bytes(int dtype, int d, int rows) {
  return (size_t)rows * (dtype == SIEVE_F32 ? lds_row_bytes<SIEVE_F32>(d)
                                            : lds_row_bytes<SIEVE_F16>(d));
}

int tile_rows_wide(int dtype, int d) {
  const int rb = dtype == SIEVE_F32 ? lds_row_bytes<SIEVE_F32>(d) : lds_row_bytes<SIEVE_F16>(d);
  int qb = (150 * 1024) / (16 * rb);
  qb = qb < 1 ? 1 : (qb > kQB ? kQB : qb);
  return 16 * qb;
}

bool scan_wide_supported(int dtype, int d) { return dtype == SIEVE_F16 && d == 768; }

bool scan_uses_rega(int dtype, int d) {
  return (dtype == SIEVE_F16 && (d == 64 || d == 128)) || (dtype == SIEVE_F32 && d == 64);
}

int scan_rega_tile_q(bool dense) { return 16 * (dense ? rega_max_qb<1>() : rega_max_qb<2>()); }

int tile_rows(int dtype, int d) {
  const int rb = dtype == SIEVE_F32 ? lds_row_bytes<SIEVE_F32>(d) : lds_row_bytes<SIEVE_F16>(d);
  int qb = (80 * 1024) / (16 * rb);
  qb = qb < 1 ? 1 : (qb > kQB ? kQB : qb);
  return 16 * qb;
}

namespace {
// Fragment-order copy of the store (the layout FragStream reads): one thread
// per 16-byte slot; slot (B nch + c) 64 + i + 16 s <- segment 4 c + s of copy
// row p = 16 B + i, which is row off[L] + (p - foff[L]) of partition L
// (foff[L] <= p < foff[L + 1]), or a padding row (zeros) past the
// partition's last row; zeros past the row's segments too.
__global__ __launch_bounds__(256) void vector_frag_kernel(
    const char* __restrict__ vectors, const int64_t* __restrict__ off,
    const int64_t* __restrict__ foff, int32_t nlist, int32_t row_bytes, int32_t nch,
    u32x4* __restrict__ frag, int64_t nslots) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nslots;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int l = (int)(i & 63);
    const int64_t bc = i >> 6;  // B nch + c
    const int64_t blk = bc / nch;
    const int c = (int)(bc - blk * nch);
    const int64_t p = blk * 16 + (l & 15);
    // partition of copy row p: the last L with foff[L] <= p
    int lo = 0, hi = nlist;  // foff[lo] <= p < foff[hi]
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (foff[mid] <= p) lo = mid; else hi = mid;
    }
    const int64_t k = p - foff[lo];
    const int seg = 4 * c + (l >> 4);
    u32x4 v = {0u, 0u, 0u, 0u};
    if (k < off[lo + 1] - off[lo] && seg * 16 < row_bytes)
      v = *(const u32x4*)(vectors + (off[lo] + k) * row_bytes + (int64_t)seg * 16);
    frag[i] = v;
  }
}
}  // namespace

size_t vector_frag_bytes(int dtype, int d, int64_t frag_rows) {
  const bool fixed = dtype == SIEVE_F32 ? (d == 64 || d == 128)
                                        : (d == 64 || d == 128 || d == 768);
  if (!fixed || frag_rows <= 0) return 0;
  const int64_t row_bytes = (int64_t)d * (dtype == SIEVE_F32 ? 4 : 2);
  return (size_t)((frag_rows + 15) / 16) * (size_t)((row_bytes + 63) / 64) * 1024;
}

hipError_t launch_vector_frag(int dtype, int d, const void* vectors, const int64_t* offsets,
                              const int64_t* frag_offsets, int32_t nlist, int64_t frag_rows,
                              void* frag, hipStream_t s) {
  const size_t bytes = vector_frag_bytes(dtype, d, frag_rows);
  if (bytes == 0 || nlist < 1) return hipSuccess;
  const int32_t row_bytes = d * (dtype == SIEVE_F32 ? 4 : 2);
  const int64_t nslots = (int64_t)(bytes / 16);
  const int64_t blocks = (nslots + 255) / 256;
  hipLaunchKernelGGL(vector_frag_kernel, dim3((unsigned)(blocks < (1 << 20) ? blocks : (1 << 20))),
                     dim3(256), 0, s, (const char*)vectors, offsets, frag_offsets, nlist,
                     row_bytes, (int32_t)((row_bytes + 63) / 64), (u32x4*)frag, nslots);
  return hipGetLastError();
}

hipError_t launch_scan(int dtype, const ScanArgs& a, int32_t grid, hipStream_t s) {
  if (dtype == SIEVE_F32) {
    switch (a.d) {
      case 64: return launch_scan_t<SIEVE_F32, 64>(a, grid, s);
      case 128: return launch_scan_t<SIEVE_F32, 128>(a, grid, s);
      default: return launch_scan_t<SIEVE_F32, 0>(a, grid, s);
    }
  }
  switch (a.d) {
    case 64: return launch_scan_t<SIEVE_F16, 64>(a, grid, s);
    case 128: return launch_scan_t<SIEVE_F16, 128>(a, grid, s);
    case 768: return launch_scan_t<SIEVE_F16, 768>(a, grid, s);
    default: return launch_scan_t<SIEVE_F16, 0>(a, grid, s);
  }
}

hipError_t launch_scan_heavy(int dtype, const HeavyArgs& a, int32_t grid, hipStream_t s) {
  if (a.nrec <= 0) return hipSuccess;
  if (a.k < 1 || a.k > 64 || grid < 1) return hipErrorInvalidValue;
  if (dtype == SIEVE_F32) {
    switch (a.d) {
      case 64: return launch_heavy_t<SIEVE_F32, 64>(a, grid, s);
      case 128: return launch_heavy_t<SIEVE_F32, 128>(a, grid, s);
      default: return launch_heavy_t<SIEVE_F32, 0>(a, grid, s);
    }
  }
  switch (a.d) {
    case 64: return launch_heavy_t<SIEVE_F16, 64>(a, grid, s);
    case 128: return launch_heavy_t<SIEVE_F16, 128>(a, grid, s);
    case 768: return launch_heavy_t<SIEVE_F16, 768>(a, grid, s);
    default: return launch_heavy_t<SIEVE_F16, 0>(a, grid, s);
  }
}

hipError_t launch_rank_scores(int dtype, const void* queries, int64_t q0, int32_t nqc,
                              const void* centroids, int32_t nlist, int32_t d, float* scores,
                              hipStream_t s) {
  if (dtype == SIEVE_F32) {
    switch (d) {
      case 64: return launch_rank_scores_t<SIEVE_F32, 64>(queries, q0, nqc, centroids, nlist, d, scores, s);
      case 128: return launch_rank_scores_t<SIEVE_F32, 128>(queries, q0, nqc, centroids, nlist, d, scores, s);
      default: return launch_rank_scores_t<SIEVE_F32, 0>(queries, q0, nqc, centroids, nlist, d, scores, s);
    }
  }
  switch (d) {
    case 128: return launch_rank_scores_t<SIEVE_F16, 128>(queries, q0, nqc, centroids, nlist, d, scores, s);
    default: return launch_rank_scores_t<SIEVE_F16, 0>(queries, q0, nqc, centroids, nlist, d, scores, s);
  }
}

}  // namespace sieve
