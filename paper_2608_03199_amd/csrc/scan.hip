// scan.hip -- partition scan (within-partition search, Sec. 2.3 and Sec. 5)
// fused with the tau test, and the centroid-screen GEMM of the ranking step
// (Sec. 4.1).  Both use the MFMA tile engine of mfma_tile.h.
//
// Partition scan: each tile holds up to 16*QB ready items (q_i, j) of one
// partition (Sec. 4.2's partition group) and one chunk of that partition's
// rows.  The queries are staged once in LDS; every wave streams 16 rows at a
// time from HBM into registers and scores them against all staged queries.
// A score that reaches tau (inclusive, Sec. 2.2) for a row whose id is not
// the query's exclusion id makes the probe a hit (Sec. 4.1): the candidate is
// appended to the hit pool and the query's highest hit rank of the round is
// raised with an atomic max.  The hit test depends only on the pair's own
// score, never on other candidates, so it is the same whatever the dispatch
// order (the property the lookahead equivalence of Sec. 4.3 needs).
//
// Work distribution: a persistent grid pulls tiles from a per-XCD work queue
// (see the kernel); every block exits after its claims run dry, at most
// tiles + 8 claims per block.
//
// Candidate pool: a block appends into a run of pool slots (its arena) that
// it claimed with one global atomic, handing out slots with one LDS atomic
// per ballot group of candidates.  A group that does not fit the arena claims
// its slots from the global counter directly, and at the end of that tile the
// block gives the arena's unused tail sentinel entries and claims a run twice
// as long (up to kArenaMax).  The arena carries over to the block's next
// launch in the same search; blocks that never meet a candidate claim nothing.
#include "mfma_tile.h"

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

template <int DT, int D, bool kAsync, int kNT>
__global__ __launch_bounds__(kNT, kNT == kScanThreads ? 2 : 1) void scan_kernel(ScanArgs a) {
  extern __shared__ u32x4 lds[];
  __shared__ int32_t s_q[2][kTileQ];     // item sets: the running tile and the next
  __shared__ int32_t s_rank[2][kTileQ];
  __shared__ int64_t s_ex[2][kTileQ];
  __shared__ int32_t s_hits[kTileQ];  // candidates per staged query in this tile
  __shared__ unsigned long long s_abase;  // first pool slot of the block's arena
  __shared__ int32_t s_asize;  // arena slots (0: no arena)
  __shared__ int32_t s_aused;  // arena slots handed out (may run past s_asize)
  __shared__ int32_t s_afill;  // arena slots actually used (a prefix of the arena)
  __shared__ int32_t s_afall;  // a group fell back to the global counter this tile

  const int d = D > 0 ? D : a.d;
  const RowGeom<DT> g = RowGeom<DT>::make(d);
  const int lane = threadIdx.x & 63;
  const int h = lane >> 4;
  const size_t row_bytes = (size_t)d * DTraits<DT>::kElem;
  const int ntiles = a.rc->ntiles;
  const char* qbase = (const char*)a.queries;
  __shared__ int s_claim;

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
  // loads); thread 0 claims the next one under each tile's MFMAs
  __shared__ int s_first[4];
  if (threadIdx.x == 0) {
    s_first[0] = claim();
    s_first[1] = claim();
    s_first[2] = claim();
    s_first[3] = claim();
  }
  if (threadIdx.x < kTileQ) s_hits[threadIdx.x] = 0;
  if (threadIdx.x == 0) {
    const ArenaRec ar = a.arenas[blockIdx.x];  // the run left by the previous launch
    s_abase = ar.base;
    s_asize = ar.size;
    s_aused = ar.fill;  // no run (size 0): every group takes the global path
    s_afill = ar.fill;
    s_afall = 0;
  }
  __syncthreads();
  int t = s_first[0], tn = s_first[1], ta = s_first[2], tb = s_first[3];
  Tile recT = load_rec(t), recN = load_rec(tn), recA = load_rec(ta);
  BItem itN = load_items(recN);
  put_items(0, recT, load_items(recT));
  int set = 0;
  __syncthreads();
  if constexpr (kAsync) {
    if (t >= 0) dma_stage<DT>(lds, g, qbase, row_bytes, s_q[0], recT.nq);
    __builtin_amdgcn_s_waitcnt(0);
  }
  __syncthreads();

  for (; t >= 0;) {
    // the next tile's items go to the other set
    const int nset = set ^ 1;
    put_items(nset, recN, itN);
    __syncthreads();
    int t_claim = -1;
    if (threadIdx.x == 0) t_claim = claim();  // published at the end of this tile
    u32x4* buf = lds;
    if constexpr (kAsync) {
      buf = lds + set * a.stage_u4;
      if (tn >= 0) dma_stage<DT>(lds + nset * a.stage_u4, g, qbase, row_bytes, s_q[nset], recN.nq);
    } else {
      const int32_t* sq = s_q[set];
      const int nq0 = recT.nq;
      stage_queries<DT>(lds, g, ((nq0 + 15) >> 4) * 16, [&](int i) -> const u32x4* {
        return i < nq0 ? (const u32x4*)(qbase + (size_t)sq[i] * row_bytes) : nullptr;
      });
      __syncthreads();
    }
    // pipeline loads, used one tile from now
    const BItem itA = load_items(recA);
    const Tile recB = load_rec(tb);
    const int32_t* sq = s_q[set];
    const int32_t* srank = s_rank[set];
    const int64_t* sex = s_ex[set];
    const int nq = recT.nq;
    const int qb_n = (nq + 15) >> 4;
    const int64_t r0 = recT.r0, r1 = recT.r0 + recT.nrows;

    // Only the tile's last 16-query block can hold padding rows (qb_n =
    // ceil(nq / 16)); its four rows of this lane get threshold +inf when they
    // are padding, so the test below needs no per-row index compares.
    const float tau = a.tau;
    float thr_last[4];
#pragma unroll
    for (int r = 0; r < 4; ++r)
      thr_last[r] = ((qb_n - 1) * 16 + 4 * h + r) < nq ? tau : INFINITY;
    stream_rows<DT, D, 8, kNT == kScanThreads ? 80 : 150>(
          buf, g, (const char*)a.vectors, row_bytes, r0, r1, qb_n,
          [&](const auto& acc, int64_t row) {
            constexpr int QB = sizeof(acc) / sizeof(acc[0]);
            // tau test: one wave-wide vote in the common (no candidate) case;
            // full query blocks through a max tree, the last one per row
            float mx = -INFINITY;
#pragma unroll
            for (int qb = 0; qb + 1 < QB; ++qb) {
#pragma unroll
              for (int r = 0; r < 4; ++r) mx = fmaxf(mx, acc[qb][r]);
            }
            bool any = mx >= tau;
#pragma unroll
            for (int r = 0; r < 4; ++r) any |= acc[QB - 1][r] >= thr_last[r];
            any = any && (row < r1);
            if (__ballot(any) == 0) return;
            // row ids, needed only here (self-exclusion and the pool records)
            const int64_t rid = a.ids[row < r1 ? row : r1 - 1];
            // Candidates: one ballot group (16 rows x 4 queries) takes its
            // pool slots with one LDS atomic on the block's arena; the
            // per-query counts go to LDS (one add per query of the group)
            // and reach global memory once per tile.
            const int r16 = lane & 15;
#pragma unroll
            for (int qb = 0; qb < QB; ++qb) {
              // skip query blocks without a candidate with one vote each
              bool qany;
              if (qb + 1 < QB)
                qany = fmaxf(fmaxf(acc[qb][0], acc[qb][1]), fmaxf(acc[qb][2], acc[qb][3])) >= tau;
              else
                qany = acc[qb][0] >= thr_last[0] || acc[qb][1] >= thr_last[1] ||
                       acc[qb][2] >= thr_last[2] || acc[qb][3] >= thr_last[3];
              if (__ballot(any && qany) == 0) continue;
#pragma unroll
              for (int r = 0; r < 4; ++r) {
                const int i = qb * 16 + 4 * h + r;
                const float sc = acc[qb][r];
                bool hit = any && (sc >= (qb + 1 < QB ? tau : thr_last[r]));
                if (__ballot(hit) == 0) continue;
                hit = hit && rid != sex[i];  // self-exclusion, read only for qualifying pairs
                const unsigned long long mask = __ballot(hit);
                if (mask == 0) continue;
                const int leader = __ffsll((long long)mask) - 1;  // wave-uniform
                const int cnt = __popcll(mask);
                int o = 0;
                if (lane == leader) {
                  o = atomicAdd(&s_aused, cnt);
                  if (o + cnt <= s_asize) atomicAdd(&s_afill, cnt);
                }
                o = __builtin_amdgcn_readlane(o, leader);
                unsigned long long base;
                if (o + cnt <= s_asize) {  // wave-uniform; the common case
                  base = s_abase + (unsigned long long)o;
                } else {
                  // The global claim sits in its own branch: waiting for its
                  // result also waits for every load in flight (the prefetched
                  // rows), which must not happen on the common path.
                  unsigned long long gb = 0;
                  if (lane == leader) {
                    gb = atomicAdd(a.pool_count, (unsigned long long)cnt);
                    s_afall = 1;
                  }
                  base = ((unsigned long long)(uint32_t)__builtin_amdgcn_readlane(
                              (int)(gb >> 32), leader) << 32) |
                         (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)gb, leader);
                }
                if (hit) {
                  const unsigned long long slot =
                      base + (unsigned long long)__popcll(mask & ((1ull << lane) - 1ull));
                  if ((int64_t)slot < a.pool_cap) {
                    Hit hv;
                    hv.score = sc;
                    hv.q = a.hitbits ? (sq[i] | (srank[i] << kRankShift)) : sq[i];
                    hv.id = rid;
                    a.pool[slot] = hv;
                  }
                }
                if (r16 == 0) {
                  const int c = __popcll((mask >> (16 * h)) & 0xffffull);
                  if (c) atomicAdd(&s_hits[i], c);
                }
              }
            }
            // The candidate path issued global stores.  While stores and
            // loads are both in flight the compiler can only wait for all
            // of them before the next row block's MFMAs (including the
            // prefetch just issued); draining the stores here, on this rare
            // path, keeps the row loop's waits partial.
            __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
          });
    if constexpr (kAsync) __builtin_amdgcn_s_waitcnt(0);  // this wave's staging copies landed
    __syncthreads();  // every wave is done with this tile's buffer and items
    {
      // candidates of the tile, for the round statistics: one add per wave
      unsigned long long c = (int)threadIdx.x < nq ? (unsigned long long)s_hits[threadIdx.x] : 0;
      for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o);
      if (lane == 0 && c) atomicAdd(&a.rc->cands, c);
    }
    if ((int)threadIdx.x < nq && s_hits[threadIdx.x] > 0) {
      // this tile's candidates of one query: one count update, one hit flag
      const int q = sq[threadIdx.x];
      atomicAdd(&a.hcount[q], s_hits[threadIdx.x]);
      atomicMax(&a.lmax[q], srank[threadIdx.x] + 1);
      if (a.hitbits) {
        const int rk = srank[threadIdx.x];
        atomicOr(&a.hitbits[(int64_t)q * a.hit_words + (rk >> 5)], 1u << (rk & 31));
      }
      s_hits[threadIdx.x] = 0;
    }
    const bool refill = s_afall != 0;  // block-uniform: written before the barrier
    if (refill) {
      // sentinels over the unused tail of the arena being replaced
      const unsigned long long ab = s_abase;
      const Hit none = {-INFINITY, -1, -1};
      for (int i = s_afill + (int)threadIdx.x; i < s_asize; i += blockDim.x) {
        const unsigned long long slot = ab + (unsigned long long)i;
        if ((int64_t)slot < a.pool_cap) a.pool[slot] = none;
      }
      __syncthreads();  // everyone has read the old arena before it is replaced
    }
    if (threadIdx.x == 0) {
      s_claim = t_claim;
      if (refill) {
        const int sz = s_asize == 0 ? kArenaMin : min(2 * s_asize, kArenaMax);
        s_abase = atomicAdd(a.pool_count, (unsigned long long)sz);
        s_asize = sz;
        s_aused = 0;
        s_afill = 0;
        s_afall = 0;
      }
    }
    __syncthreads();
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
  if (threadIdx.x == 0) {
    ArenaRec ar;
    ar.base = s_abase;
    ar.size = s_asize;
    ar.fill = s_afill;
    a.arenas[blockIdx.x] = ar;
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

template <int DT, int D, bool kAsync, int kNT>
hipError_t launch_scan_k(ScanArgs a, int32_t grid, hipStream_t s) {
  static const hipError_t attr =
      hipFuncSetAttribute((const void*)scan_kernel<DT, D, kAsync, kNT>,
                          hipFuncAttributeMaxDynamicSharedMemorySize, kMaxDynLds);
  if (attr != hipSuccess) return attr;
  const size_t one = stage_bytes<DT, D>(a.d, a.tile_q);
  const size_t lds = kAsync ? 2 * one : one;
  if (lds > (size_t)kMaxDynLds) return hipErrorInvalidValue;
  a.stage_u4 = (int32_t)(one / 16);
  hipLaunchKernelGGL((scan_kernel<DT, D, kAsync, kNT>), dim3(grid), dim3(kNT), lds, s, a);
  return hipGetLastError();
}

template <int DT, int D>
hipError_t launch_scan_t(const ScanArgs& a, int32_t grid, hipStream_t s) {
  if constexpr (D == 768) {
    if (a.wide) return launch_scan_k<DT, D, false, kScanThreadsWide>(a, grid, s);
  }
  if constexpr (async_stage_ok<DT, D>()) {
    if (use_async<DT, D>(a.d, a.tile_q)) return launch_scan_k<DT, D, true, kScanThreads>(a, grid, s);
  }
  return launch_scan_k<DT, D, false, kScanThreads>(a, grid, s);
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

int tile_rows(int dtype, int d) {
  const int rb = dtype == SIEVE_F32 ? lds_row_bytes<SIEVE_F32>(d) : lds_row_bytes<SIEVE_F16>(d);
  int qb = (80 * 1024) / (16 * rb);
  qb = qb < 1 ? 1 : (qb > kQB ? kQB : qb);
  return 16 * qb;
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
    case 128: return launch_scan_t<SIEVE_F16, 128>(a, grid, s);
    case 768: return launch_scan_t<SIEVE_F16, 768>(a, grid, s);
    default: return launch_scan_t<SIEVE_F16, 0>(a, grid, s);
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
