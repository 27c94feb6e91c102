// rank_prefix.hip -- the first R entries of many queries' centroid orders
// (Sec. 4.1's P_i prefix), exact in fp64, without materialising the query x
// centroid score matrix.
//
// A work-group stages up to 64 queries in LDS and streams every centroid
// through the MFMA engine of mfma_tile.h twice:
//   pass 1: each lane keeps, for each of its query rows, the two largest
//     screen scores of the centroids it sees (64 lanes see disjoint centroid
//     sets per query).  The R-th largest of these 128 values belongs to R
//     distinct centroids, so it is at most the R-th largest screen score v;
//     lo = that value - 2 delta is then a valid lower limit for the
//     candidates (rank_common.h);
//   pass 2: recomputes the same scores (same instruction sequence, so the
//     same bits) and appends every centroid with s32 >= lo to the query's
//     candidate list in global memory.
// A second kernel (one wave per query) sorts each list, re-scores near-tie
// runs in fp64 and writes the first R centroids.  A query with more than
// `cap` candidates (or fewer than R) sets rank_error: the caller re-ranks
// from materialised scores with a wide buffer.
#include <type_traits>

#include "mfma_tile.h"
#include "rank_common.h"

namespace sieve {
namespace {

constexpr int kPrefixQB = 4;           // 16-query blocks per 256-thread work-group, at most
constexpr int kPrefixQBWide = 6;       // the same for the 512-thread configuration
constexpr int kPrefixRowsMax = 16 * kPrefixQBWide;
// Wide configuration: one 512-thread work-group per CU with up to 150 KB of
// staged queries, for long rows (fewer passes of the centroids per query).
constexpr int kPrefixThreadsWide = 512;
constexpr int kPrefixBudgetWideKB = 150;

// values kept per query after pass 1: 2 per (column, wave)
template <int kNT>
constexpr int prefix_keep() {
  return 2 * 16 * (kNT / 64);
}

template <int DT, int D, int QB, int kNT>
__device__ __forceinline__ void prefix_body(
    u32x4* lds, const RowGeom<DT>& g, const void* __restrict__ queries, int64_t q0, int qt0,
    int nq, const void* __restrict__ centroids, const char* __restrict__ cfrag, int32_t nlist,
    int d, int32_t R, double cmax, int32_t cap, unsigned long long* __restrict__ cand,
    float* s_lo, int32_t* s_cnt) {
  // compile-time dimensions read the fragment-order centroid copy
  constexpr bool kFrag = D > 0;
  const char* crows = kFrag ? cfrag : (const char*)centroids;
  constexpr int kKeep = prefix_keep<kNT>();
  constexpr int kWaves = kNT / 64;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int h = lane >> 4, r16 = lane & 15;
  const size_t row_bytes = (size_t)d * DTraits<DT>::kElem;
  const char* qbase = (const char*)queries + (size_t)(q0 + qt0) * row_bytes;
  auto stage = [&]() {
    stage_queries<DT>(lds, g, QB * 16, [&](int i) -> const u32x4* {
      return i < nq ? (const u32x4*)(qbase + (size_t)i * row_bytes) : nullptr;
    });
  };

  // pass 1: two largest screen scores per (query row, lane)
  float m1[QB * 4], m2[QB * 4];
#pragma unroll
  for (int x = 0; x < QB * 4; ++x) m1[x] = m2[x] = -INFINITY;
  auto top2 = [&](const auto& acc, int64_t c) {
    const bool ok = c < nlist;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int x = qb * 4 + r;
        // top two of {m1 >= m2, s}: the median of the three is the new second
        const float s = ok ? acc[qb][r] : -INFINITY;
        m2[x] = __builtin_amdgcn_fmed3f(m1[x], m2[x], s);
        m1[x] = fmaxf(m1[x], s);
      }
    }
  };
  stream_rows_qb<DT, D, QB, decltype(top2), 8 * QB, kFrag>(lds, g, crows, row_bytes, 0, nlist,
                                                           top2);
  __syncthreads();  // the staged queries are dead until re-staged below

  float* keep = (float*)lds;  // [QB * 16][kKeep]
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = qb * 16 + 4 * h + r;
      float* dst = keep + i * kKeep + (wave * 16 + r16) * 2;
      dst[0] = m1[qb * 4 + r];
      dst[1] = m2[qb * 4 + r];
    }
  }
  __syncthreads();

  // lower limit per query: R-th largest kept value (bitwise search over the
  // order-preserving keys), less 2 delta, rounded down to fp32
  for (int i = wave; i < nq; i += kWaves) {
    constexpr int kPer = kKeep / 64;  // kept values per lane
    uint32_t kv[kPer];
#pragma unroll
    for (int j = 0; j < kPer; ++j) kv[j] = f2key(keep[i * kKeep + kPer * lane + j]);
    uint32_t prefix = 0;
    for (int bit = 31; bit >= 0; --bit) {
      const uint32_t c = prefix | (1u << bit);
      int cnt = 0;
#pragma unroll
      for (int j = 0; j < kPer; ++j) cnt += __popcll(__ballot(kv[j] >= c));
      if (cnt >= R) prefix = c;
    }
    double ss = 0.0;
    for (int t = lane; t < d; t += 64) {
      const double v = load_elem<DT>(queries, (q0 + qt0 + i) * d + t);
      ss += v * v;
    }
    for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
    const double delta =
        2.0 * (double)(d + 2) * 5.9604644775390625e-08 * sqrt(ss) * cmax + 1e-30;
    const double lo = (double)key2f(prefix) - 2.0 * delta;
    float lof = (float)lo;
    if ((double)lof > lo) lof = nextafterf(lof, -INFINITY);
    if (lane == 0) s_lo[i] = lof;
  }
  __syncthreads();
  stage();
  __syncthreads();

  // pass 2: append every centroid at or above the limit
  float lim[QB * 4];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = qb * 16 + 4 * h + r;
      lim[qb * 4 + r] = i < nq ? s_lo[i] : INFINITY;
    }
  }
  auto collect = [&](const auto& acc, int64_t c) {
    const bool ok = c < nlist;
    bool any = false;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
#pragma unroll
      for (int r = 0; r < 4; ++r) any |= ok && acc[qb][r] >= lim[qb * 4 + r];
    }
    if (__ballot(any) == 0) return;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float s = acc[qb][r];
        if (ok && s >= lim[qb * 4 + r]) {
          const int i = qb * 16 + 4 * h + r;
          const int slot = atomicAdd(&s_cnt[i], 1);
          if (slot < cap)
            cand[(int64_t)(qt0 + i) * cap + slot] =
                ((unsigned long long)(~f2key(s)) << 32) | (unsigned)c;
        }
      }
    }
  };
  stream_rows_qb<DT, D, QB, decltype(collect), 4 * QB, kFrag>(lds, g, crows, row_bytes, 0,
                                                              nlist, collect);
}

template <int DT, int D, int kNT>
__global__ __launch_bounds__(kNT, kNT == 256 ? 2 : 1) void rank_prefix_kernel(
    const void* __restrict__ queries, int64_t q0, int32_t nqc, const void* __restrict__ centroids,
    const char* __restrict__ cfrag, int32_t nlist, int32_t dd, int32_t R, int32_t rows,
    double cmax, int32_t cap, unsigned long long* __restrict__ cand,
    int32_t* __restrict__ ccount) {
  extern __shared__ u32x4 lds[];
  __shared__ float s_lo[kPrefixRowsMax];
  __shared__ int32_t s_cnt[kPrefixRowsMax];
  const int d = D > 0 ? D : dd;
  const RowGeom<DT> g = RowGeom<DT>::make(d);
  const int qt0 = blockIdx.x * rows;
  const int nq = min(rows, nqc - qt0);
  const int qb_n = (nq + 15) >> 4;
  if (threadIdx.x < kPrefixRowsMax) s_cnt[threadIdx.x] = 0;
  // stage once here; the body re-stages after pass 1
  const size_t row_bytes = (size_t)d * DTraits<DT>::kElem;
  const char* qbase = (const char*)queries + (size_t)(q0 + qt0) * row_bytes;
  stage_queries<DT>(lds, g, qb_n * 16, [&](int i) -> const u32x4* {
    return i < nq ? (const u32x4*)(qbase + (size_t)i * row_bytes) : nullptr;
  });
  __syncthreads();
  // the host sizes rows by the same LDS rule, so qb_n <= kQBMax
  constexpr int kCap = kNT == 256 ? qb_cap<DT, D>() : qb_cap<DT, D, kPrefixBudgetWideKB>();
  constexpr int kLim = kNT == 256 ? kPrefixQB : kPrefixQBWide;
  constexpr int kQBMax = kCap < kLim ? kCap : kLim;
#define SIEVE_BODY(QB)                                                                       \
  prefix_body<DT, D, QB, kNT>(lds, g, queries, q0, qt0, nq, centroids, cfrag, nlist, d, R, cmax, \
                              cap, cand, s_lo, s_cnt)
  switch (qb_n) {
    case 1: SIEVE_BODY(1); break;
    case 2: if constexpr (kQBMax >= 2) SIEVE_BODY(2); break;
    case 3: if constexpr (kQBMax >= 3) SIEVE_BODY(3); break;
    case 4: if constexpr (kQBMax >= 4) SIEVE_BODY(4); break;
    case 5: if constexpr (kQBMax >= 5) SIEVE_BODY(5); break;
    default: if constexpr (kQBMax >= 6) SIEVE_BODY(6); break;
  }
#undef SIEVE_BODY
  __syncthreads();
  if ((int)threadIdx.x < nq) ccount[qt0 + threadIdx.x] = s_cnt[threadIdx.x];
}

// Register-query variant for short fp16 rows (at most 128 dimensions).  The
// eight waves of a work-group form 8 / kQRSplit groups; a group owns kQW
// 16-query blocks, whose MFMA fragments each of its waves keeps in registers
// for the whole kernel, and its kQRSplit waves split the centroid row blocks
// (wave j of a group takes blocks j, j + kQRSplit, ...).  A pass over the
// centroids thus serves kQRRows = 128 queries (twice the LDS-staged kernel)
// and reads no LDS in its inner loop.  Each query row is seen by 16 kQRSplit
// lanes holding disjoint centroid sets; pass 1 keeps their two largest
// screen scores, so the R-th largest of those 128 values is at most the R-th
// largest screen score (the bound of rank_prefix_kernel, just as tight).
// Pass 2 recomputes the same scores (the same instruction sequence, so the
// same bits) and appends every centroid at or above the limit.
constexpr int kQRWaves = 8;
constexpr int kQRSplit = 4;
constexpr int kQW = 4;
constexpr int kQRRows = (kQRWaves / kQRSplit) * kQW * 16;  // queries per work-group
constexpr int kQRKeep = 2 * 16 * kQRSplit;                // kept values per query
constexpr int kQRRing = 4;                                 // centroid fragment buffers

template <int D>
__global__ __launch_bounds__(kQRWaves * 64, 1) void rank_prefix_qreg_kernel(
    const void* __restrict__ queries, int64_t q0, int32_t nqc, const char* __restrict__ cfrag,
    int32_t nlist, int32_t R, double cmax, int32_t cap, unsigned long long* __restrict__ cand,
    int32_t* __restrict__ ccount, int32_t nblk1) {
  constexpr int DT = SIEVE_F16;
  constexpr int kNC = D / DTraits<DT>::kChunkDims;
  static_assert(kNC >= 1 && kNC <= 4, "short rows only");
  __shared__ float s_keep[kQRRows * kQRKeep];
  __shared__ float s_lo[kQRRows];
  __shared__ double s_ss[kQRRows];  // squared query norms (fp64, exact from fp16)
  __shared__ int32_t s_cnt[kQRRows];
  const int lane = threadIdx.x & 63;
  const int wave = wave_id();
  const int grp = wave / kQRSplit, mem = wave % kQRSplit;
  const int h = lane >> 4, r16 = lane & 15;
  const size_t row_bytes = (size_t)D * 2;
  for (int i = threadIdx.x; i < kQRRows; i += blockDim.x) s_cnt[i] = 0;
  const int qt0 = blockIdx.x * kQRRows;  // first query of the work-group
  const int w0 = grp * kQW * 16;         // first local query row of the group
  // A operand: lane l supplies query row (block qb, row l % 16), segment 4c + l / 16
  u32x4 qf[kQW][kNC];
#pragma unroll
  for (int qb = 0; qb < kQW; ++qb) {
    const int row = qt0 + w0 + qb * 16 + r16;
    const bool ok = row < nqc;
    const char* src = (const char*)queries + (size_t)(q0 + (ok ? row : 0)) * row_bytes;
#pragma unroll
    for (int c = 0; c < kNC; ++c) {
      const u32x4 v = *(const u32x4*)(src + (size_t)(4 * c + h) * 16);
      qf[qb][c] = ok ? v : u32x4{0u, 0u, 0u, 0u};
    }
  }
  // squared norms of the group's query rows from the fragments: the four
  // lanes of a row (l / 16 = 0..3) hold its 16-byte segments 4c + l / 16
  if (mem == 0) {
#pragma unroll
    for (int qb = 0; qb < kQW; ++qb) {
      double ss = 0.0;
#pragma unroll
      for (int c = 0; c < kNC; ++c) {
        const f16x8 hv = __builtin_bit_cast(f16x8, qf[qb][c]);
#pragma unroll
        for (int e = 0; e < 8; ++e) ss += (double)hv[e] * (double)hv[e];
      }
      ss += __shfl_xor(ss, 16);
      ss += __shfl_xor(ss, 32);
      if (h == 0) s_ss[w0 + qb * 16 + r16] = ss;
    }
  }

  const int nblk = (nlist + 15) >> 4;
  // this lane's 16-byte slot of chunk 0 of block 0 in the fragment-order copy
  const char* fbase = cfrag + (size_t)lane * 16;
  // This wave's centroid row blocks (mem, mem + kQRSplit, ...) against its
  // group's query blocks.  Fragments come through a ring of kQRRing buffers
  // (kQRRing - 1 blocks in flight: the centroids come from L2, whose latency
  // one block's 16 MFMAs do not cover), and the epilogue is software-
  // pipelined: the MFMAs of block t issue interleaved with the VALU work
  // fast(acc, blk) of block t - 1, which returns whether slow(acc, blk) must
  // run for that block.  A fixed number of ring rounds runs; padding blocks
  // (past the last) skip their epilogue.
  auto sweep = [&](int nb, auto&& fast, auto&& slow) {
    u32x4 buf[kQRRing][kNC];
    f32x4 acc[2][kQW];
    // a wave's fragment load reads 1 KB of consecutive bytes (row-major
    // rows would put the 64 lanes' 16-byte pieces on 16 rows, and the
    // address unit would take each lane's piece on its own)
    auto load = [&](int blk, u32x4(&dst)[kNC]) {
      const char* p = fbase + (size_t)(blk < nb ? blk : nb - 1) * (kNC * 1024);
#pragma unroll
      for (int c = 0; c < kNC; ++c) dst[c] = *(const u32x4*)(p + 1024 * c);
    };
#pragma unroll
    for (int u = 0; u < kQRRing - 1; ++u) load(mem + u * kQRSplit, buf[u]);
    // Wait for the prologue here: with loads of the prologue (or from before
    // it) still pending where the loop is entered, the compiler's load waits
    // at the top of each ring round are for every load, not just the oldest.
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    __builtin_amdgcn_sched_barrier(0);
    const int mine = mem < nb ? (nb - mem + kQRSplit - 1) / kQRSplit : 0;
    const int rounds = (mine + kQRRing - 1) / kQRRing;
    int blk = mem;
    for (int it = 0; it < rounds; ++it) {
      unroll_steps([&](auto uc) {
        constexpr int u = decltype(uc)::value;
        constexpr int cur = u & 1, prev = cur ^ 1;  // kQRRing is even
        load(blk + (kQRRing - 1) * kQRSplit, buf[(u + kQRRing - 1) % kQRRing]);
        __builtin_amdgcn_sched_barrier(0);
        auto multiply = [&]() {
#pragma unroll
          for (int qb = 0; qb < kQW; ++qb) acc[cur][qb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int c = 0; c < kNC; ++c) {
            u32x4 a[kQW];
#pragma unroll
            for (int qb = 0; qb < kQW; ++qb) a[qb] = qf[qb][c];
            mma_chunk_qb<DT, kQW>(a, buf[u][c], acc[cur]);
          }
        };
        const int pblk = blk - kQRSplit;
        // the previous block's columns that hold real centroids (none before
        // the first block); the epilogue runs branch-free under this mask so
        // that it issues interleaved with this block's MFMAs
        // (blocks past nb are clamped re-loads of block nb - 1: when pass 1
        // covers a subset, their columns are real centroids seen twice, and
        // a duplicate kept value could raise the bound)
        const bool pok = (u > 0 || it > 0) && pblk < nb && pblk * 16 + r16 < nlist;
        multiply();
        const bool need = fast(acc[prev], pok);
#pragma unroll
        for (int x = 0; x < kQW * kNC; ++x) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
          __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);  // three VALU
        }
        if (__ballot(need) != 0) slow(acc[prev], pblk);
        blk += kQRSplit;
      }, std::make_integer_sequence<int, kQRRing>{});
    }
    // the last block's epilogue
    const int lblk = blk - kQRSplit;
    if (rounds > 0 && lblk < nb) {
      constexpr int last = (kQRRing - 1) & 1;
      if (__ballot(fast(acc[last], lblk * 16 + r16 < nlist)) != 0) slow(acc[last], lblk);
    }
  };

  // pass 1: the two largest screen scores per (lane, query row)
  float pinf = INFINITY;
  asm volatile("" : "+v"(pinf));
  float m1[kQW * 4], m2[kQW * 4];
#pragma unroll
  for (int x = 0; x < kQW * 4; ++x) m1[x] = m2[x] = -INFINITY;
  sweep(nblk1,
      [&](const f32x4(&acc)[kQW], bool ok) -> bool {
#pragma unroll
        for (int qb = 0; qb < kQW; ++qb) {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int x = qb * 4 + r;
            // top two of {m1 >= m2, s}: the median of the three is the new
            // second, the median of {m1, s, +inf} the new first (+inf passes
            // through an empty asm so that the median is not rewritten as a
            // maximum, which would canonicalise its operands first)
            const float sc = ok ? acc[qb][r] : -INFINITY;
            m2[x] = __builtin_amdgcn_fmed3f(m1[x], m2[x], sc);
            m1[x] = __builtin_amdgcn_fmed3f(m1[x], sc, pinf);
          }
        }
        return false;
      },
      [&](const f32x4(&)[kQW], int) {});
#pragma unroll
  for (int qb = 0; qb < kQW; ++qb) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float* dst = s_keep + (w0 + qb * 16 + 4 * h + r) * kQRKeep + (mem * 16 + r16) * 2;
      dst[0] = m1[qb * 4 + r];
      dst[1] = m2[qb * 4 + r];
    }
  }
  __syncthreads();

  // lower limit per query: R-th largest kept value (bitwise search over the
  // order-preserving keys), less 2 delta, rounded down to fp32
  for (int i = wave; i < kQRRows; i += kQRWaves) {
    constexpr int kPer = kQRKeep / 64;  // kept values per lane
    uint32_t kv[kPer];
#pragma unroll
    for (int j = 0; j < kPer; ++j) kv[j] = f2key(s_keep[i * kQRKeep + kPer * lane + j]);
    uint32_t prefix = 0;
    for (int bit = 31; bit >= 0; --bit) {
      const uint32_t c = prefix | (1u << bit);
      int cnt = 0;
#pragma unroll
      for (int j = 0; j < kPer; ++j) cnt += __popcll(__ballot(kv[j] >= c));
      if (cnt >= R) prefix = c;
    }
    const int row = qt0 + i;
    const double ss = s_ss[i];
    const double delta =
        2.0 * (double)(D + 2) * 5.9604644775390625e-08 * sqrt(ss) * cmax + 1e-30;
    const double lo = (double)key2f(prefix) - 2.0 * delta;
    float lof = (float)lo;
    if ((double)lof > lo) lof = nextafterf(lof, -INFINITY);
    if (lane == 0) s_lo[i] = row < nqc ? lof : INFINITY;
  }
  __syncthreads();

  // pass 2: append every centroid at or above its query's limit
  float lim[kQW * 4];
#pragma unroll
  for (int qb = 0; qb < kQW; ++qb) {
#pragma unroll
    for (int r = 0; r < 4; ++r) lim[qb * 4 + r] = s_lo[w0 + qb * 16 + 4 * h + r];
  }
  sweep(nblk,
      [&](const f32x4(&acc)[kQW], bool ok) -> bool {
        bool any = false;
#pragma unroll
        for (int qb = 0; qb < kQW; ++qb) {
#pragma unroll
          for (int r = 0; r < 4; ++r) any |= acc[qb][r] >= lim[qb * 4 + r];
        }
        return ok && any;
      },
      [&](const f32x4(&acc)[kQW], int blk) {
        const int c = blk * 16 + r16;
        const bool ok = c < nlist;
#pragma unroll
        for (int qb = 0; qb < kQW; ++qb) {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float sc = acc[qb][r];
            if (ok && sc >= lim[qb * 4 + r]) {
              const int i = w0 + qb * 16 + 4 * h + r;  // local query row
              const int slot = atomicAdd(&s_cnt[i], 1);
              if (slot < cap)
                cand[(int64_t)(qt0 + i) * cap + slot] =
                    ((unsigned long long)(~f2key(sc)) << 32) | (unsigned)c;
            }
          }
        }
      });
  __syncthreads();
  for (int i = threadIdx.x; i < kQRRows; i += blockDim.x)
    if (qt0 + i < nqc) ccount[qt0 + i] = s_cnt[i];
}

// One wave per query: sort the candidate list, order near-tie runs in fp64,
// write the first R centroids.
template <int DT>
__global__ __launch_bounds__(256) void rank_prefix_finish_kernel(
    const void* __restrict__ queries, int64_t q0, int32_t nqc, const void* __restrict__ centroids,
    int32_t d, int32_t R, int32_t cap, double cmax,
    const unsigned long long* __restrict__ cand, const int32_t* __restrict__ ccount,
    int32_t* __restrict__ P, int64_t ldp, RoundCounters* rc) {
  extern __shared__ uint8_t smem[];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t ql = (int64_t)blockIdx.x * 4 + wave;
  if (ql >= nqc) return;  // whole wave; no block barrier follows
  uint8_t* region = smem + (size_t)wave * wave_region_bytes(cap);
  unsigned long long* ck = (unsigned long long*)region;  // [cap]
  unsigned long long* out = ck + cap;                    // [cap]
  double* cs = (double*)(out + cap);                     // [cap]
  uint8_t* link = (uint8_t*)(cs + cap);                  // [cap]
  const int64_t qg = q0 + ql;
  const int m = ccount[ql];
  if (m > cap || m < R) {
    if (lane == 0) atomicExch(&rc->rank_error, 1);
    for (int r = lane; r < R; r += 64) P[ql * ldp + r] = r;  // valid placeholder
    return;
  }
  for (int i = lane; i < m; i += 64) ck[i] = cand[ql * cap + i];
  double ss = 0.0;
  for (int t = lane; t < d; t += 64) {
    const double v = load_elem<DT>(queries, qg * d + t);
    ss += v * v;
  }
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
  const double qn = sqrt(ss);
  const double delta = 2.0 * (double)(d + 2) * 5.9604644775390625e-08 * qn * cmax + 1e-30;
  wave_sync();
  finish_candidates_wave<DT>(ck, out, cs, link, m, R, 2.0 * delta, queries, qg, centroids, d, qn,
                             cmax, P + ql * ldp);
}

// Fragment-order copy of the centroids (the layout FragStream reads, one
// partition): one thread per 16-byte slot; slot (B nch + c) 64 + i + 16 s <-
// segment 4 c + s of centroid 16 B + i (zeros past the last centroid or past
// the row's segments).
__global__ __launch_bounds__(256) void centroid_frag_kernel(const char* __restrict__ centroids,
                                                           int32_t nlist, int32_t row_bytes,
                                                           int32_t nch, u32x4* __restrict__ frag,
                                                           int64_t nslots) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= nslots) return;
  const int l = (int)(i & 63);
  const int64_t bc = i >> 6;  // B nch + c
  const int64_t blk = bc / nch;
  const int c = (int)(bc - blk * nch);
  const int64_t row = blk * 16 + (l & 15);
  const int seg = 4 * c + (l >> 4);
  u32x4 v = {0u, 0u, 0u, 0u};
  if (row < nlist && seg * 16 < row_bytes)
    v = *(const u32x4*)(centroids + row * row_bytes + (int64_t)seg * 16);
  frag[i] = v;
}

constexpr int kMaxDynLds = 150 * 1024;

// Query rows per work-group: as many 16-row blocks as the LDS budget holds
// (the kernel's compile-time cap follows the same rule).
template <int DT>
int prefix_rows(int d, bool wide) {
  const int rb = lds_row_bytes<DT>(d);
  const int budget = (wide ? kPrefixBudgetWideKB : 80) * 1024;
  const int lim = wide ? kPrefixQBWide : kPrefixQB;
  int qb = budget / (16 * rb);
  qb = qb < 1 ? 1 : (qb > lim ? lim : qb);
  return 16 * qb;
}

template <int DT, int D, int kNT>
hipError_t launch_prefix_k(const void* queries, int64_t q0, int32_t nqc, const void* centroids,
                           const void* cfrag, int32_t nlist, int32_t d, int32_t R, double cmax,
                           int32_t cap, unsigned long long* cand, int32_t* ccount, hipStream_t s) {
  if (D > 0 && !cfrag) return hipErrorInvalidValue;
  static const hipError_t attr =
      hipFuncSetAttribute((const void*)rank_prefix_kernel<DT, D, kNT>,
                          hipFuncAttributeMaxDynamicSharedMemorySize, kMaxDynLds);
  if (attr != hipSuccess) return attr;
  const int rows = prefix_rows<DT>(d, kNT != 256);
  size_t lds = (size_t)rows * lds_row_bytes<DT>(d);
  const size_t keep = (size_t)rows * prefix_keep<kNT>() * sizeof(float);
  if (keep > lds) lds = keep;
  if (lds > (size_t)kMaxDynLds) return hipErrorInvalidValue;
  hipLaunchKernelGGL((rank_prefix_kernel<DT, D, kNT>), dim3((unsigned)((nqc + rows - 1) / rows)),
                     dim3(kNT), lds, s, queries, q0, nqc, centroids, (const char*)cfrag, nlist, d,
                     R, rows, cmax, cap, cand, ccount);
  return hipGetLastError();
}

// 768-dimension fp16 rows take the wide configuration: 96 queries per pass
// of the centroids instead of 48.
template <int DT, int D>
hipError_t launch_prefix_t(const void* queries, int64_t q0, int32_t nqc, const void* centroids,
                           const void* cfrag, int32_t nlist, int32_t d, int32_t R, double cmax,
                           int32_t cap, unsigned long long* cand, int32_t* ccount, hipStream_t s) {
  if constexpr (DT == SIEVE_F16 && D == 768)
    return launch_prefix_k<DT, D, kPrefixThreadsWide>(queries, q0, nqc, centroids, cfrag, nlist,
                                                      d, R, cmax, cap, cand, ccount, s);
  else
    return launch_prefix_k<DT, D, 256>(queries, q0, nqc, centroids, cfrag, nlist, d, R, cmax, cap,
                                       cand, ccount, s);
}

template <int DT>
hipError_t launch_finish_t(const void* queries, int64_t q0, int32_t nqc, const void* centroids,
                           int32_t d, int32_t R, int32_t cap, double cmax,
                           const unsigned long long* cand, const int32_t* ccount, int32_t* P,
                           int64_t ldp, RoundCounters* rc, hipStream_t s) {
  static const hipError_t attr =
      hipFuncSetAttribute((const void*)rank_prefix_finish_kernel<DT>,
                          hipFuncAttributeMaxDynamicSharedMemorySize, kMaxDynLds);
  if (attr != hipSuccess) return attr;
  const size_t lds = (size_t)4 * wave_region_bytes(cap);
  if (lds > (size_t)kMaxDynLds) return hipErrorInvalidValue;
  hipLaunchKernelGGL((rank_prefix_finish_kernel<DT>), dim3((unsigned)((nqc + 3) / 4)), dim3(256),
                     lds, s, queries, q0, nqc, centroids, d, R, cap, cmax, cand, ccount, P, ldp,
                     rc);
  return hipGetLastError();
}

}  // namespace

// The ranking kernels of compile-time dimensions (the register-query kernel
// for fp16 128, the LDS-staged one for fp16 768 and fp32 64 / 128) read the
// copy; the others read the row-major centroids.
size_t centroid_frag_bytes(int dtype, int d, int32_t nlist) {
  const bool fixed = dtype == SIEVE_F32 ? (d == 64 || d == 128) : (d == 128 || d == 768);
  if (!fixed || nlist <= 0) return 0;
  const int64_t row_bytes = (int64_t)d * (dtype == SIEVE_F32 ? 4 : 2);
  return (size_t)((nlist + 15) / 16) * (size_t)((row_bytes + 63) / 64) * 1024;
}

hipError_t launch_centroid_frag(int dtype, int d, const void* centroids, int32_t nlist, void* frag,
                                hipStream_t s) {
  const size_t bytes = centroid_frag_bytes(dtype, d, nlist);
  if (bytes == 0) return hipSuccess;
  const int32_t row_bytes = d * (dtype == SIEVE_F32 ? 4 : 2);
  const int64_t nslots = (int64_t)(bytes / 16);
  hipLaunchKernelGGL(centroid_frag_kernel, dim3((unsigned)((nslots + 255) / 256)), dim3(256), 0,
                     s, (const char*)centroids, nlist, row_bytes, (int32_t)((row_bytes + 63) / 64),
                     (u32x4*)frag, nslots);
  return hipGetLastError();
}

int rank_prefix_cap(int32_t R, int32_t nlist) {
  const int cap = R + 128;
  return cap < nlist ? cap : nlist;
}

hipError_t launch_rank_prefix(int dtype, const void* queries, int64_t q0, int32_t nqc,
                              const void* centroids, const void* cfrag, int32_t nlist, int32_t d,
                              int32_t R, double cmax, unsigned long long* cand, int32_t* ccount,
                              int32_t* P, int64_t ldp, RoundCounters* rc, int32_t pass1_div,
                              hipStream_t s) {
  if (nqc <= 0) return hipSuccess;
  if (R < 1 || R > kRankPrefixMax || R > nlist) return hipErrorInvalidValue;
  const int cap = rank_prefix_cap(R, nlist);
  hipError_t e;
  if (dtype == SIEVE_F16 && d == 128) {
    if (!cfrag) return hipErrorInvalidValue;
    const unsigned grid = (unsigned)((nqc + kQRRows - 1) / kQRRows);
    // Pass 1 may bound the R-th score from the first 1/div of the centroids
    // (a subset's R-th largest never exceeds the whole set's): a looser bound,
    // so more candidates, for a shorter first pass.  Every wave keeps at least
    // four blocks, so every kept value is finite.
    const int nblk = (nlist + 15) / 16;
    const int div = pass1_div > 1 ? pass1_div : 1;
    int nblk1 = (nblk + div - 1) / div;
    if (nblk1 < 4 * kQRSplit) nblk1 = nblk < 4 * kQRSplit ? nblk : 4 * kQRSplit;
    hipLaunchKernelGGL((rank_prefix_qreg_kernel<128>), dim3(grid), dim3(kQRWaves * 64), 0, s,
                       queries, q0, nqc, (const char*)cfrag, nlist, R, cmax, cap, cand, ccount,
                       nblk1);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return launch_finish_t<SIEVE_F16>(queries, q0, nqc, centroids, d, R, cap, cmax, cand, ccount,
                                      P, ldp, rc, s);
  }
#define SIEVE_PREFIX(DT, D)                                                                  \
  launch_prefix_t<DT, D>(queries, q0, nqc, centroids, cfrag, nlist, d, R, cmax, cap, cand, ccount, \
                         s)
  if (dtype == SIEVE_F32) {
    e = d == 64 ? SIEVE_PREFIX(SIEVE_F32, 64)
                : d == 128 ? SIEVE_PREFIX(SIEVE_F32, 128) : SIEVE_PREFIX(SIEVE_F32, 0);
  } else {
    e = d == 128   ? SIEVE_PREFIX(SIEVE_F16, 128)
        : d == 768 ? SIEVE_PREFIX(SIEVE_F16, 768)
                   : SIEVE_PREFIX(SIEVE_F16, 0);
  }
#undef SIEVE_PREFIX
  if (e != hipSuccess) return e;
  return dtype == SIEVE_F32
             ? launch_finish_t<SIEVE_F32>(queries, q0, nqc, centroids, d, R, cap, cmax, cand,
                                          ccount, P, ldp, rc, s)
             : launch_finish_t<SIEVE_F16>(queries, q0, nqc, centroids, d, R, cap, cmax, cand,
                                          ccount, P, ldp, rc, s);
}

}  // namespace sieve
