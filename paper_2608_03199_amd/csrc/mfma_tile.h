// mfma_tile.h -- the query-tile x row-block inner product engine on gfx950 MFMA.
//
// A work-group of 4 wave64 scores up to 16*QB query rows (staged once in LDS)
// against a run of stored rows (list vectors or centroids) streamed straight
// from HBM into registers, 16 rows per wave at a time.  Each output block is
// 16 queries x 16 rows, accumulated in fp32 by
//   fp32 data: v_mfma_f32_16x16x4_f32   (4 MFMAs per 16-dimension chunk)
//   fp16 data: v_mfma_f32_16x16x32_f16  (1 MFMA per 32-dimension chunk)
// The MFMA operand layout gives lane l the (row l%16, k-group l/16) element;
// the k index is remapped so that every lane reads one contiguous 16-byte
// segment per chunk from both operands (the dot product is a sum over k, so
// any bijection applied to both operands leaves it unchanged, and the fixed
// order of the chunk loop makes every score independent of tiling).  The
// 16x16 accumulator puts output (row 4*(l/16)+r, column l%16) in element r of
// lane l.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

#include "sieve_internal.h"

namespace sieve {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <int DT>
struct DTraits;
template <>
struct DTraits<SIEVE_F32> {
  static constexpr int kElem = 4;
  static constexpr int kSegDims = 4;     // dims per 16-byte segment
  static constexpr int kChunkDims = 16;  // dims consumed by the 4 lane groups per chunk
};
template <>
struct DTraits<SIEVE_F16> {
  static constexpr int kElem = 2;
  static constexpr int kSegDims = 8;
  static constexpr int kChunkDims = 32;
};

__device__ __forceinline__ f32x4 mma_chunk_f32(u32x4 a, u32x4 b, f32x4 acc) {
  // whole-vector casts: element-wise casts of vector lanes are not reliable here
  const f32x4 af = __builtin_bit_cast(f32x4, a);
  const f32x4 bf = __builtin_bit_cast(f32x4, b);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(af[0], bf[0], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(af[1], bf[1], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(af[2], bf[2], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(af[3], bf[3], acc, 0, 0, 0);
  return acc;
}

__device__ __forceinline__ f32x4 mma_chunk_f16(u32x4 a, u32x4 b, f32x4 acc) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                __builtin_bit_cast(f16x8, b), acc, 0, 0, 0);
}

template <int DT>
__device__ __forceinline__ f32x4 mma_chunk(u32x4 a, u32x4 b, f32x4 acc) {
  if constexpr (DT == SIEVE_F32)
    return mma_chunk_f32(a, b, acc);
  else
    return mma_chunk_f16(a, b, acc);
}

// One chunk against QB query blocks.  fp32 issues its four k-steps
// k-major across the query blocks, so that consecutive MFMAs write
// different accumulators (a chain of four dependent fp32 MFMAs on one
// accumulator stalls on each result).  Every accumulator still sees its
// k-steps in the same order as mma_chunk_f32: the same bits.
template <int DT, int QB, bool kZero = false>
__device__ __forceinline__ void mma_chunk_qb(const u32x4 (&a)[QB], u32x4 b, f32x4 (&acc)[QB]) {
  // kZero: the accumulators start from zero (their values are not read)
  const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
  if constexpr (DT == SIEVE_F32) {
    const f32x4 bf = __builtin_bit_cast(f32x4, b);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        const f32x4 af = __builtin_bit_cast(f32x4, a[qb]);
        acc[qb] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[k], bf[k],
                                                       (kZero && k == 0) ? zero : acc[qb], 0, 0, 0);
      }
    }
  } else {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) acc[qb] = mma_chunk_f16(a[qb], b, kZero ? zero : acc[qb]);
  }
}

// Base address of this lane's query fragments in LDS.  The offset passes
// through an empty asm so that the compiler cannot treat the fragment loads
// as invariant across row blocks and hoist them all out of the row loop
// (QB x chunks fragments would not fit in registers and would spill).
__device__ __forceinline__ const u32x4* lane_arow(const u32x4* lds, int segs) {
  const int lane = threadIdx.x & 63;
  int off = (lane & 15) * segs + (lane >> 4);
  asm volatile("" : "+v"(off));
  return lds + off;
}

// Geometry of one query row in LDS, in 16-byte segments: 4 segments per chunk
// plus one pad segment that staggers rows across LDS banks.
template <int DT>
struct RowGeom {
  int nchunks;   // ceil(d / kChunkDims)
  int segs;      // 16-byte segments per LDS row (4*nchunks + 1)
  int dsegs;     // real 16-byte segments of a stored row (d / kSegDims)
  __device__ __host__ static RowGeom make(int d) {
    RowGeom g;
    g.nchunks = (d + DTraits<DT>::kChunkDims - 1) / DTraits<DT>::kChunkDims;
    g.segs = 4 * g.nchunks + 1;
    g.dsegs = d / DTraits<DT>::kSegDims;
    return g;
  }
};

template <int DT>
__host__ __device__ inline int lds_row_bytes(int d) {
  return RowGeom<DT>::make(d).segs * 16;
}

// Stage rows of the query tile into LDS: row i (< nrows_pad) <- src(i) or 0.
// src_row(i) returns a pointer to the stored row, or nullptr for padding;
// src_row(0) must be a real row (it stands in as a safe address).  Eight
// segments per thread are loaded per step from always-valid addresses and
// masked afterwards, so their loads are in flight together.
template <int DT, typename SrcRow>
__device__ __forceinline__ void stage_queries(u32x4* lds, const RowGeom<DT>& g, int nrows_pad,
                                              SrcRow src_row) {
  const int total = nrows_pad * g.segs;
  const u32x4* safe = src_row(0);
  constexpr int kBatch = 8;
  for (int e0 = threadIdx.x; e0 < total; e0 += kBatch * blockDim.x) {
    u32x4 v[kBatch];
    bool ok[kBatch];
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {
      const int e = e0 + k * (int)blockDim.x;
      const int i = e / g.segs, s = e - i * g.segs;
      const u32x4* row = e < total ? src_row(i) : nullptr;
      ok[k] = row != nullptr && s < g.dsegs;
      const u32x4* src = ok[k] ? row + s : safe;  // select the address, load unconditionally
      v[k] = *src;
    }
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {
      const int e = e0 + k * (int)blockDim.x;
      if (e < total) lds[e] = ok[k] ? v[k] : u32x4{0u, 0u, 0u, 0u};
    }
  }
}

// Score the 16-row block whose fragments are in b[] against QB query blocks
// (compile-time dimension D: kNC chunks, fragments already in registers).
// Fully unrolled and software-pipelined: the query fragments of chunk c + 1
// are read from LDS while chunk c's MFMAs issue; a scheduling fence after
// each chunk keeps the compiler from hoisting every LDS read (which would
// cost registers and occupancy).
template <int DT, int D, int QB>
__device__ __forceinline__ void score_regs(const u32x4* __restrict__ lds, int segs,
                                           const u32x4 (&b)[D / DTraits<DT>::kChunkDims],
                                           f32x4 (&acc)[QB]) {
  constexpr int kNC = D / DTraits<DT>::kChunkDims;
  const int lane = threadIdx.x & 63;
  const int h = lane >> 4, r16 = lane & 15;
  const u32x4* arow = lane_arow(lds, segs);
  u32x4 a0[QB], a1[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    acc[qb] = f32x4{0.f, 0.f, 0.f, 0.f};
    a0[qb] = arow[qb * 16 * segs];
  }
#pragma unroll
  for (int c = 0; c < kNC; ++c) {
    u32x4(&cur)[QB] = (c & 1) ? a1 : a0;
    u32x4(&nxt)[QB] = (c & 1) ? a0 : a1;
    if (c + 1 < kNC) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) nxt[qb] = arow[qb * 16 * segs + 4 * (c + 1)];
    }
    mma_chunk_qb<DT, QB>(cur, b[c], acc);
    __builtin_amdgcn_sched_barrier(0);
  }
}

// Runtime-dimension variant: fragments are loaded chunk by chunk (one ahead).
template <int DT, int QB>
__device__ __forceinline__ void score_stream(const u32x4* __restrict__ lds, const RowGeom<DT>& g,
                                             const u32x4* __restrict__ vrow, f32x4 (&acc)[QB]) {
  const int lane = threadIdx.x & 63;
  const int h = lane >> 4, r16 = lane & 15;
  const u32x4* arow = lane_arow(lds, g.segs);
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) acc[qb] = f32x4{0.f, 0.f, 0.f, 0.f};
  const u32x4 zero = {0u, 0u, 0u, 0u};
  // segment indices past the row are clamped to segment 0 (a valid address)
  // and masked to zero, so no branch separates the loads
  u32x4 bn = vrow[h < g.dsegs ? h : 0];
  if (h >= g.dsegs) bn = zero;
  for (int c = 0; c < g.nchunks; ++c) {
    const u32x4 bc = bn;
    const int sn = 4 * (c + 1) + h;
    bn = vrow[sn < g.dsegs ? sn : 0];
    if (sn >= g.dsegs) bn = zero;
    u32x4 av[QB];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) av[qb] = arow[qb * 16 * g.segs + 4 * c];
    mma_chunk_qb<DT, QB>(av, bc, acc);
  }
}

// Rows longer than kSliceChunks MFMA chunks stream in slices of that many
// chunks, one slice ahead: two slices occupy registers instead of two rows,
// and each wave still keeps a slice of loads in flight under its MFMAs.
constexpr int kSliceChunks = 8;

// Multiply slice s (chunks [s*kSliceChunks, ...)) of a row block, whose
// fragments are in b[], into acc; the query fragments of the next chunk are
// read from LDS while the current chunk's MFMAs issue.
template <int DT, int D, int QB>
__device__ __forceinline__ void mma_slice(const u32x4* __restrict__ arow, int segs, int s,
                                          const u32x4 (&b)[kSliceChunks], f32x4 (&acc)[QB]) {
  constexpr int kNC = D / DTraits<DT>::kChunkDims;
  const int c0 = s * kSliceChunks;
  u32x4 a0[QB], a1[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) a0[qb] = arow[qb * 16 * segs + 4 * c0];
#pragma unroll
  for (int c = 0; c < kSliceChunks; ++c) {
    if (c0 + c < kNC) {
      u32x4(&cur)[QB] = (c & 1) ? a1 : a0;
      u32x4(&nxt)[QB] = (c & 1) ? a0 : a1;
      if (c + 1 < kSliceChunks && c0 + c + 1 < kNC) {
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) nxt[qb] = arow[qb * 16 * segs + 4 * (c0 + c + 1)];
      }
      mma_chunk_qb<DT, QB>(cur, b[c], acc);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
}

// Fragment buffers in flight per wave: a wave keeps (buffers - 1) row blocks
// (or slices) loading while it multiplies one, so that its loads cover the
// memory latency.  Tiles with few query blocks have few MFMAs per row and
// spare registers, so they buffer deeper.
// Reserve: VGPRs the caller's epilogue keeps live across the stream.
template <int DT, int D, int QB, int Reserve>
constexpr int ring_depth() {
  constexpr int kNC = D / DTraits<DT>::kChunkDims;
  if (kNC > kSliceChunks) return (Reserve > 0 || QB > 3) ? 2 : 3;  // slices of kSliceChunks chunks
  const int per = 4 * kNC;                             // VGPRs per buffered row block
  const int budget = (QB <= 2 ? 96 : (QB <= 4 ? 64 : 40)) - Reserve;
  const int nb = budget / per;
  return nb < 2 ? 2 : (nb > 6 ? 6 : nb);
}

// s_waitcnt immediate (gfx9 encoding): vmcnt(0), expcnt and lgkmcnt not waited.
constexpr int kWaitVmcnt0 = 0x0F70;

// The rows [r0, r1) a stream reads, addressed as a uniform base (row r0)
// plus a 32-bit per-lane byte offset, so that loads take the scalar-base
// form and row arithmetic stays 32-bit.  Callers keep (r1 - r0) * row_bytes
// below 2^31.  Row blocks past the end re-read the last row: every load is
// issued unconditionally, so the load sequence never depends on control flow
// and the compiler's wait counts stay exact.
struct RowStream {
  static constexpr uint32_t kChunkStride = 64;  // bytes from chunk c to c + 1 of a lane
  const char* base;   // row r0
  int nrows;          // r1 - r0
  uint32_t rb;        // row bytes
  __device__ __forceinline__ uint32_t lane_row(int blk) const {
    const int rl = blk * 16 + (int)(threadIdx.x & 15);
    return (uint32_t)(rl < nrows ? rl : nrows - 1);
  }
  // this lane's 16-byte segment of chunk 0 of row block blk
  __device__ __forceinline__ const char* seg_ptr(int blk) const {
    return base + (lane_row(blk) * rb + ((threadIdx.x >> 4) & 3u) * 16u);
  }
};

// The same rows read from a fragment-order copy of the store.  The copy's
// rows are the store's with padding rows (zeros) between partitions, so that
// every partition starts a 16-row block; for each 16-row block B of the copy
// and each 64-byte chunk c of a row it keeps the 64 16-byte segments that
// one fragment load of that block takes, in lane order: segment 4 c + s of
// copy row 16 B + i sits at 16-byte slot (B nch + c) 64 + i + 16 s.  A
// wave's fragment load of a stream block that starts a copy block then reads
// 1 KB of consecutive bytes (two runs per 16-lane group otherwise) instead of
// 16 separate rows, so the address unit coalesces it.  Segments past a row's
// end hold zeros.
struct FragStream {
  static constexpr uint32_t kChunkStride = 1024;
  const char* frag;   // the copy
  int64_t r0;         // stream row 0 = copy row r0
  int nrows;
  uint32_t nch;       // 64-byte chunks per row
  __device__ __forceinline__ const char* seg_ptr(int blk) const {
    const int rl = blk * 16 + (int)(threadIdx.x & 15);
    const int64_t r = r0 + (rl < nrows ? rl : nrows - 1);
    return frag + (((r >> 4) * nch) << 10) +
           (((uint32_t)(r & 15) + (threadIdx.x & 48u)) << 4);
  }
};

// The stream type of a row source: the row-major store or its fragment copy.
// fdelta: copy row minus store row of the stream's rows (fragment copy only).
template <bool kFrag>
__device__ __forceinline__ auto make_row_stream(const char* base, size_t row_bytes, int64_t r0,
                                                int64_t r1, int64_t fdelta) {
  if constexpr (kFrag)
    return FragStream{base, r0 + fdelta, (int)(r1 - r0), (uint32_t)((row_bytes + 63) / 64)};
  else
    return RowStream{base + (size_t)r0 * row_bytes, (int)(r1 - r0), (uint32_t)row_bytes};
}

// f(std::integral_constant<int, J>{}) for J = 0 .. N-1, unrolled at compile
// time (fragment ring indices must be constants: a runtime index would put
// the ring in scratch memory).
template <typename F, int... J>
__device__ __forceinline__ void unroll_steps(F&& f, std::integer_sequence<int, J...>) {
  (f(std::integral_constant<int, J>{}), ...);
}

// Index of this wave in the work-group, as a uniform (scalar) value: the row
// loops below then run on scalar branches and scalar counters.
__device__ __forceinline__ int wave_id() {
  return __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
}

// Sliced variant of stream_rows_qb (see there) for kNC > kSliceChunks.  The
// wave's row blocks form a stream of slices (block k, slice s); slice t loads
// into buffer t % NB while slice t - NB + 1 is multiplied.  NB row blocks are
// unrolled per iteration so that buffer indices are compile-time constants.
// Chunks are accumulated in the same order as in the unsliced variant, so
// scores are bit-identical.
template <int DT, int D, int QB, int Reserve, typename Epi, typename RS>
__device__ __forceinline__ void stream_rows_sliced(const u32x4* __restrict__ lds,
                                                   const RowGeom<DT>& g, const RS& rs,
                                                   int64_t r0, Epi& epi) {
  constexpr int kNC = D / DTraits<DT>::kChunkDims;
  constexpr int kNS = (kNC + kSliceChunks - 1) / kSliceChunks;  // slices per row block
  constexpr int NB = ring_depth<DT, D, QB, Reserve>();
  const int wave = wave_id();
  const int nwaves = blockDim.x >> 6;
  const int r16 = threadIdx.x & 15;
  const int nrows = rs.nrows;
  auto load = [&](int blk, int s, u32x4(&dst)[kSliceChunks]) {
    const char* p = rs.seg_ptr(blk);
#pragma unroll
    for (int c = 0; c < kSliceChunks; ++c)
      if (s * kSliceChunks + c < kNC)
        dst[c] = *(const u32x4*)(p + RS::kChunkStride * (s * kSliceChunks + c));
  };
  u32x4 buf[NB][kSliceChunks];
  int rb = wave;
  if (nrows <= 0) return;
#pragma unroll
  for (int u = 0; u < NB - 1; ++u) load(rb + (u / kNS) * nwaves, u % kNS, buf[u]);
  // Nothing issued before the stream (staging copies, record loads, queue
  // atomics) stays in flight inside it: mixed kinds of pending memory
  // operations would make every wait below a wait for all of them.  (The
  // fences keep the scheduler from moving the prefetch below the wait.)
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
  __builtin_amdgcn_sched_barrier(0);
  f32x4 acc[QB];
  for (;;) {
#pragma unroll
    for (int u = 0; u < NB * kNS; ++u) {
      const int s = u % kNS;
      const int blk = rb + (u / kNS) * nwaves;
      if (blk * 16 >= nrows) return;
      if (s == 0) {
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) acc[qb] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
      const int un = u + NB - 1;  // issue the slice NB - 1 ahead before these MFMAs
      load(rb + (un / kNS) * nwaves, un % kNS, buf[un % NB]);
      // keep the prefetch above the MFMAs (the scheduler would otherwise sink
      // loads towards their use to save registers, serialising the stream)
      __builtin_amdgcn_sched_barrier(0);
      // the fragment base is re-derived per slice: computed once, the loads
      // from it would be loop-invariant and get hoisted (and spilled)
      mma_slice<DT, D, QB>(lane_arow(lds, g.segs), g.segs, s, buf[u % NB], acc);
      if (s == kNS - 1) epi(acc, r0 + blk * 16 + r16);
    }
    rb += NB * nwaves;
  }
}

// Stream rows [r0, r1) of a row-major store through the waves of the block:
// wave w scores row blocks w, w + W, w + 2W, ... (W = waves per block)
// against QB staged query blocks and hands each finished block to
// epi(acc, row), row = the stored row this lane's column holds (it may be
// >= r1 on the last block: the epilogue masks it; loads are clamped).  With a
// compile-time dimension, fragment buffers rotate so that the next blocks'
// fragments load while the current block is multiplied.
template <int DT, int D, int QB, typename Epi, int Reserve = 0, bool kFrag = false>
__device__ __forceinline__ void stream_rows_qb(const u32x4* __restrict__ lds,
                                               const RowGeom<DT>& g,
                                               const char* __restrict__ base, size_t row_bytes,
                                               int64_t r0, int64_t r1, Epi& epi,
                                               int64_t fdelta = 0) {
  const int wave = wave_id();
  const int nwaves = blockDim.x >> 6;
  const int r16 = threadIdx.x & 15;
  static_assert(!kFrag || D > 0, "the fragment copy serves compile-time dimensions");
  const auto rs = make_row_stream<kFrag>(base, row_bytes, r0, r1, fdelta);
  using RS = decltype(rs);
  const int nrows = rs.nrows;
  constexpr int kNC = D / DTraits<DT>::kChunkDims;
  if constexpr (kNC > kSliceChunks) {
    stream_rows_sliced<DT, D, QB, Reserve>(lds, g, rs, r0, epi);
  } else if constexpr (kNC > 0) {
    // NB fragment buffers: block rb + (NB - 1) W loads while block rb is
    // multiplied; NB blocks are unrolled per iteration (compile-time indices)
    constexpr int NB = ring_depth<DT, D, QB, Reserve>();
    auto load = [&](int blk, u32x4(&dst)[kNC]) {
      const char* p = rs.seg_ptr(blk);
#pragma unroll
      for (int c = 0; c < kNC; ++c) dst[c] = *(const u32x4*)(p + RS::kChunkStride * c);
    };
    u32x4 buf[NB][kNC];
    if (nrows <= 0) return;
#pragma unroll
    for (int j = 0; j < NB - 1; ++j) load(wave + j * nwaves, buf[j]);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);  // see stream_rows_sliced
    __builtin_amdgcn_sched_barrier(0);
    int rb = wave;
    for (;;) {
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        if (rb * 16 >= nrows) return;
        load(rb + (NB - 1) * nwaves, buf[(j + NB - 1) % NB]);
        __builtin_amdgcn_sched_barrier(0);  // prefetch stays above the MFMAs
        f32x4 acc[QB];
        score_regs<DT, D, QB>(lds, g.segs, buf[j], acc);
        epi(acc, r0 + rb * 16 + r16);
        rb += nwaves;
      }
    }
  } else if constexpr (!kFrag) {
    for (int rb = wave; rb * 16 < nrows; rb += nwaves) {
      const u32x4* vrow = (const u32x4*)(rs.base + (size_t)rs.lane_row(rb) * rs.rb);
      f32x4 acc[QB];
      score_stream<DT, QB>(lds, g, vrow, acc);
      epi(acc, r0 + rb * 16 + r16);
    }
  }
}

// ---- register-held query fragments ----
// For short rows (at most kRegAChunks MFMA chunks) a wave keeps its A
// fragments for the whole tile in registers instead of reading them from
// LDS for every 16-row block: with 8 query blocks the LDS reads of the
// LDS-staged path (QB * 1 KB per chunk and row block per wave) would exceed
// the LDS bandwidth long before the MFMA pipe is busy.  qf[c][qb] is lane
// l's fragment of chunk c of query block qb (row l % 16, segment 4c + l / 16
// of the staged tile), exactly what score_regs reads, so the scores are
// bit-identical to the LDS-staged path.
constexpr int kRegAChunks = 4;

template <int DT, int D>
constexpr bool rega_ok() {
  return D > 0 && D % DTraits<DT>::kChunkDims == 0 && D / DTraits<DT>::kChunkDims <= kRegAChunks;
}

template <int DT, int D, int QB>
__device__ __forceinline__ void load_afrags(const u32x4* __restrict__ lds, int segs,
                                            u32x4 (&qf)[D / DTraits<DT>::kChunkDims][QB]) {
  constexpr int kNC = D / DTraits<DT>::kChunkDims;
  const int lane = threadIdx.x & 63;
  const u32x4* arow = lds + (lane & 15) * segs + (lane >> 4);
#pragma unroll
  for (int c = 0; c < kNC; ++c) {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) qf[c][qb] = arow[qb * 16 * segs + 4 * c];
  }
}

// Fragment buffers of the register-A stream: the A fragments take 4 * kNC * QB
// registers and the two accumulator sets 8 * QB, so the ring shrinks as QB
// grows.  kRegs: registers per lane of one wave (512 at one wave per SIMD,
// 256 at two).  The ring depth is even (accumulator sets alternate by step).
template <int DT, int D, int QB, int kRegs>
constexpr int rega_ring() {
  constexpr int kNC = D / DTraits<DT>::kChunkDims;
  const int per = 4 * kNC;  // fragments of one row block
  int nb = (kRegs - 4 * kNC * QB - 8 * QB - (kRegs > 256 ? 120 : 130)) / per;
  nb = nb > 8 ? 8 : nb;
  nb &= ~1;
  return nb < 2 ? 2 : nb;
}

// Stream rows [r0, r1) through the block's waves (wave w takes row blocks w,
// w + W, ...) against the register-held fragments qf.  Per 16-row block:
// vote(acc, row), a wave-uniform test computed with straight-line vector
// work, then cand(acc, row) when it holds.  row = the stored row of this
// lane's column; it is >= r1 on the last block and on padding blocks (loads
// are clamped), and the vote then fails.  Chunks are
// multiplied in ascending order into each accumulator, as in score_regs: the
// same bits.  The vote of block b is issued between the MFMAs of block
// b + W (two accumulator sets, interleaving hints), so that it runs under
// them.
template <int DT, int D, int QB, int kRegs, bool kFrag, typename Vote, typename Cand>
__device__ __forceinline__ void stream_rows_rega(const u32x4 (&qf)[D / DTraits<DT>::kChunkDims][QB],
                                                 const char* __restrict__ base, size_t row_bytes,
                                                 int64_t r0, int64_t r1, Vote& vote, Cand& cand,
                                                 int64_t fdelta = 0) {
  constexpr int kNC = D / DTraits<DT>::kChunkDims;
  constexpr int NB = rega_ring<DT, D, QB, kRegs>();
  const int wave = wave_id();
  const int nwaves = blockDim.x >> 6;
  const int r16 = threadIdx.x & 15;
  const auto rs = make_row_stream<kFrag>(base, row_bytes, r0, r1, fdelta);
  using RS = decltype(rs);
  const int nrows = rs.nrows;
  auto load = [&](int blk, u32x4(&dst)[kNC]) {
    const char* p = rs.seg_ptr(blk);
#pragma unroll
    for (int c = 0; c < kNC; ++c) dst[c] = *(const u32x4*)(p + RS::kChunkStride * c);
  };
  u32x4 buf[NB][kNC];
  if (nrows <= 0 || wave * 16 >= nrows) return;
#pragma unroll
  for (int j = 0; j < NB - 1; ++j) load(wave + j * nwaves, buf[j]);
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);  // see stream_rows_sliced
  __builtin_amdgcn_sched_barrier(0);
  f32x4 acc[2][QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) acc[1][qb] = f32x4{0.f, 0.f, 0.f, 0.f};
  int rb = wave;
  int64_t prev_row = r1;  // no block before the first
  // One step per row block of this wave, plus one that only runs the last
  // block's vote, rounded up to whole trips of NB steps: the steps past the
  // end multiply clamped rows whose vote is empty.  Steps are expanded NB at
  // a time at compile time, so that every ring and accumulator index is a
  // constant (a runtime index would put them in scratch), and the loop has no
  // exit inside a trip: an exit path would join the loop header with its own
  // pending loads, and the compiler's wait counts there would turn
  // conservative (a near drain of the ring per trip).
  auto step = [&](auto jc) {
    constexpr int j = decltype(jc)::value;
    constexpr int cur = j & 1, prv = cur ^ 1;  // NB is even
    load(rb + (NB - 1) * nwaves, buf[(j + NB - 1) % NB]);
    // chunk 0 starts each accumulator from zero (an inline constant operand)
    mma_chunk_qb<DT, QB, true>(qf[0], buf[j][0], acc[cur]);
#pragma unroll
    for (int c = 1; c < kNC; ++c) mma_chunk_qb<DT, QB>(qf[c], buf[j][c], acc[cur]);
    const bool some = vote(acc[prv], prev_row);
    // loads first, then the MFMAs with the previous block's vote in between
    __builtin_amdgcn_sched_group_barrier(0x020, kNC, 0);  // VMEM reads
#pragma unroll
    for (int x = 0; x < kNC * QB; ++x) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
      __builtin_amdgcn_sched_group_barrier(0x002, 1, 0);  // one VALU
    }
    if (some) cand(acc[prv], prev_row);
    prev_row = r0 + rb * 16 + r16;
    rb += nwaves;
  };
  const int nsteps = ((nrows + 15) / 16 - wave + nwaves - 1) / nwaves + 1;
  for (int t = (nsteps + NB - 1) / NB; t > 0; --t)
    unroll_steps(step, std::make_integer_sequence<int, NB>{});
}

// Largest number of 16-query blocks a tile of compile-time dimension D can
// stage (the 80 KB LDS budget that keeps two work-groups per CU; the host's
// tile size follows the same rule).  D = 0: runtime dimension, up to 8.
template <int DT, int D, int kBudgetKB = 80>
constexpr int qb_cap() {
  if (D == 0) return 8;
  const int segs = 4 * ((D + DTraits<DT>::kChunkDims - 1) / DTraits<DT>::kChunkDims) + 1;
  const int qb = (kBudgetKB * 1024) / (16 * segs * 16);
  return qb < 1 ? 1 : (qb > 8 ? 8 : qb);
}

template <int DT, int D, int QB, int kMax, bool kFrag, typename Epi>
__device__ __forceinline__ void stream_rows_from(const u32x4* __restrict__ lds,
                                                 const RowGeom<DT>& g,
                                                 const char* __restrict__ base, size_t row_bytes,
                                                 int64_t r0, int64_t r1, int qb_n, Epi& epi,
                                                 int64_t fdelta) {
  if constexpr (QB >= kMax) {
    stream_rows_qb<DT, D, kMax, Epi, 0, kFrag>(lds, g, base, row_bytes, r0, r1, epi, fdelta);
  } else {
    if (qb_n <= QB)
      stream_rows_qb<DT, D, QB, Epi, 0, kFrag>(lds, g, base, row_bytes, r0, r1, epi, fdelta);
    else
      stream_rows_from<DT, D, QB + 1, kMax, kFrag>(lds, g, base, row_bytes, r0, r1, qb_n, epi,
                                                   fdelta);
  }
}

// Dispatch on the tile's number of 16-query blocks (uniform per tile).
// QBLimit: the caller's largest tile, in 16-query blocks; kBudgetKB: the LDS
// budget the caller's tile size follows; kFrag: base is the store's
// fragment-order copy (FragStream, its rows fdelta past the store's), not the
// row-major store.
template <int DT, int D, int QBLimit = 8, int kBudgetKB = 80, bool kFrag = false, typename Epi>
__device__ __forceinline__ void stream_rows(const u32x4* __restrict__ lds, const RowGeom<DT>& g,
                                            const char* __restrict__ base, size_t row_bytes,
                                            int64_t r0, int64_t r1, int qb_n, Epi&& epi,
                                            int64_t fdelta = 0) {
  constexpr int kCap = qb_cap<DT, D, kBudgetKB>();
  constexpr int kMax = kCap < QBLimit ? kCap : QBLimit;
  stream_rows_from<DT, D, 1, kMax, kFrag>(lds, g, base, row_bytes, r0, r1, qb_n, epi, fdelta);
}

}  // namespace sieve
