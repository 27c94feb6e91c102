// rank.hip -- per-query centroid order P_i (Sec. 4.1), exact in fp64.
//
// The MFMA screen (scan.hip) gives fp32 scores s32[c].  For unit-scale data
// |s32[c] - s64[c]| <= delta, with s64 the fp64 sum of exact products in
// dimension order and delta = 2 (d + 2) 2^-24 |q| max_c |c| (twice the
// standard bound on a length-d fp32 accumulation).  Hence:
//   1. the n-th largest fp32 score v is found by an 8-bit radix select;
//   2. every centroid of the true fp64 top-n has s32 >= v - 2 delta, so the
//      candidates are all c with s32[c] >= v - 2 delta;
//   3. sorted by (s32 desc, c asc), candidates whose successive fp32 gaps are
//      all <= 2 delta form runs; a gap > 2 delta orders two centroids the
//      same way in fp64, so only members of multi-element runs need fp64
//      scores, which are then ordered by (s64 desc, c asc) inside each run;
//   4. the first n candidates are P_i.
// The result equals sorting all centroids by (fp64 score desc, index asc).
#include "sieve_internal.h"

namespace sieve {
namespace {

constexpr int kThreads = 256;

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

// fp64 sum over dimensions in ascending order of exact products q_t * c_t
// (the products of two fp32 or fp16 values are exact in fp64, so fused and
// unfused multiply-adds agree).  Rows are read 16 bytes at a time so that
// loads run ahead of the dependent accumulation.
template <int DT>
__device__ __forceinline__ double dot_fp64(const void* __restrict__ queries, int64_t q,
                                           const void* __restrict__ centroids, int c, int d) {
  typedef uint32_t u4 __attribute__((ext_vector_type(4)));
  constexpr int per = DT == SIEVE_F32 ? 4 : 8;  // elements per 16 bytes
  const int nseg = d / per;                     // d is a multiple of 8
  const u4* qa = (const u4*)((const char*)queries + (size_t)q * d * (DT == SIEVE_F32 ? 4 : 2));
  const u4* ca = (const u4*)((const char*)centroids + (size_t)c * d * (DT == SIEVE_F32 ? 4 : 2));
  double s = 0.0;
#pragma unroll 4
  for (int g = 0; g < nseg; ++g) {
    const u4 qv = qa[g], cv = ca[g];
    if constexpr (DT == SIEVE_F32) {
      const float* qf = (const float*)&qv;
      const float* cf = (const float*)&cv;
#pragma unroll
      for (int e = 0; e < 4; ++e) s += (double)qf[e] * (double)cf[e];
    } else {
      const _Float16* qh = (const _Float16*)&qv;
      const _Float16* ch = (const _Float16*)&cv;
#pragma unroll
      for (int e = 0; e < 8; ++e) s += (double)qh[e] * (double)ch[e];
    }
  }
  return s;
}

template <int DT>
__global__ __launch_bounds__(kThreads) void rank_select_kernel(
    const void* __restrict__ queries, int64_t q0, const void* __restrict__ centroids,
    int32_t nlist, int32_t d, const float* __restrict__ scores, int32_t n, int32_t cap,
    double cmax, int32_t* __restrict__ P, RoundCounters* rc) {
  extern __shared__ uint8_t smem[];
  uint32_t* keys = (uint32_t*)smem;                                    // [nlist]
  unsigned long long* ck = (unsigned long long*)(smem + ((nlist * 4 + 15) & ~15));  // [capp]
  __shared__ int hist[256];
  __shared__ uint32_t s_prefix;
  __shared__ int s_remaining;
  __shared__ int s_m;
  __shared__ double s_red[kThreads / 64];
  __shared__ int s_wsum[kThreads / 64];

  int capp = 1;
  while (capp < cap) capp <<= 1;
  double* cs = (double*)(ck + capp);  // [cap] fp64 scores of run members
  uint8_t* link = (uint8_t*)(cs + cap);  // [cap]

  const int t = threadIdx.x;
  const int64_t ql = blockIdx.x;
  const int64_t qg = q0 + ql;
  const float* row = scores + ql * nlist;

  // |q| in fp64
  double ss = 0.0;
  for (int i = t; i < d; i += kThreads) {
    const double v = load_elem<DT>(queries, qg * d + i);
    ss += v * v;
  }
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
  if ((t & 63) == 0) s_red[t >> 6] = ss;
  for (int c = t; c < nlist; c += kThreads) keys[c] = f2key(row[c]);
  if (t == 0) {
    s_prefix = 0;
    s_remaining = n;
    s_m = 0;
  }
  __syncthreads();
  double qn = 0.0;
  for (int w = 0; w < kThreads / 64; ++w) qn += s_red[w];
  qn = sqrt(qn);

  // 1. radix select of the n-th largest key, 8 bits per pass; the digit of
  // each pass is found by a block-wide inclusive scan over the 256 bins taken
  // from the highest digit down (thread t holds digit 255 - t).
  for (int shift = 24; shift >= 0; shift -= 8) {
    hist[t] = 0;  // kThreads == 256 bins
    __syncthreads();
    const uint32_t hi_mask = shift == 24 ? 0u : (0xffffffffu << (shift + 8));
    const uint32_t prefix = s_prefix;
    const int rem = s_remaining;
    for (int c = t; c < nlist; c += kThreads) {
      const uint32_t k = keys[c];
      if ((k & hi_mask) == prefix) atomicAdd(&hist[(k >> shift) & 255], 1);
    }
    __syncthreads();
    const int v = hist[255 - t];
    int incl = v;
    for (int o = 1; o < 64; o <<= 1) {
      const int u = __shfl_up(incl, o);
      if ((t & 63) >= o) incl += u;
    }
    if ((t & 63) == 63) s_wsum[t >> 6] = incl;
    __syncthreads();
    for (int w = 0; w < (t >> 6); ++w) incl += s_wsum[w];
    if (incl >= rem && incl - v < rem) {
      s_prefix = prefix | ((uint32_t)(255 - t) << shift);
      s_remaining = rem - (incl - v);
    }
    __syncthreads();
  }
  const float vth = key2f(s_prefix);
  const double delta = 2.0 * (double)(d + 2) * 5.9604644775390625e-08 * qn * cmax + 1e-30;
  const double gap = 2.0 * delta;
  const double lo = (double)vth - gap;

  // 2. gather candidates
  for (int c = t; c < nlist; c += kThreads) {
    const float v = key2f(keys[c]);
    if ((double)v >= lo) {
      const int slot = atomicAdd(&s_m, 1);
      if (slot < cap) ck[slot] = ((unsigned long long)(~keys[c]) << 32) | (unsigned)c;
    }
  }
  __syncthreads();
  const int m_all = s_m;
  if (m_all > cap && t == 0) atomicExch(&rc->rank_error, 1);
  const int m = m_all < cap ? m_all : cap;
  int mp = 1;
  while (mp < m) mp <<= 1;
  for (int i = m + t; i < mp; i += kThreads) ck[i] = ~0ull;
  __syncthreads();

  // 3a. bitonic sort by (s32 desc, c asc) == key ascending
  for (int kk = 2; kk <= mp; kk <<= 1) {
    for (int j = kk >> 1; j > 0; j >>= 1) {
      for (int i = t; i < mp; i += kThreads) {
        const int ij = i ^ j;
        if (ij > i) {
          const unsigned long long a = ck[i], b = ck[ij];
          const bool up = (i & kk) == 0;
          if ((a > b) == up) {
            ck[i] = b;
            ck[ij] = a;
          }
        }
      }
      __syncthreads();
    }
  }

  // 3b. runs of near-ties, fp64 scores of their members
  for (int i = t; i < m; i += kThreads) {
    bool l = false;
    if (i + 1 < m) {
      const double a = (double)key2f(~(uint32_t)(ck[i] >> 32));
      const double b = (double)key2f(~(uint32_t)(ck[i + 1] >> 32));
      l = (a - b) <= gap;
    }
    link[i] = l ? 1 : 0;
  }
  __syncthreads();
  for (int i = t; i < m; i += kThreads) {
    const bool member = link[i] || (i > 0 && link[i - 1]);
    if (member) cs[i] = dot_fp64<DT>(queries, qg, centroids, (int)(ck[i] & 0xffffffffu), d);
  }
  __syncthreads();
  // 3c. insertion sort of every run by (s64 desc, c asc)
  for (int i = t; i < m; i += kThreads) {
    if (link[i] && (i == 0 || !link[i - 1])) {
      int e = i;
      while (link[e]) ++e;  // run is [i, e]
      for (int a = i + 1; a <= e; ++a) {
        const unsigned long long kv = ck[a];
        const double sv = cs[a];
        const unsigned cv = (unsigned)(kv & 0xffffffffu);
        int b = a - 1;
        while (b >= i) {
          const unsigned cb = (unsigned)(ck[b] & 0xffffffffu);
          const bool before = (sv > cs[b]) || (sv == cs[b] && cv < cb);
          if (!before) break;
          ck[b + 1] = ck[b];
          cs[b + 1] = cs[b];
          --b;
        }
        ck[b + 1] = kv;
        cs[b + 1] = sv;
      }
    }
  }
  __syncthreads();
  // 4. the first n
  for (int r = t; r < n; r += kThreads) P[ql * n + r] = (int32_t)(ck[r] & 0xffffffffu);
}

}  // namespace

size_t rank_select_lds(int32_t nlist, int32_t cap) {
  int capp = 1;
  while (capp < cap) capp <<= 1;
  return (size_t)((nlist * 4 + 15) & ~15) + (size_t)capp * 8 + (size_t)cap * 8 + (size_t)cap;
}

hipError_t launch_rank_select(int dtype, const void* queries, int64_t q0, int32_t nqc,
                              const void* centroids, int32_t nlist, int32_t d, const float* scores,
                              int32_t n, double cmax, int32_t* P, RoundCounters* rc,
                              hipStream_t s) {
  if (nqc <= 0) return hipSuccess;
  const int32_t cap = nlist < kMaxCand ? nlist : kMaxCand;
  const size_t lds = rank_select_lds(nlist, cap);
  static const hipError_t a32 = hipFuncSetAttribute(
      (const void*)rank_select_kernel<SIEVE_F32>, hipFuncAttributeMaxDynamicSharedMemorySize,
      150 * 1024);
  static const hipError_t a16 = hipFuncSetAttribute(
      (const void*)rank_select_kernel<SIEVE_F16>, hipFuncAttributeMaxDynamicSharedMemorySize,
      150 * 1024);
  if (a32 != hipSuccess) return a32;
  if (a16 != hipSuccess) return a16;
  if (lds > 150 * 1024) return hipErrorInvalidValue;
  if (dtype == SIEVE_F32)
    hipLaunchKernelGGL(rank_select_kernel<SIEVE_F32>, dim3(nqc), dim3(kThreads), lds, s, queries,
                       q0, centroids, nlist, d, scores, n, cap, cmax, P, rc);
  else
    hipLaunchKernelGGL(rank_select_kernel<SIEVE_F16>, dim3(nqc), dim3(kThreads), lds, s, queries,
                       q0, centroids, nlist, d, scores, n, cap, cmax, P, rc);
  return hipGetLastError();
}

}  // namespace sieve
