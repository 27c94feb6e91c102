// rank.hip -- per-query centroid order P_i (Sec. 4.1), exact in fp64, from
// materialised fp32 screen scores (scan.hip writes them).  See rank_common.h
// for the bound delta that makes the order exact.  Steps:
//   1. the n-th largest fp32 score v is found by an 8-bit radix select;
//   2. every centroid of the true fp64 top-n has s32 >= v - 2 delta, so the
//      candidates are all c with s32[c] >= v - 2 delta;
//   3. sorted by (s32 desc, c asc), candidates whose successive fp32 gaps are
//      all <= 2 delta form runs; a gap > 2 delta orders two centroids the
//      same way in fp64, so only members of multi-element runs need fp64
//      scores, which are then ordered by (s64 desc, c asc) inside each run;
//   4. the first n candidates are P_i.
// The result equals sorting all centroids by (fp64 score desc, index asc).
#include "rank_common.h"

namespace sieve {
namespace {

// Bytes of the region holding one query's fp32 scores.
__host__ __device__ inline int keys_bytes(int nlist) { return (nlist * 4 + 15) & ~15; }

// Candidate counts up to this use the counting sort (O(m^2 / NT) compares,
// no barriers); larger ones a bitonic network.
constexpr int kRankSortMax = 1024;

// One query per block of NT threads.
template <int DT, int NT>
__global__ __launch_bounds__(NT) void rank_select_kernel(
    const void* __restrict__ queries, int64_t q0, const void* __restrict__ centroids,
    int32_t nlist, int32_t d, const float* __restrict__ scores, int32_t n, int32_t cap,
    double cmax, int32_t* __restrict__ P, int64_t ldp, RoundCounters* rc) {
  constexpr int kWaves = NT / 64;
  constexpr int kBins = 256;
  constexpr int kBPT = kBins / NT > 0 ? kBins / NT : 1;  // bins per thread
  extern __shared__ uint8_t smem[];
  float* sv = (float*)smem;  // [nlist] fp32 scores
  unsigned long long* ck = (unsigned long long*)(smem + keys_bytes(nlist));  // [capp]
  __shared__ int hist[kBins];
  __shared__ float s_min[kWaves], s_max[kWaves];
  __shared__ double s_red[kWaves];
  __shared__ int s_wsum[kWaves];
  __shared__ int s_bin, s_m;

  int capp = 1;
  while (capp < 2 * cap) capp <<= 1;
  double* cs = (double*)(ck + capp);     // [cap] fp64 scores of run members
  uint8_t* link = (uint8_t*)(cs + cap);  // [cap]

  const int t = threadIdx.x;
  const int64_t ql = blockIdx.x;
  const int64_t qg = q0 + ql;
  const float* row = scores + ql * nlist;

  // scores, their range, |q| in fp64
  float lo_v = INFINITY, hi_v = -INFINITY;
  for (int c0 = t; c0 < nlist; c0 += 8 * NT) {
    float v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int c = c0 + k * NT;
      v[k] = row[c < nlist ? c : nlist - 1];  // clamped: the loads issue together
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int c = c0 + k * NT;
      if (c < nlist) {
        sv[c] = v[k];
        lo_v = fminf(lo_v, v[k]);
        hi_v = fmaxf(hi_v, v[k]);
      }
    }
  }
  double ss = 0.0;
  for (int i = t; i < d; i += NT) {
    const double v = load_elem<DT>(queries, qg * d + i);
    ss += v * v;
  }
  for (int o = 32; o > 0; o >>= 1) {
    ss += __shfl_xor(ss, o);
    lo_v = fminf(lo_v, __shfl_xor(lo_v, o));
    hi_v = fmaxf(hi_v, __shfl_xor(hi_v, o));
  }
  if ((t & 63) == 0) {
    s_red[t >> 6] = ss;
    s_min[t >> 6] = lo_v;
    s_max[t >> 6] = hi_v;
  }
  for (int b = t; b < kBins; b += NT) hist[b] = 0;
  if (t == 0) s_m = 0;
  __syncthreads();
  double qn = 0.0;
  float smin = s_min[0], smax = s_max[0];
  for (int w = 0; w < kWaves; ++w) {
    qn += s_red[w];
    smin = fminf(smin, s_min[w]);
    smax = fmaxf(smax, s_max[w]);
  }
  qn = sqrt(qn);
  const double delta = 2.0 * (double)(d + 2) * 5.9604644775390625e-08 * qn * cmax + 1e-30;
  const double gap = 2.0 * delta;

  // 1. one histogram of the scores over [smin, smax] in 256 equal bins (bin
  // index non-decreasing in the score); the bin holding the n-th largest
  // score is found by a block-wide scan from the top bin down
  const float span = smax - smin;
  const float scale = span > 0.f ? (float)kBins / span : 0.f;
  auto bin_of = [&](float v) {
    int b = (int)((v - smin) * scale);
    return b < 0 ? 0 : (b > kBins - 1 ? kBins - 1 : b);
  };
  for (int c = t; c < nlist; c += NT) atomicAdd(&hist[bin_of(sv[c])], 1);
  __syncthreads();
  {
    int v[kBPT];
    int own = 0;
#pragma unroll
    for (int e = 0; e < kBPT; ++e) {
      const int b = kBins - 1 - (t * kBPT + e);
      v[e] = (t * kBPT + e) < kBins ? hist[b] : 0;
      own += v[e];
    }
    int incl = own;
    for (int o = 1; o < 64; o <<= 1) {
      const int u = __shfl_up(incl, o);
      if ((t & 63) >= o) incl += u;
    }
    if ((t & 63) == 63) s_wsum[t >> 6] = incl;
    __syncthreads();
    for (int w = 0; w < (t >> 6); ++w) incl += s_wsum[w];
    int before = incl - own;
#pragma unroll
    for (int e = 0; e < kBPT; ++e) {
      if (before < n && before + v[e] >= n) s_bin = kBins - 1 - (t * kBPT + e);
      before += v[e];
    }
  }
  __syncthreads();

  // 2. candidates: every score in the boundary bin or above, and any score
  // within 2 delta below it; the n-th largest fp32 score v lies in the bin,
  // so this contains { c : s32[c] >= v - 2 delta }, which holds the fp64
  // top-n.  Keys sort as (s32 desc, c asc).
  const int bstar = s_bin;
  // lower edge of the boundary bin, less the fp32 rounding of bin_of and of
  // the edge itself (a few ulps of the score range; a wider margin only adds
  // candidates)
  const double edge = (double)(smin + (float)bstar / (scale > 0.f ? scale : 1.f));
  const double lo = edge - gap - 1e-6 * ((double)fabsf(smin) + (double)fabsf(smax) + 1e-30);
  for (int c = t; c < nlist; c += NT) {
    const float v = sv[c];
    const bool take = bin_of(v) >= bstar || (double)v >= lo;
    if (take) {
      const int slot = atomicAdd(&s_m, 1);
      if (slot < cap) ck[slot] = ((unsigned long long)(~f2key(v)) << 32) | (unsigned)c;
    }
  }
  __syncthreads();
  const int m = s_m;
  if (m > cap || m < n) {
    // too many near-ties for this launch's buffer (m > cap), or a candidate
    // set that cannot be right (m < n): the caller discards this search and
    // re-ranks with the wide buffer.  The row still gets valid list ids so
    // that every kernel that runs before the check stays in bounds.
    if (t == 0) atomicExch(&rc->rank_error, 1);
    for (int r = t; r < n; r += NT) P[ql * ldp + r] = r;
    return;
  }

  // 3a. sort by key ascending == (s32 desc, c asc)
  if (m <= kRankSortMax) {
    // rank by counting: keys are distinct (the centroid index is in the low
    // bits), so a key's position is the number of smaller keys
    unsigned long long* out = ck + cap;
    for (int i = t; i < m; i += NT) {
      const unsigned long long ki = ck[i];
      int pos = 0;
#pragma unroll 8
      for (int j = 0; j < m; ++j) pos += ck[j] < ki ? 1 : 0;
      out[pos] = ki;
    }
    __syncthreads();
    for (int i = t; i < m; i += NT) ck[i] = out[i];
    __syncthreads();
  } else {
    int mp = 1;
    while (mp < m) mp <<= 1;
    for (int i = m + t; i < mp; i += NT) ck[i] = ~0ull;
    __syncthreads();
    for (int kk = 2; kk <= mp; kk <<= 1) {
      for (int j = kk >> 1; j > 0; j >>= 1) {
        for (int i = t; i < mp; i += NT) {
          const int ij = i ^ j;
          if (ij > i) {
            const unsigned long long x = ck[i], y = ck[ij];
            const bool up = (i & kk) == 0;
            if ((x > y) == up) {
              ck[i] = y;
              ck[ij] = x;
            }
          }
        }
        __syncthreads();
      }
    }
  }

  // 3b. runs of near-ties (successive fp32 gaps <= 2 delta)
  for (int i = t; i < m; i += NT) {
    bool l = false;
    if (i + 1 < m) {
      const double x = (double)key2f(~(uint32_t)(ck[i] >> 32));
      const double y = (double)key2f(~(uint32_t)(ck[i + 1] >> 32));
      l = (x - y) <= gap;
    }
    link[i] = l ? 1 : 0;
  }
  __syncthreads();
  // 3c. fp64 scores of run members, one wave per member
  refine_members<DT>(ck, cs, link, m, queries, qg, centroids, d, t >> 6, NT / 64);
  __syncthreads();
  // 3d. order inside each run (exact sequential sums where tier 1 is too close)
  {
    const double gap64 =
        2.0 * 2.0 * (double)(d + (d + 63) / 64 + 6) * 1.1102230246251565e-16 * qn * cmax + 1e-300;
    order_runs<DT>(ck, cs, link, m, queries, qg, centroids, d, gap64, t, NT);
  }
  __syncthreads();
  // 4. the first n
  for (int r = t; r < n; r += NT) P[ql * ldp + r] = (int32_t)(ck[r] & 0xffffffffu);
}

// One query per block of 256 threads, its screen scores held in registers
// (KPT per thread, nlist <= 256 * KPT): long prefixes over large centroid
// sets, where one wave per query would hold too many keys.
//   1. the n-th largest key is found bit by bit (32 steps; each step counts
//      keys >= the candidate prefix with ballot popcounts per wave and one
//      LDS exchange between the four waves);
//   2. candidates (s32 >= v - 2 delta) are compacted with ballots into LDS;
//   3. they are sorted by counting, near-tie runs are re-scored in fp64
//      (waves of the block share the members), and the first n are written.
// More than cap candidates (or fewer than n) sets rank_error.
template <int DT, int KPT>
__global__ __launch_bounds__(256) void rank_select_reg_kernel(
    const void* __restrict__ queries, int64_t q0, const void* __restrict__ centroids,
    int32_t nlist, int32_t d, const float* __restrict__ scores, int32_t n, int32_t cap,
    double cmax, int32_t* __restrict__ P, int64_t ldp, RoundCounters* rc) {
  extern __shared__ uint8_t smem[];
  unsigned long long* ck = (unsigned long long*)smem;  // [cap]
  unsigned long long* out = ck + cap;                  // [cap]
  double* cs = (double*)(out + cap);                   // [cap]
  uint8_t* link = (uint8_t*)(cs + cap);                // [cap]
  __shared__ int s_cnt[2][4];
  __shared__ double s_ss[4];
  __shared__ int s_m;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int64_t ql = blockIdx.x;
  const int64_t qg = q0 + ql;
  const float* row = scores + ql * nlist;

  uint32_t key[KPT];
#pragma unroll
  for (int j = 0; j < KPT; ++j) {
    const int c = t + 256 * j;
    const float v = row[c < nlist ? c : nlist - 1];  // clamped: the loads issue together
    key[j] = c < nlist ? f2key(v) : 0u;              // 0 sorts below every score
  }
  double ss = 0.0;
  for (int i = t; i < d; i += 256) {
    const double v = load_elem<DT>(queries, qg * d + i);
    ss += v * v;
  }
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
  if (lane == 0) s_ss[wave] = ss;
  if (t == 0) s_m = 0;
  __syncthreads();
  const double qn = sqrt(s_ss[0] + s_ss[1] + s_ss[2] + s_ss[3]);
  const double delta = 2.0 * (double)(d + 2) * 5.9604644775390625e-08 * qn * cmax + 1e-30;
  const double gap = 2.0 * delta;

  // 1. exact n-th largest key (the two count slots alternate, one barrier a step)
  uint32_t prefix = 0;
  for (int bit = 31; bit >= 0; --bit) {
    const uint32_t cand = prefix | (1u << bit);
    int cnt = 0;  // this lane's keys >= cand, then the wave's sum
#pragma unroll
    for (int j = 0; j < KPT; ++j) cnt += key[j] >= cand ? 1 : 0;
    for (int o = 32; o > 0; o >>= 1) cnt += __shfl_xor(cnt, o);
    if (lane == 0) s_cnt[bit & 1][wave] = cnt;
    __syncthreads();
    const int total = s_cnt[bit & 1][0] + s_cnt[bit & 1][1] + s_cnt[bit & 1][2] +
                      s_cnt[bit & 1][3];
    if (total >= n) prefix = cand;
  }
  const double lo = (double)key2f(prefix) - gap;

  // 2. candidates, compacted with ballots (one LDS atomic per wave and slot)
#pragma unroll
  for (int j = 0; j < KPT; ++j) {
    const int c = t + 256 * j;
    const bool take = c < nlist && (double)key2f(key[j]) >= lo;
    const unsigned long long mask = __ballot(take);
    if (mask == 0) continue;
    int base = 0;
    if (lane == __ffsll((long long)mask) - 1) base = atomicAdd(&s_m, __popcll(mask));
    base = __builtin_amdgcn_readlane(base, __ffsll((long long)mask) - 1);
    const int pos = base + __popcll(mask & ((1ull << lane) - 1ull));
    if (take && pos < cap) ck[pos] = ((unsigned long long)(~key[j]) << 32) | (unsigned)c;
  }
  __syncthreads();
  const int m = s_m;
  if (m > cap || m < n) {
    if (t == 0) atomicExch(&rc->rank_error, 1);
    for (int r = t; r < n; r += 256) P[ql * ldp + r] = r;  // valid placeholder
    return;
  }
  // 3. exact sort by counting (keys are distinct), runs, fp64 refinement
  for (int i = t; i < m; i += 256) {
    const unsigned long long ki = ck[i];
    int pos = 0;
#pragma unroll 8
    for (int j = 0; j < m; ++j) pos += ck[j] < ki ? 1 : 0;
    out[pos] = ki;
  }
  __syncthreads();
  for (int i = t; i < m; i += 256) {
    bool l = false;
    if (i + 1 < m) {
      const double x = (double)key2f(~(uint32_t)(out[i] >> 32));
      const double y = (double)key2f(~(uint32_t)(out[i + 1] >> 32));
      l = (x - y) <= gap;
    }
    link[i] = l ? 1 : 0;
  }
  __syncthreads();
  refine_members<DT>(out, cs, link, m, queries, qg, centroids, d, wave, 4);
  __syncthreads();
  {
    const double gap64 =
        2.0 * 2.0 * (double)(d + (d + 63) / 64 + 6) * 1.1102230246251565e-16 * qn * cmax + 1e-300;
    order_runs<DT>(out, cs, link, m, queries, qg, centroids, d, gap64, t, 256);
  }
  __syncthreads();
  for (int r = t; r < n; r += 256) P[ql * ldp + r] = (int32_t)(out[r] & 0xffffffffu);
}

// Boundary candidates per lane in the wave kernel (capw <= 64 * this).
constexpr int kKeysPerLane = 8;

// One query per wave, four per block; KPL = keys per lane (nlist <= 64*KPL).
// 1. the scores of the query are held in registers, KPL per lane;
// 2. the n-th largest key (the order-preserving integer image of the fp32
//    score) is found bit by bit from the top: a bit is kept when at least n
//    keys are >= the prefix with that bit set (32 counting steps, each
//    register compares and ballot popcounts);
// 3. candidates (score >= v - 2 delta) are compacted with ballots;
// 4. they are sorted exactly by counting; near-tie runs get fp64 scores and
//    an insertion sort, as in the block kernel.
// A query with more than capw candidates sets rank_error (the caller then
// re-ranks with the block kernel) and writes a valid placeholder row.
template <int DT, int KPL>
__global__ __launch_bounds__(256) void rank_select_wave_kernel(
    const void* __restrict__ queries, int64_t q0, int32_t nqc, const void* __restrict__ centroids,
    int32_t nlist, int32_t d, const float* __restrict__ scores, int32_t n, int32_t capw,
    double cmax, int32_t* __restrict__ P, int64_t ldp, RoundCounters* rc) {
  extern __shared__ uint8_t smem[];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t ql = (int64_t)blockIdx.x * 4 + wave;
  if (ql >= nqc) return;  // whole wave; no block barrier follows
  uint8_t* region = smem + (size_t)wave * wave_region_bytes(capw);
  unsigned long long* ck = (unsigned long long*)region;  // [capw]
  unsigned long long* out = ck + capw;                   // [capw]
  double* cs = (double*)(out + capw);                    // [capw]
  uint8_t* link = (uint8_t*)(cs + capw);                 // [capw]
  const int64_t qg = q0 + ql;
  const float* row = scores + ql * nlist;

  // all loads are issued before any is used: clamped addresses, no branches
  float raw[KPL];
#pragma unroll
  for (int j = 0; j < KPL; ++j) {
    const int c = lane + 64 * j;
    raw[j] = row[c < nlist ? c : nlist - 1];
  }
  uint32_t key[KPL];
#pragma unroll
  for (int j = 0; j < KPL; ++j)
    key[j] = (lane + 64 * j) < nlist ? f2key(raw[j]) : 0u;  // 0 sorts below every score
  double ss = 0.0;
  for (int i = lane; i < d; i += 64) {
    const double v = load_elem<DT>(queries, qg * d + i);
    ss += v * v;
  }
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
  const double qn = sqrt(ss);
  const double delta = 2.0 * (double)(d + 2) * 5.9604644775390625e-08 * qn * cmax + 1e-30;
  const double gap = 2.0 * delta;

  // 2. exact n-th largest key; each count is a sum of ballot popcounts, so
  // it stays in scalar registers (no cross-lane shuffles)
  uint32_t prefix = 0;
  for (int bit = 31; bit >= 0; --bit) {
    const uint32_t cand = prefix | (1u << bit);
    int cnt = 0;
#pragma unroll
    for (int j = 0; j < KPL; ++j) cnt += __popcll(__ballot(key[j] >= cand));
    if (cnt >= n) prefix = cand;
  }
  const double lo = (double)key2f(prefix) - gap;

  // 3. candidates, compacted with ballots
  int m = 0;
#pragma unroll
  for (int j = 0; j < KPL; ++j) {
    const int c = lane + 64 * j;
    const bool take = c < nlist && (double)key2f(key[j]) >= lo;
    const unsigned long long mask = __ballot(take);
    const int pos = m + __popcll(mask & ((1ull << lane) - 1ull));
    if (take && pos < capw) ck[pos] = ((unsigned long long)(~key[j]) << 32) | (unsigned)c;
    m += __popcll(mask);
  }
  if (m > capw || m < n) {
    if (lane == 0) atomicExch(&rc->rank_error, 1);
    for (int r = lane; r < n; r += 64) P[ql * ldp + r] = r;
    return;
  }
  wave_sync();

  finish_candidates_wave<DT>(ck, out, cs, link, m, n, gap, queries, qg, centroids, d, qn, cmax,
                             P + ql * ldp);
}

}  // namespace

size_t rank_select_lds(int32_t nlist, int32_t cap) {
  int capp = 1;
  while (capp < 2 * cap) capp <<= 1;
  return (size_t)keys_bytes(nlist) + (size_t)capp * 8 + (size_t)cap * 8 + (size_t)cap;
}

// `wide` (set after a launch reported more near-ties at a rank boundary than
// its buffer holds) sizes the candidate buffer for every centroid.
template <int DT, int KPL>
hipError_t launch_wave_t(const void* queries, int64_t q0, int32_t nqc, const void* centroids,
                         int32_t nlist, int32_t d, const float* scores, int32_t n, int32_t capw,
                         double cmax, int32_t* P, int64_t ldp, RoundCounters* rc,
                         hipStream_t s) {
  const size_t lds = (size_t)4 * wave_region_bytes(capw);
  static const hipError_t attr =
      hipFuncSetAttribute((const void*)rank_select_wave_kernel<DT, KPL>,
                          hipFuncAttributeMaxDynamicSharedMemorySize, 150 * 1024);
  if (attr != hipSuccess) return attr;
  if (lds > 150 * 1024) return hipErrorInvalidValue;
  hipLaunchKernelGGL((rank_select_wave_kernel<DT, KPL>), dim3((unsigned)((nqc + 3) / 4)),
                     dim3(256), lds, s, queries, q0, nqc, centroids, nlist, d, scores, n, capw,
                     cmax, P, ldp, rc);
  return hipGetLastError();
}

template <int DT>
hipError_t launch_wave(const void* queries, int64_t q0, int32_t nqc, const void* centroids,
                       int32_t nlist, int32_t d, const float* scores, int32_t n, int32_t capw,
                       double cmax, int32_t* P, int64_t ldp, RoundCounters* rc,
                       hipStream_t s) {
  if (nlist <= 256)
    return launch_wave_t<DT, 4>(queries, q0, nqc, centroids, nlist, d, scores, n, capw, cmax,
                                  P, ldp, rc, s);
  if (nlist <= 1024)
    return launch_wave_t<DT, 16>(queries, q0, nqc, centroids, nlist, d, scores, n, capw, cmax,
                                  P, ldp, rc, s);
  return launch_wave_t<DT, 64>(queries, q0, nqc, centroids, nlist, d, scores, n, capw, cmax,
                                 P, ldp, rc, s);
}

hipError_t launch_rank_select(int dtype, const void* queries, int64_t q0, int32_t nqc,
                              const void* centroids, int32_t nlist, int32_t d, const float* scores,
                              int32_t n, double cmax, int32_t* P, int64_t ldp, RoundCounters* rc,
                              bool wide, hipStream_t s) {
  if (nqc <= 0) return hipSuccess;
  // one wave per query while the boundary buffer stays small
  const int elem = dtype == SIEVE_F32 ? 4 : 2;
  int capw = n + 128 < nlist ? n + 128 : nlist;
  if (!wide && nlist <= 1024 && capw <= 64 * kKeysPerLane &&
      4 * wave_region_bytes(capw) <= 96 * 1024) {
    return dtype == SIEVE_F32
               ? launch_wave<SIEVE_F32>(queries, q0, nqc, centroids, nlist, d, scores, n, capw,
                                        cmax, P, ldp, rc, s)
               : launch_wave<SIEVE_F16>(queries, q0, nqc, centroids, nlist, d, scores, n, capw,
                                        cmax, P, ldp, rc, s);
  }
  // register-resident block kernel: large centroid sets, narrow buffer
  if (!wide && nlist > 1024 && nlist <= 256 * 64) {
    const int32_t capr = n + 512 < nlist ? n + 512 : nlist;
    const size_t ldsr = (size_t)capr * 25;
    if (ldsr <= 64 * 1024) {
      const int kpt = nlist <= 256 * 16 ? 16 : (nlist <= 256 * 32 ? 32 : 64);
#define SIEVE_REG(DT, K)                                                                       \
  hipLaunchKernelGGL((rank_select_reg_kernel<DT, K>), dim3(nqc), dim3(256), ldsr, s, queries, q0, \
                     centroids, nlist, d, scores, n, capr, cmax, P, ldp, rc)
      if (dtype == SIEVE_F32) {
        if (kpt == 16) SIEVE_REG(SIEVE_F32, 16);
        else if (kpt == 32) SIEVE_REG(SIEVE_F32, 32);
        else SIEVE_REG(SIEVE_F32, 64);
      } else {
        if (kpt == 16) SIEVE_REG(SIEVE_F16, 16);
        else if (kpt == 32) SIEVE_REG(SIEVE_F16, 32);
        else SIEVE_REG(SIEVE_F16, 64);
      }
#undef SIEVE_REG
      return hipGetLastError();
    }
  }
  // block kernel: narrow (n + 512 boundary candidates) or wide (every
  // centroid, up to kMaxCand)
  int32_t cap = nlist < kMaxCand ? nlist : kMaxCand;
  if (!wide && n + 512 < cap) cap = n + 512;
  while (cap > n && rank_select_lds(nlist, cap) > 150 * 1024) cap = (cap + n) / 2;
  const size_t lds = rank_select_lds(nlist, cap);
  if (lds > 150 * 1024) return hipErrorInvalidValue;
  if (dtype == SIEVE_F32)
    hipLaunchKernelGGL((rank_select_kernel<SIEVE_F32, 256>), dim3(nqc), dim3(256), lds, s,
                       queries, q0, centroids, nlist, d, scores, n, cap, cmax, P, ldp, rc);
  else
    hipLaunchKernelGGL((rank_select_kernel<SIEVE_F16, 256>), dim3(nqc), dim3(256), lds, s,
                       queries, q0, centroids, nlist, d, scores, n, cap, cmax, P, ldp, rc);
  return hipGetLastError();
}

}  // namespace sieve
