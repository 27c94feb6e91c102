// In-call window calibration (Appendix A, Algorithm 3).
//
// A fixed-probe search over the sampled queries leaves, per query, a bitmap
// of the ranks whose partition held a candidate (sim >= tau) and, per
// returned neighbour, the rank it was found at.  Lookahead execution always
// visits a prefix of the probe order, and a window W reaches rank f (0-based)
// exactly when no run of W empty probes closes before f.  The neighbour's
// required window is therefore 1 + the longest run of empty probes among
// ranks 0 .. f-1.  Counting neighbours by required window gives the
// histogram H; loss(W) = 1 - (H[1] + ... + H[W]) / Z, with Z the number of
// neighbours, and the chosen window is the smallest W < n with loss(W) < eps,
// else n (full probing).
#include <hip/hip_runtime.h>

#include "sieve_internal.h"

namespace sieve {
namespace {

constexpr int kThreads = 256;

__global__ void gather_i64_kernel(const int32_t* __restrict__ idx, int64_t n,
                                  const int64_t* __restrict__ src, int64_t* __restrict__ dst) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = src[idx[i]];
}

// One wave per sampled query, one lane per returned neighbour.  The LDS
// histogram (n + 1 bins) is flushed once per work-group.
__global__ __launch_bounds__(kThreads) void calib_replay_kernel(
    int64_t ns, int32_t n, int32_t k, const uint32_t* __restrict__ hitbits, int32_t words,
    const int32_t* __restrict__ frank, unsigned long long* __restrict__ hist,
    unsigned long long* __restrict__ z) {
  extern __shared__ unsigned int s_hist[];  // [n + 1]
  __shared__ unsigned int s_z;
  for (int i = threadIdx.x; i <= n; i += blockDim.x) s_hist[i] = 0;
  if (threadIdx.x == 0) s_z = 0;
  __syncthreads();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int waves = blockDim.x >> 6;
  for (int64_t q = (int64_t)blockIdx.x * waves + wave; q < ns; q += (int64_t)gridDim.x * waves) {
    const int f = lane < k ? frank[q * k + lane] : -1;
    if (f < 0 || f >= n) continue;  // padding: fewer than k neighbours
    const uint32_t* bits = hitbits + q * words;
    int run = 0, longest = 0;
    for (int r = 0; r < f; ++r) {
      const uint32_t b = (bits[r >> 5] >> (r & 31)) & 1u;
      run = b ? 0 : run + 1;
      longest = run > longest ? run : longest;
    }
    atomicAdd(&s_hist[longest + 1], 1u);  // longest <= f <= n - 1
    atomicAdd(&s_z, 1u);
  }
  __syncthreads();
  for (int i = threadIdx.x; i <= n; i += blockDim.x)
    if (s_hist[i]) atomicAdd(&hist[i], (unsigned long long)s_hist[i]);
  if (threadIdx.x == 0 && s_z) atomicAdd(z, (unsigned long long)s_z);
}

// Prefix sums of H in order; the loss is evaluated in double.
__global__ void calib_choose_kernel(int32_t n, float eps, const unsigned long long* __restrict__ hist,
                                    const unsigned long long* __restrict__ z,
                                    int32_t* __restrict__ w_out) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  const unsigned long long total = *z;
  if (total == 0) {
    *w_out = 0;  // no neighbour in the sample: the caller's fallback applies
    return;
  }
  unsigned long long retained = 0;
  for (int w = 1; w <= n - 1; ++w) {
    retained += hist[w];
    const double loss = 1.0 - (double)retained / (double)total;
    if (loss < (double)eps) {
      *w_out = w;
      return;
    }
  }
  *w_out = n;
}

}  // namespace

hipError_t launch_gather_i64(const int32_t* idx, int64_t n, const int64_t* src, int64_t* dst,
                             hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t b = (n + kThreads - 1) / kThreads;
  hipLaunchKernelGGL(gather_i64_kernel, dim3((unsigned)(b < 4096 ? b : 4096)), dim3(kThreads), 0,
                     s, idx, n, src, dst);
  return hipGetLastError();
}

hipError_t launch_calib_replay(int64_t ns, int32_t n, int32_t k, const uint32_t* hitbits,
                               int32_t words, const int32_t* frank, unsigned long long* hist,
                               unsigned long long* z, hipStream_t s) {
  if (ns <= 0) return hipSuccess;
  if (n < 1 || n > kMaxRanks || k < 1 || k > 64 || words * 32 < n) return hipErrorInvalidValue;
  const int64_t b = (ns + 3) / 4;
  const size_t lds = (size_t)(n + 1) * sizeof(unsigned int);
  hipLaunchKernelGGL(calib_replay_kernel, dim3((unsigned)(b < 1024 ? b : 1024)), dim3(kThreads),
                     lds, s, ns, n, k, hitbits, words, frank, hist, z);
  return hipGetLastError();
}

hipError_t launch_calib_choose(int32_t n, float eps, const unsigned long long* hist,
                               const unsigned long long* z, int32_t* w_out, hipStream_t s) {
  hipLaunchKernelGGL(calib_choose_kernel, dim3(1), dim3(64), 0, s, n, eps, hist, z, w_out);
  return hipGetLastError();
}

}  // namespace sieve
