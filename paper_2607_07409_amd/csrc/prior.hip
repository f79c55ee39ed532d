// Unigram log-prior estimation (App. A, prior estimation): the counts c(v) of a token
// stream, then the add-lambda smoothed log-probabilities
//   b0(v) = log((c(v) + lambda) / (N + lambda V)),  N = number of counted tokens.
// Counting uses 64-bit device atomics (tokens outside [0, V) are skipped); the logarithm is
// taken in float64 and rounded once to float32.
#include "dels_internal.hpp"

namespace dls {

namespace {

constexpr int kPT = 256;

// zero fill (a kernel rather than a memset, so that the call can be captured in a graph)
__global__ __launch_bounds__(kPT) void k_zero_u64(uint64_t* __restrict__ p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * kPT + threadIdx.x; i < n; i += (int64_t)gridDim.x * kPT) p[i] = 0ull;
}

__global__ __launch_bounds__(kPT) void k_count(const int32_t* __restrict__ tokens, int64_t n, int V,
                                               uint64_t* __restrict__ counts) {
  __shared__ uint32_t s_valid;
  if (threadIdx.x == 0) s_valid = 0;
  __syncthreads();
  uint32_t valid = 0;
  for (int64_t i = (int64_t)blockIdx.x * kPT + threadIdx.x; i < n; i += (int64_t)gridDim.x * kPT) {
    const int t = tokens[i];
    if ((unsigned)t < (unsigned)V) {
      atomicAdd((unsigned long long*)&counts[t], 1ull);
      ++valid;
    }
  }
  atomicAdd(&s_valid, valid);
  __syncthreads();
  if (threadIdx.x == 0 && s_valid) atomicAdd((unsigned long long*)&counts[V], (unsigned long long)s_valid);
}

__global__ __launch_bounds__(kPT) void k_log_prior(const uint64_t* __restrict__ counts, int V, double lambda,
                                                   float* __restrict__ out) {
  const int v = blockIdx.x * kPT + threadIdx.x;
  if (v >= V) return;
  const double denom = (double)counts[V] + lambda * (double)V;
  out[v] = (float)log(((double)counts[v] + lambda) / denom);
}

}  // namespace

hipError_t launch_unigram_prior(const int32_t* tokens, int64_t n, int32_t V, float smoothing, uint64_t* counts,
                                float* out, hipStream_t st) {
  k_zero_u64<<<(unsigned)std::min<int64_t>((V + 1 + kPT - 1) / kPT, 1024), kPT, 0, st>>>(counts, (int64_t)V + 1);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (n > 0) {
    k_count<<<(unsigned)std::min<int64_t>((n + kPT - 1) / kPT, 4096), kPT, 0, st>>>(tokens, n, V, counts);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  k_log_prior<<<(unsigned)((V + kPT - 1) / kPT), kPT, 0, st>>>(counts, V, (double)smoothing, out);
  return hipGetLastError();
}

}  // namespace dls
