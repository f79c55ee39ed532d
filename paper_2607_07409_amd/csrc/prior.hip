// Unigram log-prior estimation (App. A, prior estimation): the counts c(v) of a token
// stream, then the add-lambda smoothed log-probabilities
//   b0(v) = log((c(v) + lambda) / (N + lambda V)),  N = number of counted tokens.
// Counting runs through per-workgroup LDS caches and 64-bit device atomics (tokens outside
// [0, V) are skipped); the logarithm is taken in float64 and rounded once to float32.
#include "dels_internal.hpp"

namespace dls {

namespace {

constexpr int kPT = 256;

// zero fill (a kernel rather than a memset, so that the call can be captured in a graph)
__global__ __launch_bounds__(kPT) void k_zero_u64(uint64_t* __restrict__ p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * kPT + threadIdx.x; i < n; i += (int64_t)gridDim.x * kPT) p[i] = 0ull;
}

// Counting: each workgroup keeps a direct-mapped cache of (token, count) pairs in LDS and
// flushes it with one device atomic per occupied slot at the end.  A token probes two slots
// (a multiplicative hash and its neighbour): a slot holding the token is incremented, an empty
// one is claimed, and a token finding both taken by others falls back to a device atomic.
// Frequent tokens claim their slots early, so they are counted in LDS (real token streams are
// Zipf-like: most of the mass sits on a few thousand ids, whose device counters would
// otherwise serialise every increment).  A slot is (token + 1) << 32 | count; a workgroup
// counts at most 2^31 tokens, so the count never carries into the token field.
constexpr int kCT = 1024;               // threads per counting workgroup
constexpr int kSlotBits = 14;
constexpr int kSlots = 1 << kSlotBits;  // 128 KiB of LDS
constexpr int64_t kMaxPerGroup = (int64_t)1 << 31;

__device__ __forceinline__ void count_token(unsigned long long* tab, int t, uint64_t* __restrict__ counts) {
  const uint64_t key = (uint64_t)(uint32_t)(t + 1) << 32;
  const uint32_t h = ((uint32_t)t * 2654435761u) >> (32 - kSlotBits);
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    unsigned long long* slot = tab + (h ^ (uint32_t)p);
    unsigned long long cur = *(volatile unsigned long long*)slot;
    if (cur == 0ull) cur = atomicCAS(slot, 0ull, (unsigned long long)(key | 1ull));
    if (cur == 0ull) return;                                   // claimed with a count of one
    if ((cur & 0xffffffff00000000ull) == key) {                // the token's own slot
      atomicAdd(slot, 1ull);
      return;
    }
  }
  atomicAdd((unsigned long long*)&counts[t], 1ull);
}

__global__ __launch_bounds__(kCT) void k_count(const int32_t* __restrict__ tokens, int64_t n, int V,
                                               uint64_t* __restrict__ counts) {
  __shared__ unsigned long long s_tab[kSlots];
  __shared__ uint32_t s_valid;
  for (int i = threadIdx.x; i < kSlots; i += kCT) s_tab[i] = 0ull;
  if (threadIdx.x == 0) s_valid = 0;
  __syncthreads();
  // this workgroup's contiguous chunk of the stream
  const int64_t per = (n + gridDim.x - 1) / gridDim.x;
  const int64_t lo = (int64_t)blockIdx.x * per;
  const int64_t hi = lo + per < n ? lo + per : n;
  uint32_t valid = 0;
  int64_t i = lo + threadIdx.x;
  // four independent loads in flight per thread
  for (; i + 3 * kCT < hi; i += 4 * kCT) {
    int t[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) t[k] = tokens[i + k * kCT];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if ((unsigned)t[k] < (unsigned)V) {
        count_token(s_tab, t[k], counts);
        ++valid;
      }
    }
  }
  for (; i < hi; i += kCT) {
    const int t = tokens[i];
    if ((unsigned)t < (unsigned)V) {
      count_token(s_tab, t, counts);
      ++valid;
    }
  }
  atomicAdd(&s_valid, valid);
  __syncthreads();
  for (int j = threadIdx.x; j < kSlots; j += kCT) {
    const unsigned long long e = s_tab[j];
    if (e) atomicAdd((unsigned long long*)&counts[(uint32_t)(e >> 32) - 1u], e & 0xffffffffull);
  }
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
    // about one workgroup per CU (each holds 128 KiB of LDS), more when a chunk would exceed
    // 2^31 tokens, fewer for short streams
    int64_t groups = std::min<int64_t>((n + 4 * kCT - 1) / (4 * kCT), 256);
    groups = std::max<int64_t>(groups, (n + kMaxPerGroup - 1) / kMaxPerGroup);
    k_count<<<(unsigned)groups, kCT, 0, st>>>(tokens, n, V, counts);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  k_log_prior<<<(unsigned)((V + kPT - 1) / kPT), kPT, 0, st>>>(counts, V, (double)smoothing, out);
  return hipGetLastError();
}

}  // namespace dls
