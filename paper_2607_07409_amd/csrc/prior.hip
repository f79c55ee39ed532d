// Unigram log-prior estimation (App. A, prior estimation): the counts c(v) of a token
// stream, then the add-lambda smoothed log-probabilities
//   b0(v) = log((c(v) + lambda) / (N + lambda V)),  N = number of counted tokens.
// Counting runs through per-workgroup LDS histograms of vocabulary slices and one 64-bit device
// atomic per nonzero counter (up to 323,584 ids), else through per-workgroup LDS caches of the
// frequent ids and device atomics for the rest; tokens outside [0, V) are skipped.  The logarithm
// is taken in float64 and rounded once to float32.
#include "dels_internal.hpp"

namespace dls {

namespace {

constexpr int kPT = 256;

// zero fill (a kernel rather than a memset, so that the call can be captured in a graph)
__global__ __launch_bounds__(kPT) void k_zero_u64(uint64_t* __restrict__ p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * kPT + threadIdx.x; i < n; i += (int64_t)gridDim.x * kPT) p[i] = 0ull;
}

// Counting: the vocabulary is cut into slices that fit one workgroup's LDS as 32-bit counters,
// and the stream into chunks; workgroup (chunk g, slice s) counts the tokens of slice s in chunk
// g with LDS atomics and adds each nonzero counter to the device count once at the end.  No
// token costs a device atomic (real token streams are Zipf-like: a hashed cache of the frequent
// ids still sent the long tail of rare ids to device atomics, one per token).  Each slice reads
// the whole stream, but the workgroups of one chunk are dispatched to the same XCD (the chunk
// count is a multiple of the XCD count, and workgroup ids go round the XCDs) and run together,
// so most of those reads hit in its L2.  A chunk holds at most 2^31 tokens, so no counter overflows.
constexpr int kCT = 1024;                 // threads per counting workgroup
constexpr int kSlice = 40448;             // ids per slice: 158 KiB of 32-bit counters
constexpr int64_t kMaxPerGroup = (int64_t)1 << 31;
constexpr int kTargetGroups = 256;        // about one counting workgroup per CU
constexpr int kMaxSlices = 8;             // beyond that the stream would be read too often

__global__ __launch_bounds__(kCT) void k_count_sliced(const int32_t* __restrict__ tokens, int64_t n, int V,
                                                      int slice, uint64_t* __restrict__ counts) {
  __shared__ uint32_t s_hist[kSlice];
  __shared__ uint32_t s_valid;
  const int v0 = blockIdx.y * slice;
  const int nv = max(0, min(slice, V - v0));
  for (int i = threadIdx.x; i < nv; i += kCT) s_hist[i] = 0u;
  if (threadIdx.x == 0) s_valid = 0u;
  __syncthreads();
  // this workgroup's contiguous chunk of the stream
  const int64_t per = (n + gridDim.x - 1) / gridDim.x;
  const int64_t lo = (int64_t)blockIdx.x * per;
  const int64_t hi = lo + per < n ? lo + per : n;
  uint32_t valid = 0;
  int64_t i = lo + threadIdx.x;
  // eight independent loads in flight per thread; ids are compared as unsigned offsets from
  // the slice start, so negative ids and ids past V fall outside every slice
  for (; i + 7 * kCT < hi; i += 8 * kCT) {
    int t[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) t[k] = tokens[i + k * kCT];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const uint32_t u = (uint32_t)t[k] - (uint32_t)v0;
      if (u < (uint32_t)nv) atomicAdd(&s_hist[u], 1u);
      valid += (uint32_t)t[k] < (uint32_t)V;
    }
  }
  for (; i < hi; i += kCT) {
    const int t = tokens[i];
    const uint32_t u = (uint32_t)t - (uint32_t)v0;
    if (u < (uint32_t)nv) atomicAdd(&s_hist[u], 1u);
    valid += (uint32_t)t < (uint32_t)V;
  }
  if (blockIdx.y == 0) atomicAdd(&s_valid, valid);
  __syncthreads();
  for (int j = threadIdx.x; j < nv; j += kCT) {
    const uint32_t c = s_hist[j];
    if (c) atomicAdd((unsigned long long*)&counts[v0 + j], (unsigned long long)c);
  }
  if (blockIdx.y == 0 && threadIdx.x == 0 && s_valid) atomicAdd((unsigned long long*)&counts[V], (unsigned long long)s_valid);
}

// Counting over vocabularies too large for a few slices: each workgroup keeps a direct-mapped cache of (token, count) pairs in LDS and
// flushes it with one device atomic per occupied slot at the end.  A token probes two slots
// (a multiplicative hash and its neighbour): a slot holding the token is incremented, an empty
// one is claimed, and a token finding both taken by others falls back to a device atomic.
// Frequent tokens claim their slots early, so they are counted in LDS (real token streams are
// Zipf-like: most of the mass sits on a few thousand ids, whose device counters would
// otherwise serialise every increment).  A slot is (token + 1) << 32 | count; a workgroup
// counts at most 2^31 tokens, so the count never carries into the token field.
constexpr int kSlotBits = 14;
constexpr int kSlots = 1 << kSlotBits;  // 128 KiB of LDS

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

__global__ __launch_bounds__(kCT) void k_count_cached(const int32_t* __restrict__ tokens, int64_t n, int V,
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
    // slices of at most kSlice ids, as even as possible; about one workgroup per CU over all
    // slices (each holds 158 KiB of LDS), more chunks when one would exceed 2^31 tokens, fewer
    // for short streams.  Vocabularies of more than kMaxSlices slices use the cached counter.
    const int slices = (V + kSlice - 1) / kSlice;
    if (slices <= kMaxSlices) {
      const int slice = (V + slices - 1) / slices;
      int64_t groups = std::min<int64_t>((n + 8 * kCT - 1) / (8 * kCT), kTargetGroups / slices);
      if (groups >= 8) groups &= ~(int64_t)7;   // the slices of a chunk on one XCD
      groups = std::max<int64_t>(groups, (n + kMaxPerGroup - 1) / kMaxPerGroup);
      k_count_sliced<<<dim3((unsigned)groups, (unsigned)slices), kCT, 0, st>>>(tokens, n, V, slice, counts);
    } else {
      // about one workgroup per CU (each holds 128 KiB of LDS), more when a chunk would exceed
      // 2^31 tokens, fewer for short streams
      int64_t groups = std::min<int64_t>((n + 4 * kCT - 1) / (4 * kCT), kTargetGroups);
      groups = std::max<int64_t>(groups, (n + kMaxPerGroup - 1) / kMaxPerGroup);
      k_count_cached<<<(unsigned)groups, kCT, 0, st>>>(tokens, n, V, counts);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  k_log_prior<<<(unsigned)((V + kPT - 1) / kPT), kPT, 0, st>>>(counts, V, (double)smoothing, out);
  return hipGetLastError();
}

}  // namespace dls
