// Uncertainty of rows of long logits, for the adaptive fusion that Sec. 7 proposes (local-head
// and prior weights adjusted by the entropy or confidence of the long-context logits).
//
// Per row of V logits x (finite or -inf) the kernel keeps, over the finite entries,
//   m = the largest value, s = sum exp(x - m), t = sum exp(x - m) (x - m),
// so that log-sum-exp = m + log s, max p = 1 / s and H(p) = log s - t / s (t <= 0, s >= 1).
// The chunks of an iteration are folded with one rescale to their maximum and one exponential
// per entry.
// A row is split into `parts` contiguous ranges, one workgroup each, when rows are too few
// to cover the chip; a second kernel then merges the per-range triples of each row in a fixed
// order.  The gate g = clamp((u - h_lo) / (h_hi - h_lo), 0, 1) of the chosen measure u is
// written beside the entropy and the maximum probability.
#include "dels_internal.hpp"
#include "stream_load.hpp"

namespace dls {

namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 2;
constexpr float kEntEmpty = -2.0e38f;   // m before the first finite entry (finite: no inf - inf)
constexpr float kDMin = -1.0e30f;       // rescale offsets below this have exp(d) = 0 anyway

struct Ent {
  float m, s, t;
};

__device__ __forceinline__ Ent ent_empty() { return {kEntEmpty, 0.f, 0.f}; }

// rescale a to the maximum mn >= a.m: s' = s r, t' = r (t + s d) with d = a.m - mn, r = exp(d)
__device__ __forceinline__ void ent_rescale(Ent& a, float mn) {
  const float d = fmaxf(a.m - mn, kDMin);
  const float r = fast_exp2(d * kLog2e);
  a.t = r * __builtin_fmaf(a.s, d, a.t);
  a.s *= r;
  a.m = mn;
}

// fold N entries whose largest is cm (-inf when all are masked)
template <int N>
__device__ __forceinline__ void ent_fold(Ent& a, const float* x, float cm) {
  ent_rescale(a, fmaxf(a.m, cm));
#pragma unroll
  for (int i = 0; i < N; ++i) {
    const float d = x[i] - a.m;                    // <= 0; -inf for a masked entry
    const float e = fast_exp2(d * kLog2e);          // exp2(-inf) = 0
    a.s += e;
    a.t = __builtin_fmaf(e, fmaxf(d, kDMin), a.t);  // a masked entry: 0 * kDMin = 0
  }
}

__device__ __forceinline__ Ent ent_merge(Ent a, const Ent& b) {
  const float mn = fmaxf(a.m, b.m);
  Ent c = b;
  ent_rescale(a, mn);
  ent_rescale(c, mn);
  return {mn, a.s + c.s, a.t + c.t};
}

__device__ __forceinline__ Ent ent_wave_merge(Ent a) {
#pragma unroll
  for (int k = 32; k >= 1; k >>= 1) {
    Ent o;
    o.m = __shfl_xor(a.m, k);
    o.s = __shfl_xor(a.s, k);
    o.t = __shfl_xor(a.t, k);
    a = ent_merge(a, o);
  }
  return a;
}

__device__ __forceinline__ void ent_finalize(const Ent& a, const UncRule& ru, dls_row_uncertainty* out) {
  dls_row_uncertainty r;
  if (a.s == 0.f) {   // no finite entry: nothing is known, the local terms take full weight
    r.entropy = __builtin_nanf("");
    r.max_prob = __builtin_nanf("");
    r.u = 1.f;
  } else {
    const float inv = 1.f / a.s;
    r.entropy = fast_log2(a.s) * kLn2 - a.t * inv;
    r.max_prob = inv;
    r.u = ru.measure == DLS_UNC_ENTROPY ? r.entropy * ru.inv_log_v : (1.f - inv) * ru.maxprob_scale;
  }
  r.gate = fminf(1.f, fmaxf(0.f, (r.u - ru.h_lo) * ru.inv_width));
  *out = r;
}

template <typename T>
__device__ __forceinline__ int head_elems(const T* p, int V) {
  const int h = (int)(((16u - ((uint32_t)(uintptr_t)p & 15u)) & 15u) / sizeof(T));
  return h < V ? h : V;
}

template <typename T>
__global__ __launch_bounds__(kThreads) void k_unc_part(const T* __restrict__ L, int V, UncRule ru,
                                                       float4* __restrict__ part_out,
                                                       dls_row_uncertainty* __restrict__ out) {
  constexpr int N = Chunk<T>::N;
  __shared__ float sh[3][kThreads / 64];
  const int row = blockIdx.x, part = blockIdx.y, parts = gridDim.y;
  const T* Lr = L + (size_t)row * V;
  const int h0 = head_elems(Lr, V);
  const int nch = (V - h0) / N;
  const int tail0 = h0 + nch * N;
  const int c0 = (int)((int64_t)nch * part / parts), c1 = (int)((int64_t)nch * (part + 1) / parts);
  const int t = threadIdx.x;

  Ent a = ent_empty();
  if (part == 0 && t < h0) {
    const float x = to_f32(Lr[t]);
    ent_fold<1>(a, &x, x);
  }
  // software pipeline: the next iteration's chunks are in flight while this one is folded
  // (indices past the range clamped to its last chunk: loaded, never folded)
  const int clast = c1 > c0 ? c1 - 1 : c0;
  uint4 raw[kUnroll];
  if (c1 > c0) {
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) raw[u] = stream_load16(Lr + h0 + (size_t)min(c0 + t + u * kThreads, clast) * N);
  }
  for (int c = c0 + t; c < c1; c += kThreads * kUnroll) {
    uint4 nraw[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
      nraw[u] = stream_load16(Lr + h0 + (size_t)min(c + kThreads * kUnroll + u * kThreads, clast) * N);
    if (c + (kUnroll - 1) * kThreads < c1) {   // every chunk in range: one rescale for all of them
      float x[N * kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) Chunk<T>::widen(raw[u], x + u * N);
      float cm = x[0];
#pragma unroll
      for (int i = 1; i < N * kUnroll; ++i) cm = fmaxf(cm, x[i]);
      ent_fold<N * kUnroll>(a, x, cm);
    } else {
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int cc = c + u * kThreads;
        if (cc < c1) {
          float x[N];
          Chunk<T>::widen(raw[u], x);
          float cm = x[0];
#pragma unroll
          for (int i = 1; i < N; ++i) cm = fmaxf(cm, x[i]);
          ent_fold<N>(a, x, cm);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) raw[u] = nraw[u];
  }
  if (part == parts - 1 && t < V - tail0) {
    const float x = to_f32(Lr[tail0 + t]);
    ent_fold<1>(a, &x, x);
  }

  a = ent_wave_merge(a);
  const int wave = t >> 6;
  if ((t & 63) == 0) {
    sh[0][wave] = a.m;
    sh[1][wave] = a.s;
    sh[2][wave] = a.t;
  }
  __syncthreads();
  if (t == 0) {
    Ent b = {sh[0][0], sh[1][0], sh[2][0]};
#pragma unroll
    for (int w = 1; w < kThreads / 64; ++w) b = ent_merge(b, Ent{sh[0][w], sh[1][w], sh[2][w]});
    if (parts == 1) ent_finalize(b, ru, out + row);
    else part_out[(size_t)row * parts + part] = make_float4(b.m, b.s, b.t, 0.f);
  }
}

// one wave per row: lane i merges ranges i, i + 64, ... in order, then the wave merges the lanes
__global__ __launch_bounds__(64) void k_unc_merge(const float4* __restrict__ parts_in, int parts, UncRule ru,
                                                  dls_row_uncertainty* __restrict__ out) {
  const int row = blockIdx.x, lane = threadIdx.x;
  Ent a = ent_empty();
  for (int i = lane; i < parts; i += 64) {
    const float4 p = parts_in[(size_t)row * parts + i];
    a = ent_merge(a, Ent{p.x, p.y, p.z});
  }
  a = ent_wave_merge(a);
  if (lane == 0) ent_finalize(a, ru, out + row);
}

}  // namespace

int uncertainty_parts(int64_t rows, int32_t V) {
  // about four workgroups per CU when rows are few (from 1024 rows on one per row, no merge
  // launch); each range >= 4096 entries
  const int64_t target = 1024;
  int64_t p = (target + rows - 1) / std::max<int64_t>(rows, 1);
  p = std::min<int64_t>(p, std::max<int64_t>(1, V / 4096));
  return (int)std::max<int64_t>(1, std::min<int64_t>(p, 128));
}

size_t uncertainty_workspace_bytes(int64_t rows, int32_t V) {
  const int parts = uncertainty_parts(rows, V);
  return parts > 1 ? (size_t)rows * parts * sizeof(float4) : 0;
}

hipError_t launch_uncertainty(const UncArgs& a, hipStream_t st) {
  const int parts = uncertainty_parts(a.rows, a.V);
  dim3 grid((unsigned)a.rows, (unsigned)parts);
  if (a.dtype == DLS_BF16)
    k_unc_part<bf16_t><<<grid, kThreads, 0, st>>>((const bf16_t*)a.long_logits, a.V, a.rule, a.partials, a.out);
  else
    k_unc_part<float><<<grid, kThreads, 0, st>>>((const float*)a.long_logits, a.V, a.rule, a.partials, a.out);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || parts == 1) return e;
  k_unc_merge<<<(unsigned)a.rows, 64, 0, st>>>(a.partials, parts, a.rule, a.out);
  return hipGetLastError();
}

}  // namespace dls
