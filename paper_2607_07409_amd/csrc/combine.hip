// Fused combine + greedy argmax over independent rows (Sec. 4.3 fusion equation and
// the decode step of Algorithm 1), short logits given in HBM.
//
// A row of V elements is split into `parts` contiguous ranges, one workgroup each.
// Every thread streams 16-byte chunks of the long and short rows (coalesced across
// the workgroup, non-temporal loads), forms l = w_long*l_L + alpha*l_S - beta*l_P in float32 and folds
// the chunk into its running (max, sum exp) for l_L, l_S, l and into the top-2 of l.
// The workgroup merge is a fixed-order butterfly, so results are deterministic.
// Without row statistics or scores only the running maximum of l and its index are
// kept: the argmax needs no normaliser, and the kernel is then bound by HBM bandwidth.
// With parts > 1 a second kernel merges the per-range partials of each row.
#include "dels_internal.hpp"
#include "stream_load.hpp"

namespace dls {

namespace {

constexpr int kThreads = 256;
constexpr int kWideThreads = 1024;
constexpr int kUnroll = 2;

// l_v for one element (the GPU's float32 reading of the fusion equation).  The launch resolves
// the zero-weight cases (a term whose weight is 0 is absent, masked entries included): WLONG
// means w_long != 0, and PRIOR a prior with beta != 0, so no entry needs a test of its weight.
template <bool PRIOR, bool WLONG>
__device__ __forceinline__ float fuse1(float a, float b, float p, float wl, float al, float be) {
  float f = __builtin_fmaf(al, b, WLONG ? wl * a : 0.f);
  if (PRIOR) f = __builtin_fmaf(-be, p, f);
  return f;
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x = fmaxf(x, __shfl_xor(x, m));
  return x;
}

// running maximum and its index only (lowest index among equal values)
__device__ __forceinline__ void top1_push(Partial& p, float x, int idx) {
  const bool up = x > p.t1;
  p.t1 = up ? x : p.t1;
  p.i1 = up ? idx : p.i1;
}

template <typename T, bool PRIOR, bool STATS, bool WLONG>
__device__ __forceinline__ void fold_scalar(Partial& P, const T* Lr, const T* Sr, const float* prior,
                                            int v, float wl, float al, float be) {
  float a = to_f32(Lr[v]), b = to_f32(Sr[v]);
  float f = fuse1<PRIOR, WLONG>(a, b, PRIOR ? prior[v] : 0.f, wl, al, be);
  if (STATS) {   // finite-start states (see k_combine_part)
    lse_fold_fin<1>(P.L, &a, a);
    lse_fold_fin<1>(P.S, &b, b);
    lse_fold_fin<1>(P.F, &f, f);
    top2_push(P, f, v);
  } else {
    top1_push(P, f, v);
  }
}

template <typename T>
__device__ __forceinline__ int head_elems(const T* p, int V) {
  const int h = (int)(((16u - ((uint32_t)(uintptr_t)p & 15u)) & 15u) / sizeof(T));
  return h < V ? h : V;
}

template <typename T, bool PRIOR, bool STATS, int NT, bool WLONG>
__global__ __launch_bounds__(NT) void k_combine_part(
    const T* __restrict__ L, const T* __restrict__ S, const float* __restrict__ prior, int V,
    float wl, float al, float be, Partial* __restrict__ part_out, int32_t* __restrict__ out_token,
    dls_row_stats* __restrict__ out_stats, float* __restrict__ norm_out) {
  constexpr int N = Chunk<T>::N;
  constexpr int NU = N * kUnroll;   // entries per thread and iteration
  // Workgroups of 256 threads (four per CU from 1024 rows on) run a software pipeline: the
  // next iteration's chunks are in flight while this one is folded (indices past the range
  // clamped to its last chunk: loaded, never folded).  With row statistics they also skip the
  // top-two pushes of iterations whose entries all lie below the wave's threshold.  The one
  // 1024-thread workgroup per row of 256 to 1023 rows measured faster without either.
  constexpr bool kPipe = NT < 1024;
  __shared__ Partial sh[NT / 64];
  const int row = blockIdx.x, part = blockIdx.y, parts = gridDim.y;
  const T* Lr = L + (size_t)row * V;
  const T* Sr = S + (size_t)row * V;
  const int h0 = head_elems(Lr, V);
  const int nch = (V - h0) / N;
  const int tail0 = h0 + nch * N;
  const int c0 = (int)((int64_t)nch * part / parts), c1 = (int)((int64_t)nch * (part + 1) / parts);
  const int t = threadIdx.x;

  Partial P = partial_empty();
  if (STATS) P.L.m = P.S.m = P.F.m = kFinMin;   // the finite start of the folds below
  if (part == 0 && t < h0) fold_scalar<T, PRIOR, STATS, WLONG>(P, Lr, Sr, prior, t, wl, al, be);

  const int clast = c1 > c0 ? c1 - 1 : c0;
  uint4 ra[kUnroll], rb[kUnroll];
  if (kPipe && c1 > c0) {
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int cc = min(c0 + t + u * NT, clast);
      ra[u] = stream_load16(Lr + h0 + (size_t)cc * N);
      rb[u] = stream_load16(Sr + h0 + (size_t)cc * N);
    }
  }
  // Top two: an entry below wthr, the largest second value among the wave's lanes (so two
  // entries of the row at least that large), can be neither of the row's top two.  The
  // threshold is reduced over all 64 lanes; a full iteration runs with part of a wave inactive
  // only as that wave's last full iteration (the lanes of a wave start at most 63 chunks apart
  // and advance together by NT x kUnroll chunks), so a threshold formed then is never used.
  float wthr = -INFINITY;
  for (int c = c0 + t; c < c1; c += NT * kUnroll) {
    uint4 na[kUnroll], nb[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      if (kPipe) {
        const int cc = min(c + NT * kUnroll + u * NT, clast);
        na[u] = stream_load16(Lr + h0 + (size_t)cc * N);
        nb[u] = stream_load16(Sr + h0 + (size_t)cc * N);
      } else if (c + u * NT < c1) {
        ra[u] = stream_load16(Lr + h0 + (size_t)(c + u * NT) * N);
        rb[u] = stream_load16(Sr + h0 + (size_t)(c + u * NT) * N);
      }
    }
    if (STATS && c + (kUnroll - 1) * NT < c1) {
      // every chunk of the iteration in range: one fold per log-sum-exp, one rescale per NU entries
      float a[NU], b[NU], f[NU];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        Chunk<T>::widen(ra[u], a + u * N);
        Chunk<T>::widen(rb[u], b + u * N);
        const int v0 = h0 + (c + u * NT) * N;
#pragma unroll
        for (int i = 0; i < N; ++i)
          f[u * N + i] = fuse1<PRIOR, WLONG>(a[u * N + i], b[u * N + i], PRIOR ? prior[v0 + i] : 0.f, wl, al, be);
      }
      float ma = a[0], mb = b[0], mf = f[0];
#pragma unroll
      for (int i = 1; i < NU; ++i) {
        ma = fmaxf(ma, a[i]);
        mb = fmaxf(mb, b[i]);
        mf = fmaxf(mf, f[i]);
      }
      lse_fold_fin<NU>(P.L, a, ma);
      lse_fold_fin<NU>(P.S, b, mb);
      lse_fold_fin<NU>(P.F, f, mf);
      const bool hit = !kPipe || mf >= wthr;
      if (!kPipe || __builtin_amdgcn_ballot_w64(hit)) {
        if (hit) {
#pragma unroll
          for (int u = 0; u < kUnroll; ++u) {
            const int v0 = h0 + (c + u * NT) * N;
#pragma unroll
            for (int i = 0; i < N; ++i) top2_push(P, f[u * N + i], v0 + i);
          }
        }
        if (kPipe) wthr = wave_max(P.t2);
      }
    } else if (STATS) {
      // the last, partial iteration: chunk by chunk
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int cc = c + u * NT;
        if (cc < c1) {
          float a[N], b[N], f[N];
          Chunk<T>::widen(ra[u], a);
          Chunk<T>::widen(rb[u], b);
          const int v0 = h0 + cc * N;
#pragma unroll
          for (int i = 0; i < N; ++i) f[i] = fuse1<PRIOR, WLONG>(a[i], b[i], PRIOR ? prior[v0 + i] : 0.f, wl, al, be);
          float ma = a[0], mb = b[0], mf = f[0];
#pragma unroll
          for (int i = 1; i < N; ++i) {
            ma = fmaxf(ma, a[i]);
            mb = fmaxf(mb, b[i]);
            mf = fmaxf(mf, f[i]);
          }
          lse_fold_fin<N>(P.L, a, ma);
          lse_fold_fin<N>(P.S, b, mb);
          lse_fold_fin<N>(P.F, f, mf);
#pragma unroll
          for (int i = 0; i < N; ++i) top2_push(P, f[i], v0 + i);
        }
      }
    } else {
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int cc = c + u * NT;
        if (cc < c1) {
          float a[N], b[N];
          Chunk<T>::widen(ra[u], a);
          Chunk<T>::widen(rb[u], b);
          const int v0 = h0 + cc * N;
#pragma unroll
          for (int i = 0; i < N; ++i) top1_push(P, fuse1<PRIOR, WLONG>(a[i], b[i], PRIOR ? prior[v0 + i] : 0.f, wl, al, be), v0 + i);
        }
      }
    }
    if (kPipe) {
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        ra[u] = na[u];
        rb[u] = nb[u];
      }
    }
  }
  if (part == parts - 1 && t < V - tail0) fold_scalar<T, PRIOR, STATS, WLONG>(P, Lr, Sr, prior, tail0 + t, wl, al, be);
  if (STATS) {
    fin_to_empty(P.L);
    fin_to_empty(P.S);
    fin_to_empty(P.F);
  }

  P = block_merge(P, sh, NT / 64);
  if (t == 0) {
    if (parts == 1)
      finalize_row(P, wl, al, false, out_token + row, out_stats ? out_stats + row : nullptr,
                   norm_out ? norm_out + row : nullptr);
    else
      part_out[(size_t)row * parts + part] = P;
  }
}

__global__ __launch_bounds__(64) void k_combine_finalize(const Partial* __restrict__ parts_in, int parts,
                                                         float wl, float al, int32_t* __restrict__ out_token,
                                                         dls_row_stats* __restrict__ out_stats,
                                                         float* __restrict__ norm_out) {
  const int row = blockIdx.x, lane = threadIdx.x;
  Partial P = partial_empty();
  for (int i = lane; i < parts; i += 64) P = partial_merge(P, parts_in[(size_t)row * parts + i]);
  P = allred_partial(P, WaveXor{});
  if (lane == 0)
    finalize_row(P, wl, al, false, out_token + row, out_stats ? out_stats + row : nullptr,
                 norm_out ? norm_out + row : nullptr);
}

// c_v = l_v - (w_long * lse_long + alpha * lse_short), recomputing l_v exactly as above
template <typename T, bool PRIOR, bool WLONG>
__global__ __launch_bounds__(kThreads) void k_combine_scores(const T* __restrict__ L, const T* __restrict__ S,
                                                             const float* __restrict__ prior, int V, float wl,
                                                             float al, float be, const float* __restrict__ norm,
                                                             float* __restrict__ scores) {
  const int row = blockIdx.x;
  const T* Lr = L + (size_t)row * V;
  const T* Sr = S + (size_t)row * V;
  float* Cr = scores + (size_t)row * V;
  const float nr = norm[row];
  for (int v = blockIdx.y * kThreads + threadIdx.x; v < V; v += gridDim.y * kThreads)
    Cr[v] = fuse1<PRIOR, WLONG>(to_f32(Lr[v]), to_f32(Sr[v]), PRIOR ? prior[v] : 0.f, wl, al, be) - nr;
}

template <typename T, bool PRIOR, bool WLONG>
hipError_t launch_combine_t(const CombineArgs& a, hipStream_t st) {
  const int parts = a.parts;
  dim3 grid((unsigned)a.rows, parts);
  // the normaliser feeds only the statistics and the score rows
  const bool stats = a.out_stats != nullptr || a.out_scores != nullptr;
  float* norm = stats ? a.norm : nullptr;
  const bool wide = combine_wide(a.rows, a.V);
  auto kern = wide ? (stats ? k_combine_part<T, PRIOR, true, kWideThreads, WLONG>
                             : k_combine_part<T, PRIOR, false, kWideThreads, WLONG>)
                   : (stats ? k_combine_part<T, PRIOR, true, kThreads, WLONG> : k_combine_part<T, PRIOR, false, kThreads, WLONG>);
  kern<<<grid, wide ? kWideThreads : kThreads, 0, st>>>((const T*)a.long_logits, (const T*)a.short_logits, a.prior,
                                                        a.V, a.wl, a.al, a.be, a.partials, a.out_token, a.out_stats,
                                                        norm);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (parts > 1) {
    k_combine_finalize<<<(unsigned)a.rows, 64, 0, st>>>(a.partials, parts, a.wl, a.al, a.out_token,
                                                         a.out_stats, norm);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (a.out_scores) {
    dim3 g2((unsigned)a.rows, (unsigned)std::min<int64_t>((a.V + kThreads - 1) / kThreads, 64));
    k_combine_scores<T, PRIOR, WLONG><<<g2, kThreads, 0, st>>>((const T*)a.long_logits, (const T*)a.short_logits,
                                                        a.prior, a.V, a.wl, a.al, a.be, a.norm, a.out_scores);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace

// 256 to 1023 rows: one row per workgroup of 1024 threads (about one per CU, as many bytes in
// flight as four workgroups of 256 threads), so that no merge launch follows
bool combine_wide(int64_t rows, int32_t V) { return rows >= 256 && rows < 1024 && V >= 4 * kWideThreads; }

int combine_parts(int64_t rows, int32_t V) {
  if (combine_wide(rows, V)) return 1;
  // enough workgroups to cover the chip when rows are few (four per CU); each range >= 2048
  // elements.  From 1024 rows on every row is one workgroup and no merge launch follows.
  const int64_t target = 1024;
  int64_t p = (target + rows - 1) / std::max<int64_t>(rows, 1);
  const int64_t cap = std::max<int64_t>(1, V / 2048);
  p = std::min(p, cap);
  return (int)std::max<int64_t>(1, std::min<int64_t>(p, 256));
}

hipError_t launch_combine(const CombineArgs& a, hipStream_t st) {
  // a zero weight removes its term, masked entries included: a prior with beta = 0 is no prior
  const bool pr = a.prior != nullptr && a.be != 0.f;
  const bool wlong = a.wl != 0.f;
  if (a.dtype == DLS_BF16)
    return pr ? (wlong ? launch_combine_t<bf16_t, true, true>(a, st) : launch_combine_t<bf16_t, true, false>(a, st))
              : (wlong ? launch_combine_t<bf16_t, false, true>(a, st) : launch_combine_t<bf16_t, false, false>(a, st));
  return pr ? (wlong ? launch_combine_t<float, true, true>(a, st) : launch_combine_t<float, true, false>(a, st))
            : (wlong ? launch_combine_t<float, false, true>(a, st) : launch_combine_t<float, false, false>(a, st));
}

}  // namespace dls
