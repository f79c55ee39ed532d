// One DeLS-Spec draft block per sequence (Algorithm 1, the decoding loop), with the
// App. A RNN local head.  For each draft position j (sequential in j):
//
//   gather   x = E[u_j]              u_0 = last accepted token, u_j = d_{j-1}
//   GRU      h <- GRU(x, h)          bias-free, gate rows (r, z, n), h = 0 at j = 0
//   rank     rho = SiLU(W_rank h)
//   LM head  l_S = W_vocab rho       never written to HBM
//   combine  l = w_long l_L + alpha l_S - beta l_P, online LSEs, top-2, argmax
//   select   d_j = argmax l           fed back as u_{j+1}
//
// Phases are separate launches on the caller's stream.  Every phase spreads its
// weight matrix over the whole chip; the decoded token never leaves the device.
#include "dels_internal.hpp"

namespace dls {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kBC = 4;            // sequences handled together in the GEMV phases
constexpr int kVocabUnroll = 4;   // row sets in flight per wave in the LM-head GEMV

template <int N>
__device__ __forceinline__ float dotn(const float* a, const float* b) {
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < N; ++i) s = __builtin_fmaf(a[i], b[i], s);
  return s;
}

// ----------------------------------------------------------------------------------
// GRU cell: one wave per hidden unit k (gate rows k, H+k, 2H+k of W_ih and W_hh).
// ----------------------------------------------------------------------------------
template <typename WT>
__global__ __launch_bounds__(kThreads) void k_gru(const WT* __restrict__ emb, const WT* __restrict__ w_ih,
                                                  const WT* __restrict__ w_hh, int d, int H, int V,
                                                  const int32_t* __restrict__ tok, const float* __restrict__ h_in,
                                                  int h_zero, float* __restrict__ h_out, int batch) {
  constexpr int N = Chunk<WT>::N;
  const int lane = threadIdx.x & 63;
  const int k = blockIdx.x * kWaves + (threadIdx.x >> 6);
  if (k >= H) return;
  const WT* wr = w_ih + (size_t)k * d;
  const WT* wz = w_ih + (size_t)(H + k) * d;
  const WT* wn = w_ih + (size_t)(2 * H + k) * d;
  const WT* ur = w_hh + (size_t)k * H;
  const WT* uz = w_hh + (size_t)(H + k) * H;
  const WT* un = w_hh + (size_t)(2 * H + k) * H;
  const int dc = d / N, hc = H / N;

  for (int b0 = 0; b0 < batch; b0 += kBC) {
    float ar[kBC], az[kBC], anx[kBC], anh[kBC];
    const WT* xr[kBC];
#pragma unroll
    for (int b = 0; b < kBC; ++b) {
      ar[b] = az[b] = anx[b] = anh[b] = 0.f;
      const int bb = b0 + b < batch ? b0 + b : b0;
      const int t = tok[bb];
      xr[b] = emb + (size_t)((unsigned)t < (unsigned)V ? t : 0) * d;   // out-of-range input reads as 0
    }
#pragma unroll 2
    for (int c = lane; c < dc; c += 64) {
      float w0[N], w1[N], w2[N];
      Chunk<WT>::load(wr + c * N, w0);
      Chunk<WT>::load(wz + c * N, w1);
      Chunk<WT>::load(wn + c * N, w2);
#pragma unroll
      for (int b = 0; b < kBC; ++b) {
        if (b0 + b < batch) {
          float x[N];
          Chunk<WT>::load(xr[b] + c * N, x);
          ar[b] += dotn<N>(w0, x);
          az[b] += dotn<N>(w1, x);
          anx[b] += dotn<N>(w2, x);
        }
      }
    }
    if (!h_zero) {
#pragma unroll 2
      for (int c = lane; c < hc; c += 64) {
        float w0[N], w1[N], w2[N];
        Chunk<WT>::load(ur + c * N, w0);
        Chunk<WT>::load(uz + c * N, w1);
        Chunk<WT>::load(un + c * N, w2);
#pragma unroll
        for (int b = 0; b < kBC; ++b) {
          if (b0 + b < batch) {
            float hv[N];
            const float* hp = h_in + (size_t)(b0 + b) * H + c * N;
#pragma unroll
            for (int i = 0; i < N; ++i) hv[i] = hp[i];
            ar[b] += dotn<N>(w0, hv);
            az[b] += dotn<N>(w1, hv);
            anh[b] += dotn<N>(w2, hv);
          }
        }
      }
    }
#pragma unroll
    for (int b = 0; b < kBC; ++b) {
      const float sr = wave_sum(ar[b]), sz = wave_sum(az[b]);
      const float snx = wave_sum(anx[b]), snh = wave_sum(anh[b]);
      if (lane == 0 && b0 + b < batch) {
        const float rg = sigmoidf_(sr), zg = sigmoidf_(sz);
        const float ng = tanhf_(snx + rg * snh);
        const float hp = h_zero ? 0.f : h_in[(size_t)(b0 + b) * H + k];
        h_out[(size_t)(b0 + b) * H + k] = (1.f - zg) * ng + zg * hp;
      }
    }
  }
}

// ----------------------------------------------------------------------------------
// rho = SiLU(W_rank h): one wave per rank row.
// ----------------------------------------------------------------------------------
template <typename WT>
__global__ __launch_bounds__(kThreads) void k_rank(const WT* __restrict__ w_rank, int H, int r,
                                                   const float* __restrict__ h, float* __restrict__ rho,
                                                   int batch) {
  constexpr int N = Chunk<WT>::N;
  const int lane = threadIdx.x & 63;
  const int i = blockIdx.x * kWaves + (threadIdx.x >> 6);
  if (i >= r) return;
  const WT* wrow = w_rank + (size_t)i * H;
  for (int b0 = 0; b0 < batch; b0 += kBC) {
    float acc[kBC];
#pragma unroll
    for (int b = 0; b < kBC; ++b) acc[b] = 0.f;
    for (int c = lane; c < H / N; c += 64) {
      float w[N];
      Chunk<WT>::load(wrow + c * N, w);
#pragma unroll
      for (int b = 0; b < kBC; ++b) {
        if (b0 + b < batch) {
          const float* hp = h + (size_t)(b0 + b) * H + c * N;
          float hv[N];
#pragma unroll
          for (int e = 0; e < N; ++e) hv[e] = hp[e];
          acc[b] += dotn<N>(w, hv);
        }
      }
    }
#pragma unroll
    for (int b = 0; b < kBC; ++b) {
      const float s = wave_sum(acc[b]);
      if (lane == 0 && b0 + b < batch) rho[(size_t)(b0 + b) * r + i] = siluf_(s);
    }
  }
}

// ----------------------------------------------------------------------------------
// LM head + combine over one vocabulary slice per workgroup.  The short logits of
// the slice stay in LDS; per-(sequence, slice) partial statistics go to HBM.
// GEMV layout: 16 lanes per vocabulary row, each lane a set of 16-byte chunks of the row.
// ----------------------------------------------------------------------------------
template <typename WT, typename LT, bool PRIOR>
__global__ __launch_bounds__(kThreads) void k_lmhead(const WT* __restrict__ w_vocab, int V, int r,
                                                     const float* __restrict__ rho,
                                                     const LT* __restrict__ long_j, size_t long_bstride,
                                                     const float* __restrict__ prior, float wl, float al,
                                                     float be, int slice, int long_only,
                                                     Partial* __restrict__ partials, int batch, Sampler smp,
                                                     int j, const dls_row_uncertainty* __restrict__ unc, int B) {
  constexpr int N = Chunk<WT>::N;
  extern __shared__ float smem[];
  float* s_rho = smem;                       // kBC * r
  float* s_S = smem + kBC * r;               // kBC * slice
  __shared__ Partial sh[kWaves];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int sub = lane & 15, grp = lane >> 4;
  const int v0 = blockIdx.x * slice;
  const int nv = min(slice, V - v0);
  const int rc = r / N;

  for (int b0 = 0; b0 < batch; b0 += kBC) {
    const int nb = min(kBC, batch - b0);
    if (!long_only) {
      for (int i = threadIdx.x; i < nb * r; i += kThreads) s_rho[i] = rho[(size_t)b0 * r + i];
      __syncthreads();
      // each wave: row sets of 4 rows (one per 16-lane group), kVocabUnroll sets at a time
      for (int base = wave * 4; base < nv; base += kWaves * 4 * kVocabUnroll) {
        float acc[kVocabUnroll][kBC];
#pragma unroll
        for (int u = 0; u < kVocabUnroll; ++u)
#pragma unroll
          for (int b = 0; b < kBC; ++b) acc[u][b] = 0.f;
#pragma unroll
        for (int u = 0; u < kVocabUnroll; ++u) {
          const int row = base + u * kWaves * 4 + grp;
          if (row < nv) {
            const WT* wrow = w_vocab + (size_t)(v0 + row) * r;
            for (int c = sub; c < rc; c += 16) {
              float w[N];
              Chunk<WT>::load(wrow + c * N, w);
#pragma unroll
              for (int b = 0; b < kBC; ++b)
                if (b < nb) acc[u][b] += dotn<N>(w, s_rho + b * r + c * N);
            }
          }
        }
#pragma unroll
        for (int u = 0; u < kVocabUnroll; ++u) {
          const int row = base + u * kWaves * 4 + grp;
#pragma unroll
          for (int b = 0; b < kBC; ++b) {
            float s = acc[u][b];
            s += __shfl_xor(s, 8);
            s += __shfl_xor(s, 4);
            s += __shfl_xor(s, 2);
            s += __shfl_xor(s, 1);
            if (sub == 0 && row < nv && b < nb) s_S[b * slice + row] = s;
          }
        }
      }
      __syncthreads();
    }
    // combine over the slice, one sequence at a time; sampling folds l / T into the fused
    // log-sum-exp and l / T + g into the top-2
    const bool sample = smp.inv_temp != 0.f;
    for (int b = 0; b < nb; ++b) {
      const LT* lrow = long_j + (size_t)(b0 + b) * long_bstride;
      // adaptive fusion: this row's gate scales the local terms
      const float g = unc ? unc[(size_t)(b0 + b) * B + j].gate : 1.f;
      const float alb = al * g, beb = be * g;
      Partial P = partial_empty();
      for (int i = threadIdx.x; i < nv; i += kThreads) {
        const int v = v0 + i;
        float a = to_f32(lrow[v]);
        float f;
        if (long_only) {
          f = weighted(wl, a);
        } else {
          float s = s_S[b * slice + i];
          f = __builtin_fmaf(alb, s, weighted(wl, a));
          if (PRIOR) f = minus_weighted(f, beb, prior[v]);
          lse_fold<1>(P.S, &s, s);
        }
        lse_fold<1>(P.L, &a, a);
        if (sample) {
          f *= smp.inv_temp;
          lse_fold<1>(P.F, &f, f);
          top2_push(P, f + gumbel_at(smp, b0 + b, j, v), v);
        } else {
          lse_fold<1>(P.F, &f, f);
          top2_push(P, f, v);
        }
      }
      P = block_merge(P, sh, kWaves);
      if (threadIdx.x == 0) partials[(size_t)(b0 + b) * gridDim.x + blockIdx.x] = P;
    }
    __syncthreads();
  }
}

// ----------------------------------------------------------------------------------
// Merge the slice partials of each sequence: the drafted token of position j.
// ----------------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void k_select(const Partial* __restrict__ partials, int groups, float wl,
                                                     float al, int long_only, int j, int B,
                                                     int32_t* __restrict__ out_tokens,
                                                     dls_row_stats* __restrict__ out_stats,
                                                     int32_t* __restrict__ tok_next, Sampler smp,
                                                     const dls_row_uncertainty* __restrict__ unc) {
  __shared__ Partial sh[kWaves];
  const int b = blockIdx.x;
  Partial P = partial_empty();
  for (int i = threadIdx.x; i < groups; i += kThreads) P = partial_merge(P, partials[(size_t)b * groups + i]);
  P = block_merge(P, sh, kWaves);
  if (threadIdx.x == 0) {
    int32_t t;
    const bool sample = smp.inv_temp != 0.f;
    const int ti = P.i1 == 0x7fffffff ? 0 : P.i1;
    const float alb = unc ? al * unc[(size_t)b * B + j].gate : al;
    finalize_row(P, wl, alb, long_only != 0, &t, out_stats ? out_stats + (size_t)b * B + j : nullptr, nullptr,
                 sample ? gumbel_at(smp, b, j, ti) : 0.f, smp.temp);
    out_tokens[(size_t)b * B + j] = t;
    tok_next[b] = t;
  }
}

// Markov head state: rho[b] = E_M[u_b] (App. A, Markov variant), widened to float32.
// One thread per (sequence, rank column).
template <typename WT>
__global__ __launch_bounds__(kThreads) void k_markov_rho(const WT* __restrict__ e_m, int V, int r,
                                                         const int32_t* __restrict__ tok, float* __restrict__ rho,
                                                         int batch) {
  const int i = blockIdx.x * kThreads + threadIdx.x;
  if (i >= batch * r) return;
  const int b = i / r, c = i % r;
  const int t = tok[b];
  const int u = (unsigned)t < (unsigned)V ? t : 0;   // out-of-range input reads as 0
  rho[i] = to_f32(e_m[(size_t)u * r + c]);
}

template <typename WT, typename LT, bool PRIOR>
hipError_t launch_draft_t(const DraftArgs& a, hipStream_t st) {
  const dls_local_head& hd = a.head;
  const int batch = a.batch, B = a.B, V = hd.V, H = hd.H, r = hd.r, d = hd.d;
  char* ws = a.ws;
  float* h0 = (float*)(ws + a.lay.off_h0);
  float* h1 = (float*)(ws + a.lay.off_h1);
  float* rho = (float*)(ws + a.lay.off_rho);
  int32_t* tok = (int32_t*)(ws + a.lay.off_tok);
  Partial* part = (Partial*)(ws + a.lay.off_part);
  const WT* emb = (const WT*)hd.emb;
  const WT* w_ih = (const WT*)hd.w_ih;
  const WT* w_hh = (const WT*)hd.w_hh;
  const WT* w_rank = (const WT*)hd.w_rank;
  const WT* w_vocab = (const WT*)hd.w_vocab;
  const LT* L = (const LT*)a.long_logits;
  const size_t bstride = (size_t)B * V;
  const bool literal = (a.f.flags & DLS_FIRST_ROW_LONG_ONLY) != 0;
  const size_t lds = (size_t)(kBC * r + kBC * a.lay.slice) * sizeof(float);
  const float wl = a.f.w_long;
  hipError_t e;

  const int32_t* tok_in = a.last_token;
  float* hc = h0;   // current state
  float* hn = h1;   // next state
  bool first_head_step = true;
  for (int j = 0; j < B; ++j) {
    const bool long_only = literal && j == 0;
    const float al = a.alphas ? a.alphas[j] : a.f.alpha;
    const float be = a.prior ? (a.betas ? a.betas[j] : a.f.beta) : 0.f;
    if (!long_only && hd.kind == DLS_HEAD_MARKOV) {
      k_markov_rho<WT><<<(batch * r + kThreads - 1) / kThreads, kThreads, 0, st>>>(emb, V, r, tok_in, rho, batch);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    } else if (!long_only) {
      k_gru<WT><<<(H + kWaves - 1) / kWaves, kThreads, 0, st>>>(emb, w_ih, w_hh, d, H, V, tok_in, hc,
                                                                 first_head_step ? 1 : 0, hn, batch);
      if ((e = hipGetLastError()) != hipSuccess) return e;
      k_rank<WT><<<(r + kWaves - 1) / kWaves, kThreads, 0, st>>>(w_rank, H, r, hn, rho, batch);
      if ((e = hipGetLastError()) != hipSuccess) return e;
      std::swap(hc, hn);
      first_head_step = false;
    }
    k_lmhead<WT, LT, PRIOR><<<a.lay.groups, kThreads, lds, st>>>(
        w_vocab, V, r, rho, L + (size_t)j * V, bstride, a.prior, wl, al, be, a.lay.slice, long_only ? 1 : 0,
        part, batch, a.smp, j, a.unc, B);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    k_select<<<batch, kThreads, 0, st>>>(part, a.lay.groups, wl, al, long_only ? 1 : 0, j, B, a.out_tokens,
                                         a.out_stats, tok, a.smp, a.unc);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    tok_in = tok;
  }
  return hipSuccess;
}

template <typename WT>
hipError_t launch_draft_w(const DraftArgs& a, hipStream_t st) {
  const bool pr = a.prior != nullptr;
  if (a.long_dtype == DLS_BF16)
    return pr ? launch_draft_t<WT, bf16_t, true>(a, st) : launch_draft_t<WT, bf16_t, false>(a, st);
  return pr ? launch_draft_t<WT, float, true>(a, st) : launch_draft_t<WT, float, false>(a, st);
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

}  // namespace

DraftLayout draft_layout(const dls_local_head& h, int32_t batch, int32_t B) {
  (void)B;
  DraftLayout L;
  const int64_t per = (h.V + 1023) / 1024;
  int slice = (int)((per + 15) / 16 * 16);
  slice = std::max(64, std::min(2048, slice));
  L.slice = slice;
  L.groups = (int)((h.V + slice - 1) / slice);
  size_t o = 0;
  L.off_h0 = o; o = align256(o + (size_t)batch * h.H * 4);
  L.off_h1 = o; o = align256(o + (size_t)batch * h.H * 4);
  L.off_rho = o; o = align256(o + (size_t)batch * h.r * 4);
  L.off_tok = o; o = align256(o + (size_t)batch * 4);
  L.off_part = o; o = align256(o + (size_t)batch * L.groups * sizeof(Partial));
  L.total = o;
  return L;
}

hipError_t launch_draft(const DraftArgs& a, hipStream_t st) {
  if (a.head.dtype == DLS_BF16) return launch_draft_w<bf16_t>(a, st);
  return launch_draft_w<float>(a, st);
}

}  // namespace dls
