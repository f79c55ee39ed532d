// Device-side building blocks of the DeLS-Spec drafting kernels (gfx950, wave64).
//
//  * widening loads of 16-byte chunks (bf16 -> 8 floats, f32 -> 4 floats)
//  * the running statistics of one vocabulary range of a fused row: online
//    (max, sum of exp) pairs for the long, short and fused logits and the top-2 of
//    the fused logits with the index of the top-1 (lowest index on ties)
//  * an associative merge of two such partial statistics, used across lanes, waves
//    and workgroups in a fixed order (deterministic results)
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dls {

typedef uint16_t bf16_t;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ float to_f32(bf16_t b) { return __uint_as_float((uint32_t)b << 16); }
__device__ __forceinline__ float to_f32(float f) { return f; }

// 16-byte chunk of T, widened to float
template <typename T> struct Chunk;
template <> struct Chunk<bf16_t> {
  static constexpr int N = 8;
  __device__ __forceinline__ static void load(const bf16_t* p, float* o) {
    const uint4 v = *reinterpret_cast<const uint4*>(p);
    o[0] = bf16_lo(v.x); o[1] = bf16_hi(v.x); o[2] = bf16_lo(v.y); o[3] = bf16_hi(v.y);
    o[4] = bf16_lo(v.z); o[5] = bf16_hi(v.z); o[6] = bf16_lo(v.w); o[7] = bf16_hi(v.w);
  }
  __device__ __forceinline__ static uint4 raw(const bf16_t* p) { return *reinterpret_cast<const uint4*>(p); }
  __device__ __forceinline__ static void widen(const uint4 v, float* o) {
    o[0] = bf16_lo(v.x); o[1] = bf16_hi(v.x); o[2] = bf16_lo(v.y); o[3] = bf16_hi(v.y);
    o[4] = bf16_lo(v.z); o[5] = bf16_hi(v.z); o[6] = bf16_lo(v.w); o[7] = bf16_hi(v.w);
  }
};
template <> struct Chunk<float> {
  static constexpr int N = 4;
  __device__ __forceinline__ static void load(const float* p, float* o) {
    const float4 v = *reinterpret_cast<const float4*>(p);
    o[0] = v.x; o[1] = v.y; o[2] = v.z; o[3] = v.w;
  }
  __device__ __forceinline__ static uint4 raw(const float* p) { return *reinterpret_cast<const uint4*>(p); }
  __device__ __forceinline__ static void widen(const uint4 v, float* o) {
    o[0] = __uint_as_float(v.x); o[1] = __uint_as_float(v.y);
    o[2] = __uint_as_float(v.z); o[3] = __uint_as_float(v.w);
  }
};

// w * x, except that a zero weight gives 0 even for x = -inf: a fusion term weighted by 0 is
// absent (p^0 = 1), masked entries (-inf long logits, an unsmoothed prior's -inf) included
__device__ __forceinline__ float weighted(float w, float x) { return w == 0.f ? 0.f : w * x; }
// f - b * p with the same reading of a zero weight
__device__ __forceinline__ float minus_weighted(float f, float b, float p) {
  return b == 0.f ? f : __builtin_fmaf(-b, p, f);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

__device__ __forceinline__ float sigmoidf_(float x) { return 1.0f / (1.0f + __expf(-x)); }
__device__ __forceinline__ float tanhf_(float x) {
  // tanh x = 1 - 2 / (exp(2x) + 1); exact limits +-1 at overflow/underflow of exp
  return 1.0f - 2.0f / (__expf(2.0f * x) + 1.0f);
}
__device__ __forceinline__ float siluf_(float x) { return x * sigmoidf_(x); }

// ------------------------------------------------------------------------------
// Online log-sum-exp: value = m + ln(s), s = sum_i exp(x_i - m).  m = -inf, s = 0
// is the empty set.
// ------------------------------------------------------------------------------
struct Lse {
  float m, s;
};
__device__ __forceinline__ Lse lse_empty() { return {-INFINITY, 0.f}; }

// fold a chunk of n values whose maximum is cm
template <int n>
__device__ __forceinline__ void lse_fold(Lse& a, const float* x, float cm) {
  const float mn = fmaxf(a.m, cm);
  if (mn == -INFINITY) return;                       // everything so far is -inf
  const float ml = mn * kLog2e;
  float acc = a.s * fast_exp2(a.m * kLog2e - ml);    // exp2(-inf) = 0 covers the empty case
#pragma unroll
  for (int i = 0; i < n; ++i) acc += fast_exp2(__builtin_fmaf(x[i], kLog2e, -ml));
  a.m = mn;
  a.s = acc;
}

// Running log-sum-exps that start from a finite floor (kFinMin instead of -inf) need no test of
// their values: x = -inf adds exp2(-inf) = 0 and never becomes the maximum.  Such a state is
// empty while s == 0; fin_to_empty restores the -inf form before states are merged.
constexpr float kFinMin = -2.0e38f;   // kFinMin * log2(e) is still finite
__device__ __forceinline__ void fin_to_empty(Lse& a) { a.m = a.s > 0.f ? a.m : -INFINITY; }
// n values whose maximum is cm into a finite-start state: one rescale, one exponential per value
template <int n>
__device__ __forceinline__ void lse_fold_fin(Lse& a, const float* x, float cm) {
  const float mn = fmaxf(a.m, cm);
  const float ml = mn * kLog2e;
  float acc = a.s * fast_exp2((a.m - mn) * kLog2e);   // exactly 1 while the maximum stays
#pragma unroll
  for (int i = 0; i < n; ++i) acc += fast_exp2(__builtin_fmaf(x[i], kLog2e, -ml));
  a.m = mn;
  a.s = acc;
}

__device__ __forceinline__ Lse lse_merge(Lse a, Lse b) {
  const float mn = fmaxf(a.m, b.m);
  if (mn == -INFINITY) return lse_empty();
  const float ml = mn * kLog2e;
  return {mn, a.s * fast_exp2(a.m * kLog2e - ml) + b.s * fast_exp2(b.m * kLog2e - ml)};
}
__device__ __forceinline__ float lse_value(Lse a) {
  return a.m == -INFINITY ? -INFINITY : a.m + fast_log2(a.s) * kLn2;
}

// ------------------------------------------------------------------------------
// Partial statistics of a vocabulary range of one fused row.
// ------------------------------------------------------------------------------
struct Partial {
  Lse L, S, F;    // long, short, fused
  float t1, t2;   // top-1 and top-2 fused values
  int i1;         // index of t1 (lowest among equal values)
  int pad;
};
static_assert(sizeof(Partial) == 40, "partial layout");

__device__ __forceinline__ Partial partial_empty() {
  Partial p;
  p.L = p.S = p.F = lse_empty();
  p.t1 = p.t2 = -INFINITY;
  p.i1 = 0x7fffffff;
  p.pad = 0;
  return p;
}

// top-2 update with the values of one thread visited in increasing index order
__device__ __forceinline__ void top2_push(Partial& p, float x, int idx) {
  p.t2 = __builtin_amdgcn_fmed3f(x, p.t1, p.t2);   // t1 >= t2: the median is the new second value
  const bool up = x > p.t1;
  p.t1 = up ? x : p.t1;
  p.i1 = up ? idx : p.i1;
}

__device__ __forceinline__ Partial partial_merge(const Partial& a, const Partial& b) {
  Partial r;
  r.L = lse_merge(a.L, b.L);
  r.S = lse_merge(a.S, b.S);
  r.F = lse_merge(a.F, b.F);
  const bool a_wins = (a.t1 > b.t1) || (a.t1 == b.t1 && a.i1 < b.i1);
  r.t1 = a_wins ? a.t1 : b.t1;
  r.i1 = a_wins ? a.i1 : b.i1;
  r.t2 = a_wins ? fmaxf(a.t2, b.t1) : fmaxf(b.t2, a.t1);
  r.pad = 0;
  return r;
}

// All-reduce of a partial over lane groups, given a lane permutation `x(v, m)` (a shuffle or
// DPP rotate) applied for each m in a list: the three maxima first, then every lane rescales
// its sums once to the common maxima and the sums are added up, then the top-1 as a
// (value, lowest index) maximum and the top-2 as the largest value that is not the winner.
// One exponential per log-sum-exp per lane instead of two per merge step.
template <typename Perm>
__device__ __forceinline__ float allred_max(float v, Perm x) {
  x.each([&](int m) { v = fmaxf(v, x(v, m)); });
  return v;
}
template <typename Perm>
__device__ __forceinline__ float allred_sum(float v, Perm x) {
  x.each([&](int m) { v += x(v, m); });
  return v;
}
template <typename Perm>
__device__ __forceinline__ Lse allred_lse(Lse a, Perm x) {
  const float m = allred_max(a.m, x);
  float s = (a.m == -INFINITY) ? 0.f : a.s * fast_exp2((a.m - m) * kLog2e);
  return {m, allred_sum(s, x)};
}
template <typename Perm>
__device__ __forceinline__ Partial allred_partial(Partial p, Perm x) {
  p.L = allred_lse(p.L, x);
  p.S = allred_lse(p.S, x);
  p.F = allred_lse(p.F, x);
  float T = p.t1;
  int I = p.i1;
  x.each([&](int m) {
    const float ot = x(T, m);
    const int oi = x.i(I, m);
    const bool take = ot > T || (ot == T && oi < I);
    T = take ? ot : T;
    I = take ? oi : I;
  });
  const float c = (p.t1 == T && p.i1 == I) ? p.t2 : p.t1;
  p.t2 = allred_max(c, x);
  p.t1 = T;
  p.i1 = I;
  p.pad = 0;
  return p;
}
// xor shuffles over the 64 lanes of a wave
struct WaveXor {
  template <typename F>
  __device__ __forceinline__ void each(F f) const {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) f(m);
  }
  __device__ __forceinline__ float operator()(float v, int m) const { return __shfl_xor(v, m); }
  __device__ __forceinline__ int i(int v, int m) const { return __shfl_xor(v, m); }
};

// Merge over a workgroup of nwaves waves; the total is returned to every thread.
// `sh` must hold nwaves Partials.  The pairing is fixed, so the result is deterministic.
__device__ __forceinline__ Partial block_merge(Partial p, Partial* sh, int nwaves) {
  p = allred_partial(p, WaveXor{});
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) sh[wave] = p;
  __syncthreads();
  Partial t = sh[0];
  for (int w = 1; w < nwaves; ++w) t = partial_merge(t, sh[w]);
  return t;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m);
  return v;
}

// ------------------------------------------------------------------------------
// Temperature sampling of a draft row by the Gumbel-max rule: the token is the argmax of
// l / T + g with standard Gumbel noise g.  The noise of vocabulary entry v of row (sequence
// b, position j) is word v % 4 of Philox4x32-10 (Salmon et al. 2011) at counter
// (v / 4, j, b, 0) with key (seed low, seed high); u = ((x >> 9) + 1/2) / 2^23 in (0, 1);
// g = -log(-log u).
// ------------------------------------------------------------------------------
struct Sampler {
  float inv_temp;   // 1 / T; 0 decodes greedily
  float temp;       // T (1 when greedy)
  uint32_t seed_lo, seed_hi;
  uint32_t b0;      // index of the launch's first sequence in the call (a call split into launches)
};

__device__ __forceinline__ uint4 philox4x32_10(uint4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    // each 64-bit product is one v_mad_u64_u32 (a low and a high multiply otherwise)
    const uint64_t p0 = (uint64_t)0xD2511F53u * c.x, p1 = (uint64_t)0xCD9E8D57u * c.z;
    c = make_uint4((uint32_t)(p1 >> 32) ^ c.y ^ k0, (uint32_t)p1, (uint32_t)(p0 >> 32) ^ c.w ^ k1, (uint32_t)p0);
  }
  return c;
}

// Gumbel noise of one Philox output word x: u = ((x >> 9) + 1/2) / 2^23, g = -log(-log u).
// The hardware base-2 logarithm keeps e = -log u within 2.7 ulp relative over every one of the
// 2^23 values of u, next to u = 1 included (measured on gfx950 against float64), so e needs no
// series expansion near 1: a 13-term series there had cost 9% of a sampled batch-64 block.
__device__ __forceinline__ float gumbel_from_word(uint32_t x) {
  const float e = -fast_log2(((float)(x >> 9) + 0.5f) * 0x1p-23f) * kLn2;
  return -fast_log2(e) * kLn2;
}

__device__ __forceinline__ uint4 philox_row(const Sampler& sm, int b, int j, int v) {
  return philox4x32_10(make_uint4((uint32_t)v >> 2, (uint32_t)j, sm.b0 + (uint32_t)b, 0u), sm.seed_lo, sm.seed_hi);
}

__device__ __forceinline__ float gumbel_at(const Sampler& sm, int b, int j, int v) {
  const uint4 x4 = philox_row(sm, b, j, v);
  const int w4 = v & 3;
  return gumbel_from_word(w4 == 0 ? x4.x : (w4 == 1 ? x4.y : (w4 == 2 ? x4.z : x4.w)));
}

}  // namespace dls
