// Persistent, weight-stationary DeLS-Spec block drafting (Algorithm 1 decoding loop with
// the App. A RNN head) for bf16 heads prepared by dls_prepare_head.
//
// One workgroup per CU stays resident for the whole block.  Each workgroup owns a
// contiguous range of 16-row vocabulary tiles of W_vocab: the first tiles live in the
// AGPRs of its four waves (fed straight into v_mfma_f32_16x16x32_bf16 as the B operand),
// the rest in LDS.  The first NG = H/16 workgroups ("GRU workgroups") also own 16 hidden
// units each (their W_hh rows in LDS) and r/NG rows of W_rank.  Per draft position j:
//
//   GRU wgs  merge the argmax keys of position j-1 -> tokens u_j (all sequences); with
//            several M tiles workgroup NG + b merges sequence b and they read its token
//            gi = T[u_j] (folded table) + gh (from the previous step) -> gates -> h_{j+1}
//            of the owned units, published
//            rho_i = SiLU(W_rank h_{j+1}) for the owned rank rows (MFMA), published; then
//            gh = W_hh h_{j+1} for the next position from the same staged h (MFMA)
//   all wgs  S = W_vocab rho on the owned tiles (MFMA), fused with the long logits
//            (prefetched into LDS while waiting), online LSEs and top-2; one packed argmax
//            key per (sequence, workgroup) published first, the LSE partials after it
//
// fp32 activations enter the bf16 matrix cores as two bf16 halves (hi + lo), split once
// when they are staged into LDS.
//
// Cross-workgroup data moves through device-coherent 64-bit words that carry a tag
// (epoch of the call, position); a consumer spins on the word itself until the tag
// matches, so each hand-off costs one propagation, with no counters and no cache
// flushes.  Batches of more than four sequences (the wide form) load two such words per
// 16-byte load and hand h over as 32-bit words (24-bit value, 8-bit position tag) in two
// sets that alternate between calls.  Every wait is bounded; on expiry an error word is
// set and all waves leave.
#pragma once
#include <atomic>

#include "dels_internal.hpp"

namespace dls {

namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;

constexpr int kT = 256;          // threads per workgroup (one wave per SIMD)
constexpr int kOps = 56;         // MFMA B operands of 16 bytes per lane held in AGPRs (224 of
                                 // the 256; the rest take the accumulators)
constexpr long kMaxSpins = 1L << 22;
constexpr int kInflight = 8;     // hand-off loads a thread issues before checking any of them (one
                                 // 64-bit word each for narrow batches, 16 bytes for wide ones)
constexpr int kStageK = 256;     // K chunk of staged hand-off values (16 slots x 256 floats in LDS)
constexpr int kStatWords = 9;    // tagged words of one published partial
constexpr int kRhoCopies = 1;    // copies of the published rank vector (more copies measured slower: their stores sit on the critical path)

__device__ __forceinline__ uint64_t ld64(const uint64_t* p) {
  return __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st64(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t ld32(const uint32_t* p) {
  return __hip_atomic_load(const_cast<uint32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st32(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Test builds (DLS_STRESS_DELAYS defined; libdels_stress.so): a pseudo-random pause of 0 to
// about 10 us before each hand-off publish, different for every call, workgroup, wave, position
// and publish site, so that the hand-offs run under other interleavings; the drafted tokens and
// statistics must not change.  The pause count is wave-uniform, and every pause is far inside the
// bounded waits.  In the product library the hook is empty.
#ifdef DLS_STRESS_DELAYS
__device__ __forceinline__ void stress_pause(uint32_t epoch, int w, int j, int site) {
  const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  uint32_t h = epoch * 0x9E3779B1u ^ (uint32_t)w * 0x85EBCA77u ^ (uint32_t)(j + 1) * 0xC2B2AE3Du ^
               (uint32_t)site * 0x27D4EB2Fu ^ wave * 0x165667B1u;
  h ^= h >> 15;
  h *= 0x2C1B3C6Du;
  h ^= h >> 12;
  h *= 0x297A2D39u;
  h ^= h >> 15;
  const int rounds = (h & 3u) == 0u ? (int)((h >> 8) & 3u) : 0;   // about one publish in five pauses
  for (int i = 0; i < rounds; ++i) __builtin_amdgcn_s_sleep(127);   // 127 x 64 cycles each
}
#define DLS_STRESS(ep, w, j, site) stress_pause((ep), (w), (j), (site))
#else
#define DLS_STRESS(ep, w, j, site) ((void)0)
#endif

__device__ __forceinline__ void stf(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ldf(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Agent-coherent 16-byte loads (the cache policy of ld64: sc1) through a buffer resource over
// `bytes` bytes from `base`; offsets past the end read as zeros.  A 16-byte aligned load lies
// within one cache line: each of its two 64-bit words is read whole, as by ld64.  Polling loops
// put a compiler barrier (poll_fence) before each round, so that every round loads again.
// The base and size are wave-uniform wherever this is used; readfirstlane tells the compiler so,
// which keeps the descriptor in scalar registers (a descriptor it takes for per-lane would turn
// every load into a loop over the lanes' distinct descriptors).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t coherent_rsrc(const void* base, uint32_t bytes) {
  const uint64_t b = (uint64_t)(uintptr_t)base;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)b), hi = __builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
  void* ub = (void*)(uintptr_t)(((uint64_t)hi << 32) | lo);
  return __builtin_amdgcn_make_buffer_rsrc(ub, (short)0, (int)__builtin_amdgcn_readfirstlane(bytes), 0x00020000);
}
__device__ __forceinline__ u32x4 ld128(__amdgpu_buffer_rsrc_t rs, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 16);   // sc1
}
__device__ __forceinline__ void poll_fence() { asm volatile("" ::: "memory"); }
// the thread index, recomputed where it is used: values derived from it are not hoisted out of
// the drafting loop and kept live across it (the wide kernels have no registers to spare)
__device__ __forceinline__ int local_tid() {
  int t = (int)threadIdx.x;
  asm volatile("" : "+v"(t));
  return t;
}
// all earlier vector-memory operations of this wave have completed
__device__ __forceinline__ void vm_wait() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

__device__ __forceinline__ uint64_t tagged(float v, uint32_t tag) {
  return ((uint64_t)tag << 32) | __float_as_uint(v);
}

// wait until (word >> 32) == tag; false after the spin budget or when another wave failed
__device__ __forceinline__ bool wait_tag(const uint64_t* p, uint32_t tag, uint32_t* err, uint64_t& v) {
  v = ld64(p);
  if ((uint32_t)(v >> 32) == tag) return true;
  for (long s = 1;; ++s) {
    __builtin_amdgcn_s_sleep(2);
    v = ld64(p);
    if ((uint32_t)(v >> 32) == tag) return true;
    if ((s & 63) == 0 && ld32(err)) return false;
    if (s > kMaxSpins) {
      st32(err, kErrStalled);
      return false;
    }
  }
}
// keys carry an 8-bit position tag in their low byte
__device__ __forceinline__ bool wait_key(const uint64_t* p, uint32_t tag8, uint32_t* err, uint64_t& v) {
  v = ld64(p);
  if ((uint32_t)(v & 0xffu) == tag8) return true;
  for (long s = 1;; ++s) {
    __builtin_amdgcn_s_sleep(2);
    v = ld64(p);
    if ((uint32_t)(v & 0xffu) == tag8) return true;
    if ((s & 63) == 0 && ld32(err)) return false;
    if (s > kMaxSpins) {
      st32(err, kErrStalled);
      return false;
    }
  }
}

// argmax key: orderable fused value | (2^24 - 1 - index) | position tag
__device__ __forceinline__ uint64_t make_key(float t1, int i1, uint32_t tag8) {
  t1 += 0.0f;   // -0 -> +0, so that equal values compare equal
  const uint32_t u = __float_as_uint(t1);
  const uint32_t o = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  const uint32_t ix = (i1 == 0x7fffffff) ? 0u : (0xffffffu - (uint32_t)i1);
  return ((uint64_t)o << 32) | ((uint64_t)ix << 8) | tag8;
}
__device__ __forceinline__ float key_value(uint64_t k) {
  const uint32_t o = (uint32_t)(k >> 32);
  return __uint_as_float((o & 0x80000000u) ? (o & 0x7fffffffu) : ~o);
}
__device__ __forceinline__ int key_index(uint64_t k, int V) {
  const int i = (int)(0xffffffu - (uint32_t)((k >> 8) & 0xffffffu));
  return i < V ? i : 0;   // no finite value anywhere: the first index
}
__device__ __forceinline__ uint64_t key_max(uint64_t a, uint64_t b) { return (a >> 8) >= (b >> 8) ? a : b; }

// fp32 -> bf16 hi + bf16 lo (v = hi + lo to ~2^-17 relative)
__device__ __forceinline__ uint32_t bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}
__device__ __forceinline__ void split_pair(float x0, float x1, uint32_t& hi, uint32_t& lo) {
  const uint32_t h0 = bf16_rne(x0), h1 = bf16_rne(x1);
  const uint32_t l0 = bf16_rne(x0 - __uint_as_float(h0 << 16));
  const uint32_t l1 = bf16_rne(x1 - __uint_as_float(h1 << 16));
  hi = h0 | (h1 << 16);
  lo = l0 | (l1 << 16);
}
__device__ __forceinline__ void split8(const float* x, uint4& hi, uint4& lo) {
  split_pair(x[0], x[1], hi.x, lo.x);
  split_pair(x[2], x[3], hi.y, lo.y);
  split_pair(x[4], x[5], hi.z, lo.z);
  split_pair(x[6], x[7], hi.w, lo.w);
}

__device__ __forceinline__ bf16x8_t as_bf(uint4 v) {
  union { uint4 u; bf16x8_t b; } c;
  c.u = v;
  return c.b;
}
__device__ __forceinline__ f32x4_t mfma_vv(uint4 a, uint4 b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf(a), as_bf(b), c, 0, 0, 0);
}
// B operand resident in AGPRs (the matrix core reads it from there; the compiler keeps
// track of the MFMA result hazards)
__device__ __forceinline__ f32x4_t mfma_va(uint4 a, u32x4 b_agpr, f32x4_t c) {
  union { u32x4 u; bf16x8_t b; } bb;
  bb.u = b_agpr;
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf(a), bb.b, c, 0, 0, 0);
}
// A operand resident in AGPRs (a W_vocab tile as the rows of the product)
__device__ __forceinline__ f32x4_t mfma_av(u32x4 a_agpr, uint4 b, f32x4_t c) {
  union { u32x4 u; bf16x8_t b; } aa;
  aa.u = a_agpr;
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(aa.b, as_bf(b), c, 0, 0, 0);
}
__device__ __forceinline__ u32x4 in_agpr(u32x4 r) {
  asm volatile("; weights -> agpr" : "=a"(r) : "0"(r));
  return r;
}

__device__ __forceinline__ float sigm(float x) { return 1.0f / (1.0f + __expf(-x)); }

// Online log-sum-exp with one exponential per element: exp(-|x - m|) serves both the case of
// a new maximum (rescale the sum) and of a smaller value (add it).  -inf adds nothing.
__device__ __forceinline__ void lse_push(Lse& a, float x) {
  const float d = x - a.m;
  const float e = fast_exp2(-fabsf(d) * kLog2e);
  const bool up = d > 0.f;
  const float s_new = up ? __builtin_fmaf(a.s, e, 1.0f) : a.s + e;
  a.s = (x == -INFINITY) ? a.s : s_new;
  a.m = up ? x : a.m;
}

// lse_push for a running maximum that starts finite (kFinMin instead of -inf): no test of the
// value is needed, since x = -inf gives d = -inf, a zero term and no new maximum.  Such a
// state is empty while s == 0 (a push sets s >= 1); fin_to_empty restores the -inf form.
__device__ __forceinline__ void lse_push_fin(Lse& a, float x) {
  const float d = x - a.m;
  const float e = fast_exp2(-fabsf(d) * kLog2e);
  const bool up = d > 0.f;
  a.s = up ? __builtin_fmaf(a.s, e, 1.0f) : a.s + e;
  a.m = up ? x : a.m;
}
// four values at once into a finite-start state: one new maximum, one rescale of the sum and
// one exponential per value (values of -inf add nothing)
__device__ __forceinline__ void lse_push4_fin(Lse& a, const float (&x)[4]) {
  const float mn = fmaxf(a.m, fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])));
  const float ml = mn * kLog2e;
  float s = a.s * fast_exp2((a.m - mn) * kLog2e);   // exactly 1 while the maximum stays
#pragma unroll
  for (int i = 0; i < 4; ++i) s += fast_exp2(__builtin_fmaf(x[i], kLog2e, -ml));
  a.m = mn;
  a.s = s;
}

// value of the lane N places further along in the same row of 16 lanes (DPP row rotate)
template <int N>
__device__ __forceinline__ float row_ror(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x120 + N, 0xf, 0xf, false));
}
template <int N>
__device__ __forceinline__ int row_ror_i(int v) {
  return __builtin_amdgcn_update_dpp(0, v, 0x120 + N, 0xf, 0xf, false);
}
template <int N>
__device__ __forceinline__ uint64_t row_ror_u64(uint64_t v) {
  const uint32_t lo = (uint32_t)row_ror_i<N>((int)(uint32_t)v), hi = (uint32_t)row_ror_i<N>((int)(uint32_t)(v >> 32));
  return ((uint64_t)hi << 32) | lo;
}
// largest key over the 16 lanes of a row (every lane of the row gets it)
__device__ __forceinline__ uint64_t row_key_max(uint64_t k) {
  k = key_max(k, row_ror_u64<8>(k));
  k = key_max(k, row_ror_u64<4>(k));
  k = key_max(k, row_ror_u64<2>(k));
  k = key_max(k, row_ror_u64<1>(k));
  return k;
}
// The value of lane l ^ 16 (or l ^ 32) through the permlane swaps of gfx950: VALU operations,
// where a shuffle across rows would take an LDS round trip (ds_bpermute).  With both operands
// equal, each swap returns this lane's value and its partner's, in an order that depends on
// the lane; a symmetric operation can take the pair as it is.
__device__ __forceinline__ uint32_t lane_xor16(uint32_t v) {
  const auto q = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  return (threadIdx.x & 16) ? q[0] : q[1];
}
__device__ __forceinline__ uint32_t lane_xor32(uint32_t v) {
  const auto q = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return (threadIdx.x & 32) ? q[0] : q[1];
}
// largest key over the wave (every lane gets it)
__device__ __forceinline__ uint64_t wave_key_max(uint64_t k) {
  k = row_key_max(k);
  {
    const auto lo = __builtin_amdgcn_permlane16_swap((uint32_t)k, (uint32_t)k, false, false);
    const auto hi = __builtin_amdgcn_permlane16_swap((uint32_t)(k >> 32), (uint32_t)(k >> 32), false, false);
    k = key_max(((uint64_t)hi[0] << 32) | lo[0], ((uint64_t)hi[1] << 32) | lo[1]);
  }
  {
    const auto lo = __builtin_amdgcn_permlane32_swap((uint32_t)k, (uint32_t)k, false, false);
    const auto hi = __builtin_amdgcn_permlane32_swap((uint32_t)(k >> 32), (uint32_t)(k >> 32), false, false);
    k = key_max(((uint64_t)hi[0] << 32) | lo[0], ((uint64_t)hi[1] << 32) | lo[1]);
  }
  return k;
}

// largest key over the lanes l, l ^ 16, l ^ 32 and l ^ 48 (every one of them gets it)
__device__ __forceinline__ uint64_t groups_key_max(uint64_t k) {
  k = key_max(k, ((uint64_t)lane_xor16((uint32_t)(k >> 32)) << 32) | lane_xor16((uint32_t)k));
  k = key_max(k, ((uint64_t)lane_xor32((uint32_t)(k >> 32)) << 32) | lane_xor32((uint32_t)k));
  return k;
}
// lane permutation for allred_partial over the lanes l, l ^ 16, l ^ 32 and l ^ 48
struct GroupXor {
  template <typename F>
  __device__ __forceinline__ void each(F f) const {
    f(16);
    f(32);
  }
  __device__ __forceinline__ int i(int v, int m) const {
    return (int)(m == 16 ? lane_xor16((uint32_t)v) : lane_xor32((uint32_t)v));
  }
  __device__ __forceinline__ float operator()(float v, int m) const { return __int_as_float(i(__float_as_int(v), m)); }
};

// lane permutations for allred_partial: DPP rotations within each row of 16 lanes, then
// (FULL) xor shuffles across the four rows
template <bool FULL>
struct RowRor {
  template <typename F>
  __device__ __forceinline__ void each(F f) const {
    f(8); f(4); f(2); f(1);
    if (FULL) { f(16); f(32); }
  }
  __device__ __forceinline__ int i(int v, int m) const {
    switch (m) {
      case 8: return row_ror_i<8>(v);
      case 4: return row_ror_i<4>(v);
      case 2: return row_ror_i<2>(v);
      case 1: return row_ror_i<1>(v);
      case 16: return (int)lane_xor16((uint32_t)v);
      default: return (int)lane_xor32((uint32_t)v);
    }
  }
  __device__ __forceinline__ float operator()(float v, int m) const { return __int_as_float(i(__float_as_int(v), m)); }
};

}  // namespace

// ------------------------------------------------------------------------------------------
// tile ownership (shared with the host)
// ------------------------------------------------------------------------------------------
// cap_a: vocabulary tiles a workgroup holds in AGPRs; gcap (<= cap_a): tiles of a GRU workgroup
// when the tiles do not fit in the AGPRs of all workgroups (the rest go to the others, which
// hold the surplus in LDS)
__host__ __device__ inline void persist_tile_range(int w, int G, int NG, int NT, int cap_a, int gcap, int* t0,
                                                   int* n) {
  if (NT <= G * cap_a) {
    const int q = NT / G, rm = NT % G;
    *t0 = w * q + (w < rm ? w : rm);
    *n = q + (w < rm ? 1 : 0);
    return;
  }
  const int ga = NG * gcap;
  if (w < NG) {
    *t0 = w * gcap;
    *n = gcap;
    return;
  }
  const int rest = NT - ga, m = G - NG, i = w - NG;
  const int q = rest / m, rm = rest % m;
  *t0 = ga + i * q + (i < rm ? i : rm);
  *n = q + (i < rm ? 1 : 0);
}

namespace {

// Copy n 16-byte words from global memory into LDS, 8 loads in flight per thread (indices past
// the end re-read the last word, so that every load is unconditional).
// Eight loads per thread in flight, then eight stores.  Threads past the end copy the last
// element again (the same value to the same place) instead of branching: a store under a branch
// let the compiler sink each load into it and wait for each one in turn.
__device__ __forceinline__ void copy_to_lds(uint4* dst, const uint4* src, int n) {
  for (int base = 0; base < n; base += kT * 8) {
    u32x4 v[8];   // (a uint4 array here was kept in scratch memory)
#pragma unroll
    for (int m = 0; m < 8; ++m) {
      const int i = base + m * kT + (int)threadIdx.x;
      v[m] = *(const u32x4*)(src + (i < n ? i : n - 1));
    }
#pragma unroll
    for (int m = 0; m < 8; ++m) {
      const int i = base + m * kT + (int)threadIdx.x;
      *(u32x4*)(dst + (i < n ? i : n - 1)) = v[m];
    }
  }
}

// Operand planes: staged hand-off values as bf16 hi and lo halves, 16 slots x (K + 8) each
// (the 8-element pad spreads the slots' rows over the LDS banks).
constexpr int kPlane = 16 * (kStageK + 8);

// one staged value: its bf16 hi and lo halves (hi + lo = x to about 2^-17 relative)
__device__ __forceinline__ void put_split(uint16_t* hi, uint16_t* lo, int idx, uint32_t bits) {
  const float x = __uint_as_float(bits);
  const uint32_t h = bf16_rne(x);
  hi[idx] = (uint16_t)h;
  lo[idx] = (uint16_t)bf16_rne(x - __uint_as_float(h << 16));
}

// Stage rows x width tagged words (row stride `stride` words) into the operand planes at
// [row * pitch + c], one word per load and INF words per thread at a time: every thread
// re-reads only its words whose tag does not match yet, all of them in flight together, until
// none is left (or the spin budget runs out).  A consumer that arrives when the producers are
// about done pays one round trip per poll, and data that is already there costs one round trip
// per INF words a thread.  Used for narrow batches, where a round or two covers the hand-off
// and 8-byte loads spread over all threads arrive sooner than half as many 16-byte loads.
template <int INF>
__device__ __forceinline__ bool stage_poll_words(const uint64_t* src, int rows, int width, size_t stride, uint32_t tag,
                                           uint16_t* hi, uint16_t* lo, int pitch, uint32_t* err) {
  const int q = kT / width, rm = kT % width;
  int row = (int)threadIdx.x / width, col = (int)threadIdx.x % width;
  bool ok = true;
  for (int base = 0; base < rows * width; base += kT * INF) {
    int rc[INF];   // row << 16 | column (rows <= 16, columns < 2^16)
    uint32_t pend = 0;
#pragma unroll
    for (int m = 0; m < INF; ++m) {
      rc[m] = (row << 16) | col;
      if (row < rows) pend |= 1u << m;
      col += rm;
      row += q;
      if (col >= width) {
        col -= width;
        ++row;
      }
    }
    for (long sp = 0; pend; ++sp) {
      uint64_t v[INF];
#pragma unroll
      for (int m = 0; m < INF; ++m)
        v[m] = (pend >> m) & 1u ? ld64(src + (size_t)(rc[m] >> 16) * stride + (rc[m] & 0xffff)) : 0ull;
#pragma unroll
      for (int m = 0; m < INF; ++m) {
        if (((pend >> m) & 1u) && (uint32_t)(v[m] >> 32) == tag) {
          put_split(hi, lo, (rc[m] >> 16) * pitch + (rc[m] & 0xffff), (uint32_t)v[m]);
          pend &= ~(1u << m);
        }
      }
      if (!pend) break;
      __builtin_amdgcn_s_sleep(2);
      if ((sp & 63) == 63 && ld32(err)) {
        ok = false;
        break;
      }
      if (sp > kMaxSpins) {
        st32(err, kErrStalled);
        ok = false;
        break;
      }
    }
  }
  return ok;
}

// two staged values (an even index): their bf16 hi and lo halves
__device__ __forceinline__ void put_split2(uint16_t* hi, uint16_t* lo, int idx, uint32_t b0, uint32_t b1) {
  uint32_t h, l;
  split_pair(__uint_as_float(b0), __uint_as_float(b1), h, l);
  *(uint32_t*)(hi + idx) = h;
  *(uint32_t*)(lo + idx) = l;
}

// As stage_poll_words, two adjacent words per 16-byte load (width, stride and the word offset
// of src even, src 16-byte aligned), INF loads per thread at a time: data that is already there
// costs one round trip per 2 INF words a thread.  Used for wide batches, whose hand-offs are
// 16 to 64 times larger.
template <int INF>
__device__ __forceinline__ bool stage_poll_pairs(const uint64_t* src, int rows, int width, int stride, uint32_t tag,
                                           uint16_t* hi, uint16_t* lo, int pitch, uint32_t* err) {
  const int wp = width >> 1;   // pairs per row
  const __amdgpu_buffer_rsrc_t rs = coherent_rsrc(src, (uint32_t)(((size_t)(rows - 1) * stride + width) * 8));
  const int q = kT / wp, rm = kT % wp;
  const int t = local_tid();
  int row = t / wp, col = t % wp;
  bool ok = true;
  for (int base = 0; base < rows * wp; base += kT * INF) {
    int rc[INF];   // row << 16 | pair column (rows <= 16, columns < 2^16)
    uint32_t pend = 0;
#pragma unroll
    for (int m = 0; m < INF; ++m) {
      rc[m] = (row << 16) | col;
      if (row < rows) pend |= 1u << m;
      col += rm;
      row += q;
      if (col >= wp) {
        col -= wp;
        ++row;
      }
    }
    for (long sp = 0; pend; ++sp) {
      poll_fence();
      u32x4 v[INF];
#pragma unroll
      for (int m = 0; m < INF; ++m)
        v[m] = (pend >> m) & 1u ? ld128(rs, (uint32_t)(((rc[m] >> 16) * stride + 2 * (rc[m] & 0xffff)) * 8))
                                : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
      for (int m = 0; m < INF; ++m) {
        if (((pend >> m) & 1u) && v[m].y == tag && v[m].w == tag) {
          put_split2(hi, lo, (rc[m] >> 16) * pitch + 2 * (rc[m] & 0xffff), v[m].x, v[m].z);
          pend &= ~(1u << m);
        }
      }
      if (!pend) break;
      __builtin_amdgcn_s_sleep(2);
      if ((sp & 63) == 63 && ld32(err)) {
        ok = false;
        break;
      }
      if (sp > kMaxSpins) {
        st32(err, kErrStalled);
        ok = false;
        break;
      }
    }
  }
  return ok;
}

// Wide batches hand h over as 32-bit words: the value rounded to 24 bits (sign, exponent, 15
// mantissa bits) over an 8-bit position tag, so a 16-byte load carries four values.  The bf16
// hi + lo split of such a value is exact (hi its top 16 bits, lo the remaining 8 significant
// bits), as precise as the split of a full fp32 value into two round-to-nearest bf16 halves.
__device__ __forceinline__ uint32_t pack_h24(float v, uint32_t tag8) {
  const uint32_t u = __float_as_uint(v);
  return ((u + 0x7fu + ((u >> 8) & 1u)) & 0xffffff00u) | tag8;
}
__device__ __forceinline__ void split_h24(uint32_t wd, uint32_t& hi, uint32_t& lo) {
  const uint32_t x = wd & 0xffffff00u, h = wd & 0xffff0000u;
  hi = h >> 16;
  lo = __float_as_uint(__uint_as_float(x) - __uint_as_float(h)) >> 16;
}
// Eight consecutive 24-bit words (two loaded quads) as an MFMA operand: their bf16 hi and lo halves
__device__ __forceinline__ void split_h24x8(const u32x4& q0, const u32x4& q1, uint4& hi, uint4& lo) {
  uint32_t h[8], l[8];
  split_h24(q0.x, h[0], l[0]);
  split_h24(q0.y, h[1], l[1]);
  split_h24(q0.z, h[2], l[2]);
  split_h24(q0.w, h[3], l[3]);
  split_h24(q1.x, h[4], l[4]);
  split_h24(q1.y, h[5], l[5]);
  split_h24(q1.z, h[6], l[6]);
  split_h24(q1.w, h[7], l[7]);
  hi = make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16));
  lo = make_uint4(l[0] | (l[1] << 16), l[2] | (l[3] << 16), l[4] | (l[5] << 16), l[6] | (l[7] << 16));
}
__device__ __forceinline__ bool quad_tagged(const u32x4& q, uint32_t tag8) {
  return ((q.x & 0xffu) == tag8) & ((q.y & 0xffu) == tag8) & ((q.z & 0xffu) == tag8) & ((q.w & 0xffu) == tag8);
}
// Wait until one (ALL = false) or every (ALL = true) of np producers has published (one lane
// per producer, polling one word of each).  Narrow batches stage after the first producer: the
// rest of their small hand-off follows within a fraction of a microsecond.  A wide batch of one
// M tile waits for the last one, so that the 16-byte loads of its larger hand-off find every
// word there in one round instead of polling again for the late producers.
template <bool ALL>
__device__ __forceinline__ void wait_producers(const uint64_t* src0, size_t pstride, int np, uint32_t tag,
                                               uint32_t* err) {
  if (threadIdx.x < 64) {
    const int l = (int)threadIdx.x;
    bool done = l >= np;   // a published word keeps its tag until this workgroup moves on
    for (long sp = 0;; ++sp) {
      const bool seen = !done && (uint32_t)(ld64(src0 + (size_t)l * pstride) >> 32) == tag;
      done |= seen;
      if (ALL ? __all(done) : __any(seen)) break;
      __builtin_amdgcn_s_sleep(4);
      if ((sp & 63) == 63 && ld32(err)) break;
      if (sp > kMaxSpins) {
        st32(err, kErrStalled);
        break;
      }
    }
  }
  __syncthreads();
}

// Workgroup barrier that also tells whether any thread failed.  A failure is final (all waves
// leave), so the LDS flag is set once and never cleared.
// The flag lives in LDS and is accessed through an LDS-qualified pointer: through a generic
// pointer the volatile access becomes a flat load, whose wait also waits for every store the
// wave still has in flight (the hand-off stores take a microsecond to complete).
typedef __attribute__((address_space(3))) volatile int lds_flag_t;
__device__ __forceinline__ bool fail_barrier(bool failed, lds_flag_t* s_fail) {
  if (failed) *s_fail = 1;
  __syncthreads();
  return *s_fail != 0;
}

// A operand (16 slots x 32 k) at column k of the planes: lane (slot n16, group g4) takes
// k + 8 g4 .. +7 of its slot.  Lanes of slots >= nb read slot 0 instead: an MFMA output row
// depends on its own A row only, and the rows of empty slots are never used.
__device__ __forceinline__ void plane_operand(const uint16_t* hi, const uint16_t* lo, int pitch, int nb, int n16,
                                              int g4, int k, uint4& ahi, uint4& alo) {
  const int o = (n16 < nb ? n16 : 0) * pitch + k + 8 * g4;
  ahi = *(const uint4*)(hi + o);
  alo = *(const uint4*)(lo + o);
}

// NARROW: at most 4 sequences (one M tile whose useful rows all sit in lanes 0..15)
// MARKOV: the Markov head of App. A, rho_j = E_M[u_j]: no GRU workgroups and no hand-off
//         but the argmax keys (and, with several M tiles, the merged tokens); every workgroup
//         gets the tokens and reads the E_M row itself
// the value of lane l ^ k within its quad (k = 1, 2, 3): a DPP quad permutation
__device__ __forceinline__ uint32_t quad_xor(uint32_t v, int k) {
  switch (k) {
    case 1: return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xf, 0xf, false);   // [1, 0, 3, 2]
    case 2: return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xf, 0xf, false);   // [2, 3, 0, 1]
    default: return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x1B, 0xf, 0xf, false);  // [3, 2, 1, 0]
  }
}
// Gumbel noise g[i] of sequences bq0 + i (i < n <= 4) at this lane's vocabulary entry v, for
// temperature sampling.  The four lanes of a quad hold v = 4k .. 4k + 3 (one Philox block
// counter): each runs the block of one sequence, bq0 + (lane & 3), and the quad exchanges
// the words, so a lane runs one block instead of four.  Every lane of the wave must be active.
__device__ __forceinline__ void gumbel_quad(const Sampler& sm, int bq0, int j, int v, int n, float g[4]) {
  const int q = threadIdx.x & 3;
  const uint4 x4 = philox_row(sm, bq0 + q, j, v);
  uint32_t r[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    // round k: lane q ^ k of the quad needs word q ^ k of this lane's block
    const int want = q ^ k;
    const uint32_t send = want == 0 ? x4.x : (want == 1 ? x4.y : (want == 2 ? x4.z : x4.w));
    r[k] = k == 0 ? send : quad_xor(send, k);
  }
  // r[k] is word q (entry v) of the block of sequence bq0 + (q ^ k)
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    g[i] = 0.f;
    if (i < n) {
      const int k = q ^ i;
      g[i] = gumbel_from_word(k == 0 ? r[0] : (k == 1 ? r[1] : (k == 2 ? r[2] : r[3])));
    }
  }
}

template <int KK, typename LT, bool PRIOR, bool NARROW, bool MARKOV, bool SAMPLE>
__global__ __launch_bounds__(kT, 1) void k_draft_persistent(PersistArgs a) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  constexpr int TPW = kOps / KK;   // AGPR tiles per wave
  constexpr int kInf = kInflight;   // hand-off loads in flight per thread
  // At most 4 sequences use at most 4 of an MFMA's 16 A rows, so the hi and lo halves of rho
  // share one operand (rows 0..3 hi, 4..7 lo): one MFMA chain per tile instead of two.  The
  // two halves' products are summed when the tile is folded, in the same order as before.
  constexpr bool PACK = NARROW && !MARKOV;
  const int w = blockIdx.x, G = gridDim.x, tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, n16 = lane & 15, g4 = lane >> 4;
  const int V = a.V, H = a.H, r = a.r, batch = a.batch, Bk = a.B, rpg = a.rpg;
  const bool gru = w < a.NG;
  const int KKH = H / 32;
  uint32_t* err = a.hdr + 1;
  const uint32_t epoch_full = ld32(a.hdr);
  const uint32_t epoch = epoch_full & 0xffffffu;
  const int set = (int)(epoch & 1u);
  const int Gp = (G + 1) & ~1;                         // key row stride: even, for 16-byte loads of pairs
  const size_t kstride = (size_t)kMaxBatch * Gp;      // one (set, parity) plane of keys

  int t0, nt;
  persist_tile_range(w, G, a.NG, a.NT, a.cap_a, a.gcap, &t0, &nt);
  const int na = nt < a.cap_a ? nt : a.cap_a;
  const int nl = nt - na;
  const int v_base = 16 * t0;
  const int nrows = 16 * nt;
  const int mtiles = (batch + 15) / 16;
  const int ll_slots = batch < 16 ? batch : 16;

  // ---- LDS carve-up (offsets identical to the host's size computation)
  char* p = smem;
  uint4* s_wtiles = (uint4*)p;                      // nl tiles x KK x 64 (non-GRU wgs)
  uint4* s_whh = (uint4*)p;                         // 3 x KKH x 64 (GRU wgs)
  bf16_t* s_wrank = (bf16_t*)(p + (size_t)3 * KKH * 1024);   // rpg x H (GRU wgs)
  p += a.lds_region_a;
  LT* s_ll = (LT*)p;                                // ll_slots x rows_max long logits
  p += ((size_t)ll_slots * a.rows_max * sizeof(LT) + 15) & ~(size_t)15;
  float* s_prior = (float*)p;                       // rows_max
  p += (size_t)a.rows_max * 4 * (PRIOR ? 1 : 0);
  // operand planes; at other times the gh partials (12 x 64 x f32x4) and the gathered gi (16 x 48)
  uint16_t* s_hi = (uint16_t*)p;
  uint16_t* s_lo = s_hi + kPlane;
  f32x4_t* s_red = (f32x4_t*)p;
  float* s_gi = (float*)p;
  p += (size_t)2 * kPlane * 2;
  f32x4_t* s_rred = (f32x4_t*)p;                    // rank partials [wave][g4][rpg]
  p += (size_t)16 * rpg * 16;
  float* s_gh = (float*)p;                          // per M tile: 16 slots x 48 (W_hh h for the next step)
  p += (size_t)mtiles * 16 * 48 * 4;
  Partial* s_part = (Partial*)p;                    // 4 waves x 16 slots
  p += (size_t)4 * 16 * sizeof(Partial);
  uint64_t* s_wkey = (uint64_t*)p;                  // 4 waves x 16 slots; the merge's per-sequence maxima
  uint64_t* s_best = s_wkey;
  p += (size_t)kMaxBatch * 8;
  int* s_tok = (int*)p;                             // kMaxBatch
  p += (size_t)kMaxBatch * 4;
  float* s_gate = (float*)p;                        // 16 slots: the M tile's adaptive-fusion gates
  p += (size_t)16 * 4;
  lds_flag_t* s_fail = (lds_flag_t*)p;              // sticky failure flag

  // A failed call leaves outputs that cannot pass for a draft: token -1 at every position
  // unless the drafting itself had finished (workgroup 0 is the only writer of tokens), and
  // NaN in every statistics row (row q is merged, and on failure overwritten, by workgroup
  // q mod G alone).
  bool tokens_done = false;
  auto bail = [&]() {
    if (w == 0 && !tokens_done)
      for (int i = tid; i < batch * Bk; i += kT) a.out_tokens[i] = -1;
    if (a.out_stats && tid < 6)
      for (int q = w; q < batch * Bk; q += G) ((float*)(a.out_stats + q))[tid] = __builtin_nanf("");
  };
  // Entry check, evaluated once the resident weights are in flight: an earlier failure on this
  // workspace (the error word is sticky until the workspace is zero-filled), or a prepared
  // buffer that does not belong to this head (its header holds the shapes and tensor pointers
  // dls_prepare_head was given; the host has checked its size, so the loads below stay inside
  // it either way), ends the call.
  PreparedHeader ph;
  uint32_t err_at_entry = 0u;
  if (tid == 0) {
    ph = *a.prep;
    err_at_entry = ld32(err);
  }

  // ---- clear this workgroup's key slots of the other set (read by the next call)
  for (int i = tid; i < 2 * kMaxBatch; i += kT) {
    const int par = i / kMaxBatch, b = i % kMaxBatch;
    st64(a.keys + (size_t)(1 - set) * 2 * kstride + par * kstride + (size_t)b * Gp + w, 0ull);
  }
  // ---- clear this workgroup's share of the other set of the wide h words, in every call (a
  // narrow or Markov call too): the next call then starts from zeros, whatever earlier calls
  // wrote, which the 8-bit tags of those words need
  {
    uint64_t* hz = (uint64_t*)(a.h32 + (size_t)(1 - set) * kH32Set);
    const size_t n64 = kH32Set / 2, per = (n64 + G - 1) / G;
    for (size_t i = (size_t)w * per + tid; i < (size_t)(w + 1) * per && i < n64; i += kT) st64(hz + i, 0ull);
  }

  // ---- resident weights: every load of the wave's tiles is issued before any is moved into
  // its AGPRs (moved one by one, each move waited for its own load before the next was issued)
  u32x4 wr[TPW * KK];
#pragma unroll
  for (int q = 0; q < TPW; ++q) {
    const int lt = wave * TPW + q;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (lt < na) v = a.wv[((size_t)(t0 + lt) * KK + kk) * 64 + lane];
      wr[q * KK + kk] = u32x4{v.x, v.y, v.z, v.w};
    }
  }
#pragma unroll
  for (int i = 0; i < TPW * KK; ++i) wr[i] = in_agpr(wr[i]);
  if (gru) {
    copy_to_lds(s_whh, a.whh + (size_t)w * 3 * KKH * 64, 3 * KKH * 64);
    // the owned rank rows are rows w rpg ... w rpg + rpg - 1 of W_rank, one contiguous block
    copy_to_lds((uint4*)s_wrank, (const uint4*)(a.w_rank + (size_t)w * rpg * H), rpg * H / 8);
  } else {
    copy_to_lds(s_wtiles, a.wv + ((size_t)(t0 + na) * KK) * 64, nl * KK * 64);
  }
  if (PRIOR) {   // four loads per thread in flight; past the end a thread copies the last row again
    for (int base = 0; base < nrows; base += 4 * kT) {
      float pv[4];
      int ix[4];
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        const int i = base + m * kT + tid;
        ix[m] = i < nrows ? i : nrows - 1;
        pv[m] = v_base + ix[m] < V ? a.prior[v_base + ix[m]] : 0.f;
      }
#pragma unroll
      for (int m = 0; m < 4; ++m) s_prior[ix[m]] = pv[m];
    }
  }
  if (tid == 0) {
    const PreparedHeader& ex = a.expect;
    const bool mismatch = ph.magic != ex.magic || ph.V != ex.V || ph.d != ex.d || ph.H != ex.H || ph.r != ex.r ||
                          ph.emb != ex.emb || ph.w_ih != ex.w_ih || ph.w_hh != ex.w_hh || ph.w_vocab != ex.w_vocab;
    if (mismatch) st32(err, kErrPrepared);
    *s_fail = (mismatch || err_at_entry != 0u) ? 1 : 0;
  }
  __syncthreads();
  if (*s_fail) {
    bail();
    return;
  }

  const LT* L = (const LT*)a.L;
  const float wl = a.wl;

  // Tokens of position jm (the argmax keys of all workgroups) into s_tok; workgroup 0 also
  // writes the drafted tokens.  Narrow batches: thread t loads the keys of workgroup t and
  // max-reduces them through LDS atomics.  Wide batches: wave v merges sequences v, v + 4, ...;
  // each lane loads the key pairs (workgroups 2c, 2c + 1) c = lane and lane + 64 of a sequence
  // with 16-byte loads, four sequences per round; each row of 16 lanes reduces them with DPP and
  // its first lane max-reduces the result into LDS (four atomics per sequence, where 256 would
  // serialise and cross-row shuffles cost LDS round trips).  Workgroup-uniform result.
  auto merge_position = [&](int jm) -> bool {
    const uint32_t tag8 = (uint32_t)(jm + 1);
    const uint64_t* kp = a.keys + (size_t)set * 2 * kstride + (size_t)(jm & 1) * kstride;
    bool ok = true;
    if (NARROW) {
      for (int b = tid; b < batch; b += kT) s_best[b] = 0ull;
      __syncthreads();
      if (tid < G) {
        uint64_t v[4];
#pragma unroll
        for (int m = 0; m < 4; ++m) v[m] = m < batch ? ld64(kp + (size_t)m * Gp + tid) : 0ull;
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          if (m < batch) {
            if ((uint32_t)(v[m] & 0xffu) != tag8) ok &= wait_key(kp + (size_t)m * Gp + tid, tag8, err, v[m]);
            atomicMax((unsigned long long*)&s_best[m], v[m]);
          }
        }
      }
    } else {
      for (int b = tid; b < batch; b += kT) s_best[b] = 0ull;
      __syncthreads();
      const __amdgpu_buffer_rsrc_t rs = coherent_rsrc(kp, (uint32_t)((size_t)batch * Gp * 8));
      constexpr int SPR = kInf / 2;   // sequences per round (two loads each)
      const int lane = local_tid() & 63;
      for (int b0 = wave; b0 < batch; b0 += 4 * SPR) {   // wave-uniform
        uint32_t pend = 0;
#pragma unroll
        for (int m = 0; m < kInf; ++m) {
          const int b = b0 + 4 * (m >> 1), c = lane + 64 * (m & 1);
          if (b < batch && 2 * c < G) pend |= 1u << m;
        }
        uint64_t best[SPR];
#pragma unroll
        for (int k = 0; k < SPR; ++k) best[k] = 0ull;
        for (long sp = 0; pend; ++sp) {
          poll_fence();
          u32x4 v[kInf];
#pragma unroll
          for (int m = 0; m < kInf; ++m) {
            const int b = b0 + 4 * (m >> 1), c = lane + 64 * (m & 1);
            v[m] = (pend >> m) & 1u ? ld128(rs, (uint32_t)(((size_t)b * Gp + 2 * c) * 8)) : u32x4{0u, 0u, 0u, 0u};
          }
#pragma unroll
          for (int m = 0; m < kInf; ++m) {
            if ((pend >> m) & 1u) {
              const int c = lane + 64 * (m & 1);
              const bool has1 = 2 * c + 1 < G;   // the pad column of an odd grid is never written
              if ((v[m].x & 0xffu) == tag8 && (!has1 || (v[m].z & 0xffu) == tag8)) {
                const uint64_t k0 = ((uint64_t)v[m].y << 32) | v[m].x;
                const uint64_t k1 = has1 ? ((uint64_t)v[m].w << 32) | v[m].z : 0ull;
                best[m >> 1] = key_max(best[m >> 1], key_max(k0, k1));
                pend &= ~(1u << m);
              }
            }
          }
          if (!pend) break;
          __builtin_amdgcn_s_sleep(2);
          if ((sp & 63) == 63 && ld32(err)) {
            ok = false;
            break;
          }
          if (sp > kMaxSpins) {
            st32(err, kErrStalled);
            ok = false;
            break;
          }
        }
#pragma unroll
        for (int k = 0; k < SPR; ++k) {
          const int b = b0 + 4 * k;
          if (b < batch) {   // wave-uniform
            const uint64_t kb = row_key_max(best[k]);
            if ((lane & 15) == 0) atomicMax((unsigned long long*)&s_best[b], kb);
          }
        }
      }
    }
    if (fail_barrier(!ok, s_fail)) return false;
    if (tid < batch) {
      const int tok = key_index(s_best[tid], V);
      s_tok[tid] = tok;
      if (w == 0) a.out_tokens[(size_t)tid * Bk + jm] = tok;
    }
    __syncthreads();
    return true;
  };

  // Batches of several M tiles delegate the merge: workgroup NG + b (the first non-GRU
  // workgroups, which wait for rho anyway) merges the keys of sequence b alone and publishes its
  // token as one tagged word; the workgroups that need the tokens (the GRU workgroups, or every
  // workgroup of the Markov head) read batch words instead of batch x G keys (128 KB at batch
  // 64), at the price of one more hand-off.  With one M tile the keys are few and the merging
  // workgroups would be the last to finish the position, so every reader merges for itself.
  // Needs G - NG >= batch.
  const bool delegate = !NARROW && mtiles > 1 && G - a.NG >= batch;
  const int merge_seq = delegate && w >= a.NG && w - a.NG < batch ? w - a.NG : -1;   // this workgroup's sequence
  auto merge_one = [&](int jm, int b) -> bool {
    const uint32_t tag8 = (uint32_t)(jm + 1);
    const uint64_t* kp = a.keys + (size_t)set * 2 * kstride + (size_t)(jm & 1) * kstride + (size_t)b * Gp;
    uint64_t k = 0ull;
    bool ok = true;
    if (tid < G) {
      k = ld64(kp + tid);
      if ((uint32_t)(k & 0xffu) != tag8) ok = wait_key(kp + tid, tag8, err, k);
    }
    k = wave_key_max(k);
    if ((tid & 63) == 0) s_wkey[tid >> 6] = k;
    if (fail_barrier(!ok, s_fail)) return false;
    if (tid == 0) {
      uint64_t m = s_wkey[0];
      for (int q = 1; q < 4; ++q) m = key_max(m, s_wkey[q]);
      DLS_STRESS(epoch, w, jm, 7);
      st64(a.tokw + (size_t)(jm & 1) * kMaxBatch + b,
           ((uint64_t)((epoch << 8) | tag8) << 32) | (uint32_t)key_index(m, V));
    }
    __syncthreads();   // s_wkey read
    return true;
  };
  // the tokens of position jm from the merging workgroups into s_tok (workgroup 0 also writes
  // the drafted tokens)
  auto fetch_tokens = [&](int jm) -> bool {
    const uint32_t tg = (epoch << 8) | (uint32_t)(jm + 1);
    bool ok = true;
    if (tid < batch) {
      const uint64_t* tp = a.tokw + (size_t)(jm & 1) * kMaxBatch + tid;
      uint64_t v = ld64(tp);
      if ((uint32_t)(v >> 32) != tg) ok = wait_tag(tp, tg, err, v);
      const int tok = (int)(uint32_t)v;
      s_tok[tid] = tok;
      if (w == 0) a.out_tokens[(size_t)tid * Bk + jm] = tok;
    }
    return !fail_barrier(!ok, s_fail);
  };
  auto tokens_of = [&](int jm) -> bool { return delegate ? fetch_tokens(jm) : merge_position(jm); };

  // Publish the row-statistics partial of this workgroup for position jp (slots of M tile mtp,
  // per-wave partials in s_part): merged over the waves by a butterfly over the lanes of wave
  // `by` (each lane loads one wave's partial of one slot), then nine tagged words per slot,
  // spread over the slot's four lanes (a wave's loads wait for its earlier stores, so the
  // stores go to a wave that loads nothing critical soon after).  The butterfly replaced three
  // merges in a row on 16 lanes: 3% off every block.
  auto publish_stats = [&](int jp, int mtp, int nbp, int by) {
    DLS_STRESS(epoch, w, jp, 5);
    if (wave == by) {   // lane 16 q + sl holds wave q's partial of slot sl; a butterfly merges them
      const int sl = lane & 15, q = lane >> 4;
      Partial T = s_part[q * 16 + sl];
      T = allred_partial(T, GroupXor{});
      if (sl < nbp) {
        const uint32_t stag = (epoch << 8) | (uint32_t)(jp + 1);
        uint64_t* sp = a.stats + (((size_t)jp * batch + mtp * 16 + sl) * G + w) * kStatWords;
        // the four lanes of the slot hold the same merged partial; lane q stores words q, q + 4, q + 8
        const float w0 = q == 0 ? T.L.m : q == 1 ? T.L.s : q == 2 ? T.S.m : T.S.s;
        const float w1 = q == 0 ? T.F.m : q == 1 ? T.F.s : q == 2 ? T.t1 : T.t2;
        st64(sp + q, tagged(w0, stag));
        st64(sp + 4 + q, tagged(w1, stag));
        if (q == 0) st64(sp + 8, tagged(__int_as_float(T.i1), stag));
      }
    }
  };
  // GRU workgroups with a single M tile hand their statistics of position j over during
  // the gather of position j + 1: right after the argmax key they are on the critical path
  // to the next merge.  -1: nothing pending.
  int pending_stats = -1;
  // wide batches: the state of the owned units of this lane's slots (the gate pairs of its
  // wave), kept in registers across positions: the published 24-bit copy feeds only the
  // matrix products
  float hown[4] = {0.f, 0.f, 0.f, 0.f};

  for (int j = 0; j < Bk; ++j) {
    const uint32_t tag = (epoch << 8) | (uint32_t)(j + 1);
    const uint32_t tag8 = (uint32_t)(j + 1);
    const int par = j & 1;
    const float al = a.al_j[j], be = a.be_j[j];   // this position's fusion weights
    const bool long_only = a.literal && j == 0;
    const int hs = a.literal ? j - 1 : j;          // head step index (the first one starts from h = 0)

    // the merging workgroups of the RNN head: the keys of their sequence at the previous position
    if (!MARKOV && merge_seq >= 0 && j > 0) {
      if (!merge_one(j - 1, merge_seq)) {
        bail();
        return;
      }
    }

    // ======================= GRU and rank (GRU workgroups) =======================
    if (!MARKOV && gru && !long_only) {
      const uint32_t tag_prev = (epoch << 8) | (uint32_t)j;   // h published at position j-1
      const uint64_t* hprev = a.hbuf + (size_t)((j - 1) & 1) * batch * H;
      uint64_t* hnew = a.hbuf + (size_t)par * batch * H;
      // wide batches: the h words of this position, in a.hrep replicas (every GRU workgroup reads
      // all of h; the replicas spread the readers over the memory channels)
      const size_t hrep_stride = (size_t)batch * H;
      uint32_t* h32new = NARROW ? nullptr : a.h32 + (size_t)set * kH32Set + (size_t)par * a.hrep * hrep_stride;
      if (j > 0) {
        if (!tokens_of(j - 1)) {
          bail();
          return;
        }
      } else {
        for (int b = tid; b < batch; b += kT) {
          const int u = a.last[b];
          s_tok[b] = (unsigned)u < (unsigned)V ? u : 0;   // out-of-range input reads as 0
        }
        __syncthreads();
      }
      // gates of the owned units: gi = T[u] (folded input projection) for all sequences at once,
      // 16-byte loads; gh from the previous step.  The (M tile, slot group i) pairs are spread
      // over the waves, mtiles pairs each: wave v takes pairs v * mtiles + k, pair p being M tile
      // p / 4 and slots 4 g4 + p % 4 of it (one M tile: wave v computes slot group v).
      {
        const int npw = mtiles;   // pairs per wave (mtiles <= 4)
        uint64_t hv[4];   // narrow: the owned units' previous state, in flight together with the gather
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int pp = wave * npw + k, mt = pp >> 2, slot = 4 * g4 + (pp & 3);
          hv[k] = (NARROW && hs > 0 && k < npw && mt * 16 + slot < batch && slot < 16)
                      ? ld64(hprev + (size_t)(mt * 16 + slot) * H + 16 * w + n16)
                      : 0ull;
        }
        // with statistics of the previous position pending (one M tile), wave 3 publishes them
        // while the other waves gather (the gather is latency-bound; wave 3 loads nothing until
        // the rank stage, so its stores delay no load of its own)
        const int gthreads = pending_stats >= 0 ? 192 : kT;
        const int ngi = batch * 12;   // (sequence, gate, 4 units) loads
        if (tid < gthreads) {
          for (int i0 = local_tid(); i0 < ngi; i0 += 4 * gthreads) {
            f32x4_t x[4];
#pragma unroll
            for (int m = 0; m < 4; ++m) {
              const int i = i0 + m * gthreads;
              const int slot = i / 12, q = (i % 12) >> 2, u4 = i & 3;
              x[m] = i < ngi ? *(const f32x4_t*)(a.T + (size_t)s_tok[slot] * 3 * H + q * H + 16 * w + 4 * u4)
                             : f32x4_t{0.f, 0.f, 0.f, 0.f};
            }
#pragma unroll
            for (int m = 0; m < 4; ++m) {
              const int i = i0 + m * gthreads;
              if (i < ngi) *(f32x4_t*)(s_gi + (i / 12) * 48 + ((i % 12) >> 2) * 16 + 4 * (i & 3)) = x[m];
            }
          }
        } else {
          publish_stats(pending_stats, 0, batch, 3);
        }
        pending_stats = -1;
        __syncthreads();
        bool ok = true;
        float hn[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int pp = wave * npw + k, mt = pp >> 2, slot = 4 * g4 + (pp & 3), bb = mt * 16 + slot;
          if (k < npw && bb < batch && slot < 16) {
            float hp = 0.f, ghr = 0.f, ghz = 0.f, ghn = 0.f;
            if (hs > 0) {
              if (NARROW) {
                if ((uint32_t)(hv[k] >> 32) != tag_prev)
                  ok &= wait_tag(hprev + (size_t)bb * H + 16 * w + n16, tag_prev, err, hv[k]);
                hp = __uint_as_float((uint32_t)hv[k]);
              } else {
                hp = hown[k];
              }
              const float* gh = s_gh + mt * 16 * 48;
              ghr = gh[slot * 48 + n16];
              ghz = gh[slot * 48 + 16 + n16];
              ghn = gh[slot * 48 + 32 + n16];
            }
            const float* gi = s_gi + bb * 48;
            const float rg = sigm(gi[n16] + ghr);
            const float zg = sigm(gi[16 + n16] + ghz);
            const float ng = tanhf_(gi[32 + n16] + rg * ghn);
            hn[k] = (1.f - zg) * ng + zg * hp;
          }
        }
        // the stores after all the values: a store ahead of the arithmetic of the next slot
        // would make the wave wait for its completion
        DLS_STRESS(epoch, w, j, 1);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int pp = wave * npw + k, mt = pp >> 2, slot = 4 * g4 + (pp & 3), bb = mt * 16 + slot;
          if (k < npw && bb < batch && slot < 16) {
            if (NARROW) {
              st64(hnew + (size_t)bb * H + 16 * w + n16, tagged(hn[k], tag));
            } else {
              hown[k] = hn[k];
              const uint32_t word = pack_h24(hn[k], tag8);
              for (int rep = 0; rep < a.hrep; ++rep) st32(h32new + rep * hrep_stride + (size_t)bb * H + 16 * w + n16, word);
            }
          }
        }
        if (fail_barrier(!ok, s_fail)) {
          bail();
          return;
        }
      }
      // rho_i = SiLU(W_rank h_{j+1}) for the owned rank rows and W_hh h_{j+1} for the next
      // position, from h_{j+1} of all GRU workgroups.
      //
      // Wide batches: the A operands come straight from the 32-bit hand-off words, with no LDS
      // staging: lane (slot n16, group g4) loads columns 32 kk + 8 g4 .. +7 of its slot (two
      // 16-byte loads, split into bf16 hi and lo halves in registers).  The M tiles are taken in
      // order and the four waves split K (wave v: kk = v mod 4), so the rho of M tile m is out
      // (and the other workgroups fold it) while M tile m + 1 is still being multiplied; the
      // partial sums of the four waves are added in LDS in wave order.
      if (!NARROW) {
        const bool with_gh = j + 1 < Bk;
        constexpr int NB = 8;   // K steps per round of loads and wave (two 16-byte loads each)
        bool ok = true;
        for (int mt = 0; mt < mtiles; ++mt) {
          const int nb = batch - mt * 16 < 16 ? batch - mt * 16 : 16;
          f32x4_t racc = f32x4_t{0.f, 0.f, 0.f, 0.f}, g0 = racc, g1 = racc, g2 = racc;
          const __amdgpu_buffer_rsrc_t rs =
              coherent_rsrc(h32new + (size_t)(w % a.hrep) * hrep_stride + (size_t)mt * 16 * H, (uint32_t)(nb * H * 4));
          const bool have = n16 < nb;   // lanes of slots past the batch multiply zeros
          const uint32_t rowoff = (uint32_t)((have ? n16 : 0) * H + 8 * g4);
          for (int c0 = 0; ok && wave + c0 * 4 < KKH; c0 += NB) {
            u32x4 q[2 * NB];
            uint32_t pend = 0;
#pragma unroll
            for (int t = 0; t < NB; ++t) {
              q[2 * t] = q[2 * t + 1] = u32x4{0u, 0u, 0u, 0u};
              if (have && wave + (c0 + t) * 4 < KKH) pend |= 3u << (2 * t);
            }
            for (long sp = 0; pend; ++sp) {
              poll_fence();
#pragma unroll
              for (int m = 0; m < 2 * NB; ++m)
                if ((pend >> m) & 1u)
                  q[m] = ld128(rs, (rowoff + 32u * (uint32_t)(wave + (c0 + m / 2) * 4) + 4u * (m & 1)) * 4u);
#pragma unroll
              for (int m = 0; m < 2 * NB; ++m)
                if (((pend >> m) & 1u) && quad_tagged(q[m], tag8)) pend &= ~(1u << m);
              if (!pend) break;
              __builtin_amdgcn_s_sleep(2);
              if ((sp & 63) == 63 && ld32(err)) {
                ok = false;
                break;
              }
              if (sp > kMaxSpins) {
                st32(err, kErrStalled);
                ok = false;
                break;
              }
            }
            if (!ok) break;
#pragma unroll
            for (int t = 0; t < NB; ++t) {
              const int kk = wave + (c0 + t) * 4;
              if (kk < KKH) {   // wave-uniform
                uint4 ahi, alo;
                split_h24x8(q[2 * t], q[2 * t + 1], ahi, alo);
                const uint4 bw = n16 < rpg ? *(const uint4*)(s_wrank + (size_t)n16 * H + 32 * kk + 8 * g4)
                                           : make_uint4(0, 0, 0, 0);
                racc = mfma_vv(alo, bw, mfma_vv(ahi, bw, racc));
                if (with_gh) {
                  const uint4 b0 = s_whh[(0 * KKH + kk) * 64 + lane];
                  const uint4 b1 = s_whh[(1 * KKH + kk) * 64 + lane];
                  const uint4 b2 = s_whh[(2 * KKH + kk) * 64 + lane];
                  g0 = mfma_vv(alo, b0, mfma_vv(ahi, b0, g0));
                  g1 = mfma_vv(alo, b1, mfma_vv(ahi, b1, g1));
                  g2 = mfma_vv(alo, b2, mfma_vv(ahi, b2, g2));
                }
              }
            }
          }
          // the four waves' partial sums, added in wave order by wave 0 (the planes are free
          // here: the vocabulary phase stages rho into them only after the barrier that ends
          // this M tile loop)
          if (mt) __syncthreads();   // wave 0 is done reading the previous M tile's partials
          s_red[(wave * 4 + 0) * 64 + lane] = racc;
          s_red[(wave * 4 + 1) * 64 + lane] = g0;
          s_red[(wave * 4 + 2) * 64 + lane] = g1;
          s_red[(wave * 4 + 3) * 64 + lane] = g2;
          if (fail_barrier(!ok, s_fail)) {
            bail();
            return;
          }
          if (wave == 0) {
            for (int k = 1; k < 4; ++k) {
              racc += s_red[(k * 4 + 0) * 64 + lane];
              g0 += s_red[(k * 4 + 1) * 64 + lane];
              g1 += s_red[(k * 4 + 2) * 64 + lane];
              g2 += s_red[(k * 4 + 3) * 64 + lane];
            }
            DLS_STRESS(epoch, w, j, 2);
            if (n16 < rpg) {
#pragma unroll
              for (int i = 0; i < 4; ++i) {
                const int slot = 4 * g4 + i;
                if (slot < nb) {
                  const uint64_t word = tagged(siluf_(racc[i]), tag);
                  for (int c = 0; c < kRhoCopies; ++c)
                    st64(a.rbuf + ((size_t)c * 2 + par) * batch * r + (size_t)(mt * 16 + slot) * r + w * rpg + n16,
                         word);
                }
              }
            }
            if (with_gh) {
              float* gh = s_gh + mt * 16 * 48;
#pragma unroll
              for (int i = 0; i < 4; ++i) {
                gh[(4 * g4 + i) * 48 + 0 * 16 + n16] = g0[i];
                gh[(4 * g4 + i) * 48 + 1 * 16 + n16] = g1[i];
                gh[(4 * g4 + i) * 48 + 2 * 16 + n16] = g2[i];
              }
            }
          }
        }
        __syncthreads();   // s_red read, gh written: the planes and s_gh are free for what follows
      }
      for (int mt = 0; NARROW && mt < mtiles; ++mt) {
        const int nb = batch - mt * 16 < 16 ? batch - mt * 16 : 16;
        const int HC = nb * (H + 8) <= kPlane ? H : kStageK;
        const int pitch = HC + 8;
        const uint64_t* hsrc = hnew + (size_t)mt * 16 * H;
        bool ok = true;
        f32x4_t racc = f32x4_t{0.f, 0.f, 0.f, 0.f};
        // W_hh h_{j+1} accumulates here too: with several K chunks (wide batches) each staged
        // chunk serves both products, instead of being staged again after rho is out
        const bool chunked = HC < H;
        const bool with_gh = j + 1 < Bk;
        f32x4_t g0 = f32x4_t{0.f, 0.f, 0.f, 0.f}, g1 = g0, g2 = g0;   // gates r, z, n
        auto gh_chunk = [&](int k0) __attribute__((always_inline)) {
          for (int kk = wave; kk < HC / 32; kk += 4) {
            uint4 ahi, alo;
            plane_operand(s_hi, s_lo, pitch, nb, n16, g4, 32 * kk, ahi, alo);
            const uint4 b0 = s_whh[(0 * KKH + k0 / 32 + kk) * 64 + lane];
            const uint4 b1 = s_whh[(1 * KKH + k0 / 32 + kk) * 64 + lane];
            const uint4 b2 = s_whh[(2 * KKH + k0 / 32 + kk) * 64 + lane];
            g0 = mfma_vv(alo, b0, mfma_vv(ahi, b0, g0));
            g1 = mfma_vv(alo, b1, mfma_vv(ahi, b1, g1));
            g2 = mfma_vv(alo, b2, mfma_vv(ahi, b2, g2));
          }
        };
        // the owned rank rows and, with several chunks, W_hh h of the chunk staged at column k0
        auto chunk_products = [&](int k0) __attribute__((always_inline)) {
          for (int kk = wave; kk < HC / 32; kk += 4) {
            uint4 ahi, alo;
            plane_operand(s_hi, s_lo, pitch, nb, n16, g4, 32 * kk, ahi, alo);
            const uint4 bw = n16 < rpg ? *(const uint4*)(s_wrank + (size_t)n16 * H + k0 + 32 * kk + 8 * g4)
                                       : make_uint4(0, 0, 0, 0);
            racc = mfma_vv(ahi, bw, racc);
            racc = mfma_vv(alo, bw, racc);
          }
          if (chunked && with_gh) gh_chunk(k0);
        };
        // the other GRU workgroups publish h at about the same time: poll the words directly
        for (int k0 = 0; k0 < H; k0 += HC) {
          if (k0) __syncthreads();
          ok &= stage_poll_words<kInf>(hsrc + k0, nb, HC, H, tag, s_hi, s_lo, pitch, err);
          __syncthreads();
          chunk_products(k0);
        }
        if (n16 < rpg) s_rred[(wave * 4 + g4) * rpg + n16] = racc;
        if (fail_barrier(!ok, s_fail)) {
          bail();
          return;
        }
        DLS_STRESS(epoch, w, j, 3);
        if (wave == 0 && n16 < rpg) {
          f32x4_t sm = s_rred[g4 * rpg + n16];
          for (int q = 1; q < 4; ++q) sm += s_rred[(q * 4 + g4) * rpg + n16];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int slot = 4 * g4 + i;
            if (slot < nb) {
              const uint64_t word = tagged(siluf_(sm[i]), tag);
              for (int c = 0; c < kRhoCopies; ++c)
                st64(a.rbuf + ((size_t)c * 2 + par) * batch * r + (size_t)(mt * 16 + slot) * r + w * rpg + n16, word);
            }
          }
        }
        if (with_gh) {
          if (!chunked) gh_chunk(0);   // one chunk: after rho is out, from the same staged h
          __syncthreads();   // planes read: their space takes the partial sums
          s_red[(wave * 3 + 0) * 64 + lane] = g0;
          s_red[(wave * 3 + 1) * 64 + lane] = g1;
          s_red[(wave * 3 + 2) * 64 + lane] = g2;
          __syncthreads();
          if (wave == 0) {
            float* gh = s_gh + mt * 16 * 48;
            for (int q = 0; q < 3; ++q) {
              f32x4_t sm = s_red[q * 64 + lane];
              for (int k = 1; k < 4; ++k) sm += s_red[(k * 3 + q) * 64 + lane];
#pragma unroll
              for (int i = 0; i < 4; ++i) gh[(4 * g4 + i) * 48 + q * 16 + n16] = sm[i];
            }
          }
        }
        if (fail_barrier(!ok, s_fail)) {
          bail();
          return;
        }
      }
    }

    // ======================= Markov head: the previous token (all workgroups) =======================
    if (MARKOV && !long_only) {
      if (j > 0) {
        if ((merge_seq >= 0 && !merge_one(j - 1, merge_seq)) || !tokens_of(j - 1)) {
          bail();
          return;
        }
      } else {
        for (int b = tid; b < batch; b += kT) {
          const int u = a.last[b];
          s_tok[b] = (unsigned)u < (unsigned)V ? u : 0;   // out-of-range input reads as 0
        }
        __syncthreads();
      }
    }

    // ======================= vocabulary head + fused combine (all workgroups) =======================
    for (int mt = 0; mt < mtiles; ++mt) {
      const int nb = batch - mt * 16 < 16 ? batch - mt * 16 : 16;
      // the slots' gates (1 without adaptive fusion), read by the folds after the staging barrier
      if (tid < 16) s_gate[tid] = (a.unc && tid < nb) ? a.unc[(size_t)(mt * 16 + tid) * Bk + j].gate : 1.f;
      // long logits of the owned rows (independent of rho: in flight while rho is awaited).
      // Wide batches: 16-byte loads over [slot][row] flattened, eight per thread in flight, so
      // that 16 slots cost a round trip or two rather than one each
      constexpr int EPI = 16 / (int)sizeof(LT);   // long logits per 16-byte load
      if (NARROW) {
        for (int slot = 0; slot < nb; ++slot) {
          const LT* src = L + ((size_t)(mt * 16 + slot) * Bk + j) * V + v_base;
          LT* dst = s_ll + (size_t)slot * a.rows_max;
          for (int r0 = 0; r0 < nrows; r0 += 4 * kT) {
            LT x[4];
#pragma unroll
            for (int m = 0; m < 4; ++m) {
              const int row = r0 + m * kT + tid;
              x[m] = (row < nrows && v_base + row < V) ? src[row] : LT(0);
            }
#pragma unroll
            for (int m = 0; m < 4; ++m) {
              const int row = r0 + m * kT + tid;
              if (row < nrows) dst[row] = x[m];
            }
          }
        }
      } else if (nrows > 0 && V % EPI == 0) {
        // every 16-byte piece lies wholly inside or wholly past the vocabulary (V and v_base are
        // multiples of EPI); rows past V are stored as zeros and never folded
        const int ipr = nrows / EPI;                                   // pieces per slot
        const int nvalid = (V - v_base < nrows ? V - v_base : nrows) / EPI;
        const int n = nb * ipr;
        for (int i0 = local_tid(); i0 < n; i0 += 8 * kT) {
          uint4 x[8];
#pragma unroll
          for (int m = 0; m < 8; ++m) {
            const int i = i0 + m * kT;
            const int sl = i / ipr, c = i - sl * ipr;
            x[m] = (i < n && c < nvalid)
                       ? *(const uint4*)(L + ((size_t)(mt * 16 + sl) * Bk + j) * V + v_base + EPI * c)
                       : make_uint4(0u, 0u, 0u, 0u);
          }
#pragma unroll
          for (int m = 0; m < 8; ++m) {
            const int i = i0 + m * kT;
            const int sl = i / ipr, c = i - sl * ipr;
            if (i < n) *(uint4*)(s_ll + (size_t)sl * a.rows_max + EPI * c) = x[m];
          }
        }
      } else if (nrows > 0) {
        int sl = 0, rw = tid;   // this thread's first element of the group
        while (sl < nb && rw >= nrows) { rw -= nrows; ++sl; }
        while (sl < nb) {
          LT x[16];
          int s2 = sl, r2 = rw;
#pragma unroll
          for (int m = 0; m < 16; ++m) {
            x[m] = (s2 < nb && v_base + r2 < V) ? L[((size_t)(mt * 16 + s2) * Bk + j) * V + v_base + r2] : LT(0);
            r2 += kT;
            while (s2 < nb && r2 >= nrows) { r2 -= nrows; ++s2; }
          }
#pragma unroll
          for (int m = 0; m < 16; ++m) {
            if (sl < nb) s_ll[(size_t)sl * a.rows_max + rw] = x[m];
            rw += kT;
            while (sl < nb && rw >= nrows) { rw -= nrows; ++sl; }
          }
        }
      }
      // rho of the slots, staged as bf16 hi + lo planes, then held as the A operands
      uint4 ahi[KK], alo[KK];
      if (MARKOV && !long_only) {
        // rho = E_M[u]: bf16 values, exact in the hi plane (the lo half would be zero)
        for (int i = tid; i < nb * (r / 8); i += kT) {
          const int slot = i / (r / 8), c = i % (r / 8);
          *(uint4*)(s_hi + slot * (r + 8) + 8 * c) =
              *(const uint4*)(a.e_m + (size_t)s_tok[mt * 16 + slot] * r + 8 * c);
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
          ahi[kk] = *(const uint4*)(s_hi + (n16 < nb ? n16 : 0) * (r + 8) + 32 * kk + 8 * g4);
          alo[kk] = make_uint4(0, 0, 0, 0);
        }
      } else if (!long_only) {
        const uint64_t* rsrc = a.rbuf + ((size_t)(w % kRhoCopies) * 2 + par) * batch * r + (size_t)mt * 16 * r;
        // GRU workgroups come here after W_hh h, when rho is about complete: they poll the words
        // directly; the others wait (gently) for the first producer, or with one wide M tile for
        // all of them (several M tiles: the rho of the later tiles is out long before), then poll
        if (!gru) {
          if (!NARROW && mtiles == 1) wait_producers<true>(rsrc, (size_t)rpg, a.NG, tag, err);
          else wait_producers<false>(rsrc, (size_t)rpg, a.NG, tag, err);
        }
        const bool ok = NARROW ? stage_poll_words<kInf>(rsrc, nb, r, r, tag, s_hi, s_lo, r + 8, err)
                               : stage_poll_pairs<kInf>(rsrc, nb, r, r, tag, s_hi, s_lo, r + 8, err);
        if (fail_barrier(!ok, s_fail)) {
          bail();
          return;
        }
        if (PACK) {
          // rows 0..3 of the A operand carry the hi halves of slots 0..3, rows 4..7 the lo
          // halves (rows past the batch repeat slot 0, rows 8..15 are unused)
          const uint16_t* pl = (n16 & 4) ? s_lo : s_hi;
          const int row = (n16 & 3) < nb ? (n16 & 3) : 0;
#pragma unroll
          for (int kk = 0; kk < KK; ++kk) {
            ahi[kk] = *(const uint4*)(pl + row * (r + 8) + 32 * kk + 8 * g4);
            alo[kk] = make_uint4(0, 0, 0, 0);
          }
        } else {
#pragma unroll
          for (int kk = 0; kk < KK; ++kk) plane_operand(s_hi, s_lo, r + 8, nb, n16, g4, 32 * kk, ahi[kk], alo[kk]);
        }
      } else {
        __syncthreads();   // s_ll complete
      }
      // With at most 4 sequences every useful MFMA output sits in lanes 0..15 (rows = slots).
      // Such "narrow" tiles are stashed in LDS (the planes, free once the A operands are in
      // registers) and folded four tiles at a time, one tile per 16-lane group.
      //
      // Wider batches multiply the other way round: the resident W_vocab tile is the A operand
      // and rho the B operand (the two operands take the same per-lane layout), so a product
      // tile is vocabulary rows x slots and lane (slot n16, group g4) holds rows 4 g4 .. 4 g4 + 3
      // of its one slot.  Its running statistics are then those of a single slot, its four long
      // logits are one LDS read, its four entries share one Philox block, and the statistics
      // reduce over the slot's four lanes instead of over sixteen lanes for each of four slots.
      constexpr bool narrow = NARROW;
      float* s_stash = (float*)s_hi + wave * (PACK ? 512 : 256);   // narrow: [halves][4 tiles][slots][16 rows]
      if (narrow) __syncthreads();

      Partial P[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        P[i] = partial_empty();
        P[i].L.m = P[i].S.m = P[i].F.m = kFinMin;   // the fold's finite start
      }

      // keep the useful rows of a tile's result at stash position tq (narrow: slots < nb of
      // lane group 0)
      auto stash = [&](const f32x4_t& acc, int tq) {
        if (PACK) {   // lane group 0 holds the hi products, group 1 the lo products
          if (g4 < 2) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
              if (i < nb) s_stash[((g4 * 4 + tq) * 4 + i) * 16 + n16] = acc[i];
          }
        } else if (g4 == 0) {
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (i < nb) s_stash[(tq * 4 + i) * 16 + n16] = acc[i];
        }
      };
      // The fused value f of an entry: greedy decoding ranks f; sampling folds f / T into the
      // log-sum-exp and ranks f / T + g (Gumbel-max), g the entry's noise.
      // narrow: fold stashed tiles base + stride * tq (tq < ntile), lane group tq taking tile tq;
      // lanes without an entry (past the vocabulary, or a group past ntile) fold -inf
      auto fold_narrow = [&](int base, int stride, int ntile) {
        float gz[4] = {0.f, 0.f, 0.f, 0.f};
        if (SAMPLE) gumbel_quad(a.smp, mt * 16, j, v_base + 16 * (base + stride * g4) + n16, nb, gz);
        const int row = 16 * (base + stride * g4) + (local_tid() & 15);
        const int v = v_base + row;
        const bool ok = g4 < ntile && v < V;
        const int rowc = ok ? row : 0;   // an in-range LDS row for lanes without an entry
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if (i < nb) {   // uniform
            const float alx = long_only ? 0.f : al * s_gate[i], bex = long_only ? 0.f : be * s_gate[i];
            const float xr = to_f32(s_ll[i * a.rows_max + rowc]);
            const float x = ok ? xr : -INFINITY;
            const float sv = PACK ? s_stash[(g4 * 4 + i) * 16 + n16] + s_stash[((4 + g4) * 4 + i) * 16 + n16]
                                  : s_stash[(g4 * 4 + i) * 16 + n16];
            float f = __builtin_fmaf(alx, sv, weighted(wl, x));
            if (PRIOR) f = minus_weighted(f, bex, s_prior[rowc]);
            f = ok ? f : -INFINITY;
            lse_push_fin(P[i].S, ok && !long_only ? sv : -INFINITY);
            lse_push_fin(P[i].L, x);
            if (SAMPLE) f *= a.smp.inv_temp;
            lse_push_fin(P[i].F, f);
            top2_push(P[i], SAMPLE ? f + gz[i] : f, v);
          }
        }
      };

      // wide: fold a product tile (rows x slots) of tile lt.  Entries past the batch or the
      // vocabulary enter as -inf (no term, no maximum, no top-2 change) rather than behind
      // per-lane branches.
      auto fold4 = [&](const f32x4_t& acc, int lt) {
        const int lt16 = local_tid() & 63;
        const int sl_own = lt16 & 15;                      // the lane's slot
        const int row0 = 16 * lt + 4 * (lt16 >> 4);        // its first row in the owned range
        const int v0 = v_base + row0;
        const bool sok = sl_own < nb;
        const int sl = sok ? sl_own : 0;
        // the long-only first row of the literal schedule: no head term, no prior, no short sum
        const float gs = s_gate[sl];
        const float alx = long_only ? 0.f : al * gs, bex = long_only ? 0.f : be * gs;
        float x[4];
        if constexpr (sizeof(LT) == 2) {
          const uint2 raw = *(const uint2*)(s_ll + (size_t)sl * a.rows_max + row0);
          x[0] = bf16_lo(raw.x);
          x[1] = bf16_hi(raw.x);
          x[2] = bf16_lo(raw.y);
          x[3] = bf16_hi(raw.y);
        } else {
          const float4 raw = *(const float4*)(s_ll + (size_t)sl * a.rows_max + row0);
          x[0] = raw.x;
          x[1] = raw.y;
          x[2] = raw.z;
          x[3] = raw.w;
        }
        float4 pr = make_float4(0.f, 0.f, 0.f, 0.f);
        if (PRIOR) pr = *(const float4*)(s_prior + row0);
        float gz[4] = {0.f, 0.f, 0.f, 0.f};
        if (SAMPLE) {   // entries v0 .. v0 + 3 are the four words of one Philox block (v0 % 4 == 0)
          const uint4 x4 = philox_row(a.smp, mt * 16 + sl, j, v0);
          gz[0] = gumbel_from_word(x4.x);
          gz[1] = gumbel_from_word(x4.y);
          gz[2] = gumbel_from_word(x4.z);
          gz[3] = gumbel_from_word(x4.w);
        }
        const float prv[4] = {pr.x, pr.y, pr.z, pr.w};
        float xl[4], xs[4], f[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const bool ok = sok && v0 + i < V;
          xl[i] = ok ? x[i] : -INFINITY;
          xs[i] = (ok && !long_only) ? acc[i] : -INFINITY;
          float fi = __builtin_fmaf(alx, acc[i], weighted(wl, x[i]));
          if (PRIOR) fi = minus_weighted(fi, bex, prv[i]);
          fi = ok ? fi : -INFINITY;
          if (SAMPLE) fi *= a.smp.inv_temp;
          f[i] = fi;
        }
        lse_push4_fin(P[0].L, xl);
        lse_push4_fin(P[0].S, xs);
        lse_push4_fin(P[0].F, f);
#pragma unroll
        for (int i = 0; i < 4; ++i) top2_push(P[0], SAMPLE ? f[i] + gz[i] : f[i], v0 + i);
      };

      // AGPR-resident tiles of this wave, two at a time: four independent MFMA chains
      // (hi and lo halves of rho for each tile) keep the matrix pipe busy
#pragma unroll
      for (int q = 0; q < TPW; q += 2) {
        const int lt = wave * TPW + q;
        const bool two = q + 1 < TPW;   // constant once unrolled (TPW may be odd)
        const int q2 = two ? q + 1 : q;
        if (lt < na) {
          f32x4_t c0 = f32x4_t{0.f, 0.f, 0.f, 0.f}, c1 = c0, c2 = c0, c3 = c0;
          if (!long_only) {
#pragma unroll
            for (int kk = 0; kk < KK; ++kk) {
              if (narrow) {
                c0 = mfma_va(ahi[kk], wr[q * KK + kk], c0);
                if (!MARKOV && !PACK) c1 = mfma_va(alo[kk], wr[q * KK + kk], c1);
                if (two) {
                  c2 = mfma_va(ahi[kk], wr[q2 * KK + kk], c2);
                  if (!MARKOV && !PACK) c3 = mfma_va(alo[kk], wr[q2 * KK + kk], c3);
                }
              } else {
                c0 = mfma_av(wr[q * KK + kk], ahi[kk], c0);
                if (!MARKOV) c1 = mfma_av(wr[q * KK + kk], alo[kk], c1);
                if (two) {
                  c2 = mfma_av(wr[q2 * KK + kk], ahi[kk], c2);
                  if (!MARKOV) c3 = mfma_av(wr[q2 * KK + kk], alo[kk], c3);
                }
              }
            }
          }
          if (narrow) {
            stash(PACK ? c0 : c0 + c1, q % 4);
            if (two) stash(PACK ? c2 : c2 + c3, q % 4 + 1);
          } else {
            fold4(c0 + c1, lt);
            if (two && lt + 1 < na) fold4(c2 + c3, lt + 1);
          }
        }
        if (narrow && (q % 4 == 2 || q + 2 >= TPW)) {   // a group of four tiles (or the last) is stashed
          const int g0 = q - q % 4;
          const int cnt = (TPW - g0 < 4 ? TPW - g0 : 4);
          const int avail = na - (wave * TPW + g0);
          const int nf = avail < cnt ? (avail > 0 ? avail : 0) : cnt;
          fold_narrow(wave * TPW + g0, 1, nf);
        }
      }
      // LDS-resident tiles, round robin over the waves (narrow: four at a time)
      auto lds_tile = [&](int lq) -> f32x4_t {
        f32x4_t c0 = f32x4_t{0.f, 0.f, 0.f, 0.f}, c1 = c0;
        if (!long_only) {
#pragma unroll
          for (int kk = 0; kk < KK; ++kk) {
            const uint4 bw = s_wtiles[((size_t)lq * KK + kk) * 64 + lane];
            if (narrow) {
              c0 = mfma_vv(ahi[kk], bw, c0);
              if (!MARKOV && !PACK) c1 = mfma_vv(alo[kk], bw, c1);
            } else {
              c0 = mfma_vv(bw, ahi[kk], c0);
              if (!MARKOV) c1 = mfma_vv(bw, alo[kk], c1);
            }
          }
        }
        return PACK ? c0 : c0 + c1;
      };
      if (narrow) {
        for (int m0 = 0; wave + 4 * m0 < nl; m0 += 4) {
          int cnt = 0;
          for (int tq = 0; tq < 4; ++tq) {
            const int lq = wave + 4 * (m0 + tq);
            if (lq < nl) {
              stash(lds_tile(lq), tq);
              ++cnt;
            }
          }
          fold_narrow(na + wave + 4 * m0, 4, cnt);
        }
      } else {
        for (int lq = wave; lq < nl; lq += 4) fold4(lds_tile(lq), na + lq);
      }
      // argmax key of each slot: narrow, over the wave (slot i spread over it); wide, over the
      // slot's four lanes; then over the waves
      if (narrow) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if (i < nb) {
            const uint64_t k = wave_key_max(make_key(P[i].t1, P[i].i1, tag8));
            if (lane == 0) s_wkey[wave * 16 + i] = k;
          }
        }
      } else {
        const uint64_t k = groups_key_max(make_key(P[0].t1, P[0].i1, tag8));
        if (g4 == 0 && n16 < nb) s_wkey[wave * 16 + n16] = k;
      }
      __syncthreads();
      DLS_STRESS(epoch, w, j, 4);
      if (tid < nb) {
        uint64_t k = s_wkey[tid];
        for (int q = 1; q < 4; ++q) k = key_max(k, s_wkey[q * 16 + tid]);
        st64(a.keys + (size_t)set * 2 * kstride + par * kstride + (size_t)(mt * 16 + tid) * Gp + w, k);
      }
      // the full partials (LSEs, top-2) for the row statistics: off the critical path
      if (a.out_stats) {
        if (narrow) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            if (i < nb) {
              fin_to_empty(P[i].L);
              fin_to_empty(P[i].S);
              fin_to_empty(P[i].F);
              P[i] = allred_partial(P[i], RowRor<true>{});   // over the wave
              if (lane == 0) s_part[wave * 16 + i] = P[i];
            }
          }
        } else {
          fin_to_empty(P[0].L);
          fin_to_empty(P[0].S);
          fin_to_empty(P[0].F);
          P[0] = allred_partial(P[0], GroupXor{});   // over the slot's four lanes
          if (g4 == 0 && n16 < nb) s_part[wave * 16 + n16] = P[0];
        }
        if (gru && mtiles == 1 && j + 1 < Bk) {
          pending_stats = j;
        } else {
          __syncthreads();
          publish_stats(j, mt, nb, 0);
        }
      }
      __syncthreads();
    }
  }

  // ---- the last position's tokens (workgroup 0)
  if (merge_seq >= 0 && !merge_one(Bk - 1, merge_seq)) {
    bail();
    return;
  }
  if (w == 0) {
    if (!tokens_of(Bk - 1)) {
      bail();
      return;
    }
    tokens_done = true;
  }
  // ---- row statistics: row (b, j) is merged by workgroup (b * B + j) % G from the tagged partials,
  // up to four rows at a time, one per wave: lane l merges the partials of workgroups l, l + 64,
  // ... in that order, then the wave merges its lanes (a fixed butterfly)
  if (a.out_stats) {
    const int lane64 = local_tid() & 63;
    for (int q0 = w; q0 < batch * Bk; q0 += 4 * G) {
      const int q = q0 + wave * G;
      bool ok = true;
      if (q < batch * Bk) {   // wave-uniform
        const int b = q / Bk, jm = q % Bk;
        const uint32_t stag = (epoch << 8) | (uint32_t)(jm + 1);
        Partial P = partial_empty();
        for (int sl = lane64; sl < G; sl += 64) {
          const uint64_t* sp = a.stats + (((size_t)jm * batch + b) * G + sl) * kStatWords;
          uint64_t w9[kStatWords];
#pragma unroll
          for (int e = 0; e < kStatWords; ++e) w9[e] = ld64(sp + e);
          float q9[kStatWords];
#pragma unroll
          for (int e = 0; e < kStatWords; ++e) {
            if ((uint32_t)(w9[e] >> 32) != stag) ok &= wait_tag(sp + e, stag, err, w9[e]);
            q9[e] = __uint_as_float((uint32_t)w9[e]);
          }
          Partial Q;
          Q.L.m = q9[0]; Q.L.s = q9[1];
          Q.S.m = q9[2]; Q.S.s = q9[3];
          Q.F.m = q9[4]; Q.F.s = q9[5];
          Q.t1 = q9[6]; Q.t2 = q9[7];
          Q.i1 = __float_as_int(q9[8]);
          Q.pad = 0;
          P = sl == lane64 ? Q : partial_merge(P, Q);
        }
        P = allred_partial(P, WaveXor{});
        if (lane64 == 0 && ok) {
          int t;
          const int ti = P.i1 == 0x7fffffff ? 0 : P.i1;   // the token finalize_row decodes
          const float alr = a.unc ? a.al_j[jm] * a.unc[(size_t)b * Bk + jm].gate : a.al_j[jm];
          finalize_row(P, wl, alr, a.literal && jm == 0, &t, a.out_stats + (size_t)b * Bk + jm, nullptr,
                       SAMPLE ? gumbel_at(a.smp, b, jm, ti) : 0.f, a.smp.temp);
        }
      }
      if (fail_barrier(!ok, s_fail)) {
        bail();
        return;
      }
    }
  }
  if (w == 0 && tid == 0) {
    DLS_STRESS(epoch, w, Bk, 6);
    vm_wait();
    st32(a.hdr, epoch_full + 1u);
  }
}

template <int KK, typename LT, bool PRIOR, bool NARROW, bool MARKOV, bool SAMPLE>
hipError_t launch_k(const PersistArgs& pa, int G, size_t lds, hipStream_t st) {
  auto kern = k_draft_persistent<KK, LT, PRIOR, NARROW, MARKOV, SAMPLE>;
  // the dynamic LDS limit is raised to the maximum once per device (a per-call attribute
  // change costs microseconds of host time)
  static std::atomic<uint64_t> raised{0};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  const uint64_t bit = dev < 64 ? (uint64_t)1 << dev : 0;
  if (!bit || !(raised.load(std::memory_order_acquire) & bit)) {
    e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kMaxLds);
    if (e != hipSuccess) return e;
    raised.fetch_or(bit, std::memory_order_acq_rel);
  }
  (void)lds;
  PersistArgs copy = pa;
  void* args[] = {&copy};
  // A cooperative dispatch makes the runtime check co-residency and keep other kernels off the
  // device, at about 17 us per call; the caller may waive it (the grid never exceeds one
  // workgroup per CU, so on an otherwise idle device every workgroup is resident at once).
  if (pa.ordinary_launch) return hipLaunchKernel((const void*)kern, dim3(G), dim3(kT), args, lds, st);
  return hipLaunchCooperativeKernel((const void*)kern, dim3(G), dim3(kT), args, (unsigned)lds, st);
}

}  // namespace

// One rank size (KK = r / 32) and decoding mode: dispatch over the long-logit type, the
// prior, the batch width and the head kind.  Each (KK, SAMPLE) pair is instantiated in a
// translation unit of its own.
template <int KK, bool SAMPLE>
hipError_t launch_persistent_kk(const PersistArgs& pa, int G, size_t lds, dls_dtype long_dtype, hipStream_t st) {
  const bool narrow = pa.batch <= kNarrowBatch, prior = pa.prior != nullptr, markov = pa.e_m != nullptr;
#define DLS_PK(LT, P, N, M) \
  if (prior == P && narrow == N && markov == M) return launch_k<KK, LT, P, N, M, SAMPLE>(pa, G, lds, st);
#define DLS_PK_LT(LT)                                                                              \
  DLS_PK(LT, false, false, false) DLS_PK(LT, false, false, true) DLS_PK(LT, false, true, false)   \
  DLS_PK(LT, false, true, true) DLS_PK(LT, true, false, false) DLS_PK(LT, true, false, true)      \
  DLS_PK(LT, true, true, false) DLS_PK(LT, true, true, true)
  if (long_dtype == DLS_BF16) {
    DLS_PK_LT(bf16_t)
  } else {
    DLS_PK_LT(float)
  }
#undef DLS_PK_LT
#undef DLS_PK
  return hipErrorInvalidValue;
}

}  // namespace dls
