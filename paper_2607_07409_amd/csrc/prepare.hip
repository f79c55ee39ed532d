// One-time preparation of a bf16 RNN local head for the persistent drafting kernel.
//
// * Folded input projection.  The GRU input is always a row of the frozen target
//   embedding (App. A), so W_ih E[u] depends on the token only.  The table
//   T[u, :] = W_ih E[u]  ([V, 3H], float32, accumulated exactly from bf16 products by
//   MFMA) replaces the per-step input GEMV by a gather of 3H floats per sequence.
// * Vocabulary head in MFMA operand order: 16-row tiles, each split into K-chunks of 32,
//   each chunk stored as the 64 lanes x 16 bytes a v_mfma_f32_16x16x32_bf16 B operand
//   reads (lane l: row 16t + l%16, columns 32kk + 8(l/16) .. +7).
// * Recurrent weights W_hh in the same operand order, grouped by 16 hidden units and gate.
#include "dels_internal.hpp"

namespace dls {

namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 v) {
  union { uint4 u; bf16x8_t b; } c;
  c.u = v;
  return c.b;
}

// T[v, q] = sum_c E[v, c] * W_ih[q, c]; one wave computes a 32 x 32 block with 2 x 2 MFMA tiles.
__global__ __launch_bounds__(256) void k_fold_input(const bf16_t* __restrict__ emb, const bf16_t* __restrict__ w_ih,
                                                    int V, int d, int Q, float* __restrict__ T) {
  const int lane = threadIdx.x & 63;
  const int wave = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int qblocks = Q / 32;
  const int vb = wave / qblocks, qb = wave % qblocks;
  const int v0 = vb * 32, q0 = qb * 32;
  if (v0 >= V) return;
  const int n = lane & 15, g = lane >> 4;
  f32x4_t acc[2][2];
  for (int a = 0; a < 2; ++a)
    for (int b = 0; b < 2; ++b) acc[a][b] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  const uint4 zero = make_uint4(0, 0, 0, 0);
  for (int c0 = 0; c0 < d; c0 += 32) {
    const int c = c0 + 8 * g;
    uint4 av[2], bv[2];
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      const int v = v0 + 16 * a + n;
      av[a] = (v < V && c < d) ? *reinterpret_cast<const uint4*>(emb + (size_t)v * d + c) : zero;
      const int q = q0 + 16 * a + n;
      bv[a] = (c < d) ? *reinterpret_cast<const uint4*>(w_ih + (size_t)q * d + c) : zero;
    }
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int b = 0; b < 2; ++b)
        acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(av[a]), as_bf16x8(bv[b]), acc[a][b], 0, 0, 0);
  }
  // D layout: lane holds rows 4g + i of the M tile, column n of the N tile
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int v = v0 + 16 * a + 4 * g + i;
        if (v < V) T[(size_t)v * Q + q0 + 16 * b + n] = acc[a][b][i];
      }
}

// W_vocab [V, r] -> tiles [NT][KK][64 lanes] of 16 bytes
__global__ void k_pack_vocab(const bf16_t* __restrict__ w, int V, int r, int NT, uint4* __restrict__ out) {
  const int KK = r / 32;
  const size_t total = (size_t)NT * KK * 64;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (size_t)gridDim.x * blockDim.x) {
    const int l = (int)(i & 63);
    const size_t tk = i >> 6;
    const int kk = (int)(tk % KK);
    const int t = (int)(tk / KK);
    const int row = 16 * t + (l & 15);
    const int col = 32 * kk + 8 * (l >> 4);
    out[i] = row < V ? *reinterpret_cast<const uint4*>(w + (size_t)row * r + col) : make_uint4(0, 0, 0, 0);
  }
}

// W_hh [3H, H] -> [H/16 groups][3 gates][H/32 chunks][64 lanes] of 16 bytes
__global__ void k_pack_whh(const bf16_t* __restrict__ w, int H, uint4* __restrict__ out) {
  const int KK = H / 32;
  const size_t total = (size_t)(H / 16) * 3 * KK * 64;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (size_t)gridDim.x * blockDim.x) {
    const int l = (int)(i & 63);
    size_t x = i >> 6;
    const int kk = (int)(x % KK);
    x /= KK;
    const int q = (int)(x % 3);
    const int grp = (int)(x / 3);
    const int row = q * H + 16 * grp + (l & 15);
    const int col = 32 * kk + 8 * (l >> 4);
    out[i] = *reinterpret_cast<const uint4*>(w + (size_t)row * H + col);
  }
}

}  // namespace

PreparedLayout prepared_layout(const dls_local_head& h) {
  PreparedLayout L;
  L.NT = (h.V + 15) / 16;
  L.KK = h.r / 32;
  L.off_T = 256;
  size_t o = L.off_T + (size_t)h.V * 3 * h.H * sizeof(float);
  o = (o + 255) & ~(size_t)255;
  L.off_wv = o;
  o += (size_t)L.NT * L.KK * 1024;
  L.off_whh = o;
  o += (size_t)(h.H / 16) * 3 * (h.H / 32) * 1024;
  L.total = (o + 255) & ~(size_t)255;
  return L;
}

__global__ void k_write_header(PreparedHeader hdr, PreparedHeader* out) { *out = hdr; }

hipError_t launch_prepare(const dls_local_head& h, void* buf, hipStream_t st) {
  const PreparedLayout L = prepared_layout(h);
  char* base = (char*)buf;
  PreparedHeader hdr;
  hdr.magic = kPreparedMagic;
  hdr.V = h.V;
  hdr.d = h.d;
  hdr.H = h.H;
  hdr.r = h.r;
  hdr.emb = h.emb;
  hdr.w_ih = h.w_ih;
  hdr.w_hh = h.w_hh;
  hdr.w_vocab = h.w_vocab;
  k_write_header<<<1, 1, 0, st>>>(hdr, (PreparedHeader*)base);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const bool markov = h.kind == DLS_HEAD_MARKOV;   // no GRU: W_M only
  if (!markov) {
    const int Q = 3 * h.H;
    const int waves = ((h.V + 31) / 32) * (Q / 32);
    k_fold_input<<<(waves + 3) / 4, 256, 0, st>>>((const bf16_t*)h.emb, (const bf16_t*)h.w_ih, h.V, h.d, Q,
                                                 (float*)(base + L.off_T));
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  k_pack_vocab<<<2048, 256, 0, st>>>((const bf16_t*)h.w_vocab, h.V, h.r, L.NT, (uint4*)(base + L.off_wv));
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (!markov) k_pack_whh<<<512, 256, 0, st>>>((const bf16_t*)h.w_hh, h.H, (uint4*)(base + L.off_whh));
  return hipGetLastError();
}

}  // namespace dls
