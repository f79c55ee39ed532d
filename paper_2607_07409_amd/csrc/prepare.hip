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

// T[v, q] = sum_c E[v, c] * W_ih[q, c], an LDS-tiled MFMA GEMM.  A workgroup computes a 128 x 128
// block of T (four waves of 64 x 64, each 4 x 4 tiles of v_mfma_f32_16x16x32_bf16) over K steps
// of 64; the next step's pieces are loaded from HBM while the current one is multiplied from LDS.
// Rows past V, columns past Q and K past d read as zeros (d is a multiple of 8, so a 16-byte
// piece lies wholly inside or outside).  Workgroups are ordered so that each XCD runs all column
// blocks of a row block back to back (workgroup ids go round the 8 XCDs): every 128-row slice
// of E, the large operand, then comes from HBM once, later column blocks finding it in L2.
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
constexpr int kFM = 128, kFN = 128, kFK = 64;
constexpr int kFRow = kFK + 8;   // LDS row stride in bf16 (the pad spreads rows over the banks)

__device__ __forceinline__ bf16x8_t as_bf16x8(u32x4 v) {
  union { u32x4 u; bf16x8_t b; } c;
  c.u = v;
  return c.b;
}

__global__ __launch_bounds__(256) void k_fold_input(const bf16_t* __restrict__ emb, const bf16_t* __restrict__ w_ih,
                                                    int V, int d, int Q, int nvb, int nqb, float* __restrict__ T) {
  __shared__ __attribute__((aligned(16))) bf16_t sA[2][kFM * kFRow];
  __shared__ __attribute__((aligned(16))) bf16_t sB[2][kFN * kFRow];
  const int xcd = blockIdx.x & 7, k8 = blockIdx.x >> 3;
  const int vb = 8 * (k8 / nqb) + xcd, qb = k8 % nqb;
  if (vb >= nvb) return;
  const int v0 = vb * kFM, q0 = qb * kFN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;   // the wave's 64 x 64 sub-block
  const int n = lane & 15, g = lane >> 4;
  const u32x4 zero = {0u, 0u, 0u, 0u};

  // a K step of either tile is 128 rows x 8 pieces of 16 bytes; thread t moves pieces t + 256 m
  u32x4 ra[4], rb[4];
  auto load = [&](int c0) {
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      const int pc = tid + 256 * m, row = pc >> 3, c = c0 + 8 * (pc & 7);
      const int v = v0 + row, q = q0 + row;
      ra[m] = (v < V && c < d) ? *(const u32x4*)(emb + (size_t)v * d + c) : zero;
      rb[m] = (q < Q && c < d) ? *(const u32x4*)(w_ih + (size_t)q * d + c) : zero;
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      const int pc = tid + 256 * m, row = pc >> 3, kp = pc & 7;
      *(u32x4*)(sA[buf] + row * kFRow + 8 * kp) = ra[m];
      *(u32x4*)(sB[buf] + row * kFRow + 8 * kp) = rb[m];
    }
  };

  f32x4_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int jt = 0; jt < 4; ++jt) acc[i][jt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  const int nk = (d + kFK - 1) / kFK;
  load(0);
  store(0);
  __syncthreads();
  for (int ks = 0; ks < nk; ++ks) {
    const int cur = ks & 1;
    if (ks + 1 < nk) load((ks + 1) * kFK);
#pragma unroll
    for (int sub = 0; sub < kFK / 32; ++sub) {
      bf16x8_t av[4], bv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        av[i] = as_bf16x8(*(const u32x4*)(sA[cur] + (wm * 64 + 16 * i + n) * kFRow + 32 * sub + 8 * g));
        bv[i] = as_bf16x8(*(const u32x4*)(sB[cur] + (wn * 64 + 16 * i + n) * kFRow + 32 * sub + 8 * g));
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int jt = 0; jt < 4; ++jt) acc[i][jt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[i], bv[jt], acc[i][jt], 0, 0, 0);
    }
    // the other buffer was last read before the previous barrier
    if (ks + 1 < nk) store(cur ^ 1);
    __syncthreads();
  }
  // D layout: lane holds rows 4g + e of an M tile, column n of an N tile
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int jt = 0; jt < 4; ++jt)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int v = v0 + wm * 64 + 16 * i + 4 * g + e, q = q0 + wn * 64 + 16 * jt + n;
        if (v < V && q < Q) T[(size_t)v * Q + q] = acc[i][jt][e];
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
    const int nvb = (h.V + kFM - 1) / kFM, nqb = (Q + kFN - 1) / kFN;
    const int64_t groups = (int64_t)8 * nqb * ((nvb + 7) / 8);   // whole rounds of the 8 XCDs
    k_fold_input<<<(unsigned)groups, 256, 0, st>>>((const bf16_t*)h.emb, (const bf16_t*)h.w_ih, h.V, h.d, Q, nvb,
                                                   nqb, (float*)(base + L.off_T));
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  k_pack_vocab<<<2048, 256, 0, st>>>((const bf16_t*)h.w_vocab, h.V, h.r, L.NT, (uint4*)(base + L.off_wv));
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (!markov) k_pack_whh<<<512, 256, 0, st>>>((const bf16_t*)h.w_hh, h.H, (uint4*)(base + L.off_whh));
  return hipGetLastError();
}

}  // namespace dls
