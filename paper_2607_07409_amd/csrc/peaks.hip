// Measurement helpers: the attainable HBM read bandwidth and bf16 matrix-core throughput of
// the device, reported beside the vendor peaks that the rooflines are quoted against.  They
// compute nothing of the method.
#include "peaks.hpp"

namespace dls {

namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;

// Streams n16 16-byte pieces once with non-temporal loads, kUnroll per thread in flight, and
// folds them into one checksum word per workgroup (XOR of every 32-bit word) so that no load can
// be dropped.  Non-temporal loads and 8 in flight read about 15% faster than plain loads and 4.
typedef __attribute__((ext_vector_type(4))) unsigned u32x4_t;
constexpr int kUnroll = 8;
__global__ __launch_bounds__(256) void k_measure_read(const u32x4_t* __restrict__ buf, size_t n16,
                                                      uint32_t* __restrict__ out) {
  __shared__ uint32_t sh[4];
  const size_t stride = (size_t)gridDim.x * 256;
  size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  uint32_t acc = 0;
  for (; i + (kUnroll - 1) * stride < n16; i += kUnroll * stride) {
    u32x4_t v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) v[u] = __builtin_nontemporal_load(buf + i + u * stride);
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (; i < n16; i += stride) {
    const u32x4_t a = __builtin_nontemporal_load(buf + i);
    acc ^= a.x ^ a.y ^ a.z ^ a.w;
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) acc ^= (uint32_t)__shfl_xor((int)acc, m);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) out[blockIdx.x] = sh[0] ^ sh[1] ^ sh[2] ^ sh[3];
}

// iters rounds of kChains independent v_mfma_f32_32x32x16_bf16 products (32768 flops each) per
// wave, which the compiler keeps in place in the accumulation registers (the 16x16x32 form with 8
// chains gets its accumulators shuffled through VGPRs every round).  Every input element is x (a
// power of two given by the caller), so every output element of one product is 16 x^2 and each
// lane's sum over its kChains x 16 accumulators after iters rounds is iters * 1024 x^2, exact in
// float32 for the iteration counts the ABI allows.
constexpr int kChains = 4;
typedef __attribute__((ext_vector_type(16))) float f32x16_t;
__global__ __launch_bounds__(256) void k_measure_mfma(int iters, float x, float* __restrict__ out) {
  const __bf16 xb = (__bf16)x;
  const bf16x8_t a = {xb, xb, xb, xb, xb, xb, xb, xb};
  f32x16_t acc[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c) acc[c] = f32x16_t{};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < kChains; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, a, acc[c], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kChains; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) s += acc[c][e];
  out[(size_t)blockIdx.x * 256 + threadIdx.x] = s;
}

}  // namespace

hipError_t launch_measure_read(const void* buf, size_t bytes, uint32_t* out, hipStream_t st) {
  k_measure_read<<<kMeasureReadGroups, 256, 0, st>>>((const u32x4_t*)buf, bytes / 16, out);
  return hipGetLastError();
}

hipError_t launch_measure_mfma(int groups, int iters, float x, float* out, hipStream_t st) {
  k_measure_mfma<<<groups, 256, 0, st>>>(iters, x, out);
  return hipGetLastError();
}

}  // namespace dls
