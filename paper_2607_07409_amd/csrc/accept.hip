// Prefix-acceptance length (verification step of Algorithm 1): the number of leading
// positions where the draft equals the target.  One wave per sequence; a ballot over
// 64 positions at a time finds the first mismatch.
#include "dels_internal.hpp"

namespace dls {

namespace {

__global__ __launch_bounds__(256) void k_accept_len(const int32_t* __restrict__ draft,
                                                    const int32_t* __restrict__ target, int batch, int B,
                                                    int32_t* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const int b = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (b >= batch) return;
  const int32_t* dr = draft + (size_t)b * B;
  const int32_t* tg = target + (size_t)b * B;
  int a = B;
  for (int j0 = 0; j0 < B; j0 += 64) {
    const int j = j0 + lane;
    const bool mis = j < B && dr[j] != tg[j];
    const unsigned long long m = __ballot(mis);
    if (m) {
      a = j0 + __ffsll((long long)m) - 1;
      break;
    }
  }
  if (lane == 0) out[b] = a;
}

}  // namespace

hipError_t launch_accept(const int32_t* draft, const int32_t* target, int32_t batch, int32_t B, int32_t* out,
                         hipStream_t st) {
  k_accept_len<<<(unsigned)((batch + 3) / 4), 256, 0, st>>>(draft, target, batch, B, out);
  return hipGetLastError();
}

}  // namespace dls
