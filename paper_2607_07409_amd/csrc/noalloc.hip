// The device scratch of dls_draft_block_noalloc: drafting without a caller workspace, for
// callers that cannot allocate (graph capture, serving loops, allocation-free harnesses).
//
// The scratch is a file-scope __device__ array, so every GPU the library runs on holds its
// own copy from the moment the code object is loaded until the process ends.  In host code
// `scratch` names a host-side stand-in, not device memory: the device address of each GPU's
// copy comes from hipGetSymbolAddress, taken once per device with that device current, and
// only that address is handed to kernels.
#include <mutex>
#include <type_traits>

#include "dels_internal.hpp"

namespace dls {

namespace {

static __device__ __align__(256) uint8_t scratch[kNoallocScratchBytes];

struct ScratchAddr {
  std::once_flag once;
  hipError_t err;
  void* ptr;
};
static_assert(std::is_trivially_destructible<ScratchAddr>::value, "no exit-time destructor");
ScratchAddr g_scratch[64];

// One workgroup: when the previous call on this scratch left its error word set (a failed
// persistent call), zero-fill the whole scratch, the error word last, so that the next call
// starts from the state a fresh workspace has.  Otherwise it only reads the word.
__global__ __launch_bounds__(1024) void k_scratch_guard(uint32_t* s, size_t words) {
  __shared__ uint32_t flag;
  if (threadIdx.x == 0) flag = __hip_atomic_load(s + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  if (flag == 0) return;
  uint4* s4 = (uint4*)s;
  for (size_t i = 64 + threadIdx.x; i < words / 4; i += blockDim.x) s4[i] = make_uint4(0u, 0u, 0u, 0u);
  __syncthreads();
  __threadfence();
  if (threadIdx.x < 256) s[threadIdx.x] = 0u;   // the 1 KiB head: epoch and error word
}

}  // namespace

void* noalloc_scratch(int dev, hipError_t* err) {
  if (dev < 0 || dev >= 64) {
    *err = hipErrorInvalidDevice;
    return nullptr;
  }
  ScratchAddr& sa = g_scratch[dev];
  // set-up, once per device, with that device current (the caller's current device)
  std::call_once(sa.once, [&]() {
    void* p = nullptr;
    sa.err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    sa.ptr = sa.err == hipSuccess ? p : nullptr;
  });
  *err = sa.err;
  return sa.ptr;
}

hipError_t launch_scratch_guard(void* dev_scratch, hipStream_t st) {
  k_scratch_guard<<<1, 1024, 0, st>>>((uint32_t*)dev_scratch, kNoallocScratchBytes / 4);
  return hipGetLastError();
}

}  // namespace dls
