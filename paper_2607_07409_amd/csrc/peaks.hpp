// Measurement helpers (peaks.hip): attainable HBM read bandwidth and bf16 matrix-core throughput.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace dls {
constexpr int kMeasureReadGroups = 8192;   // workgroups (and checksum words) of the read measurement
hipError_t launch_measure_read(const void* buf, size_t bytes, uint32_t* out, hipStream_t st);
hipError_t launch_measure_mfma(int groups, int iters, float x, float* out, hipStream_t st);
}  // namespace dls
