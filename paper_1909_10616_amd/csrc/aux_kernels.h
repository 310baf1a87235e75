// Launchers of the runtime's helper kernels.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

namespace gt {
hipError_t launch_fill_zero(float* p, int64_t n, hipStream_t s);
hipError_t launch_reference(const void* A, const void* B, float* C, int64_t M, int64_t N, int64_t K,
                            int dtype, hipStream_t s);
hipError_t launch_compare(const float* C, const float* R, int64_t n, unsigned* out, hipStream_t s);
}  // namespace gt
