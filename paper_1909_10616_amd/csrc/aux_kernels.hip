// Helper kernels of the runtime: clearing C before split-K accumulation, the
// plain reference product the search checks candidates against, and a
// normwise difference reduction.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "aux_kernels.h"

namespace gt {
namespace {

__global__ void fill_zero_kernel(float* __restrict__ p, int64_t n) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride)
    p[i] = 0.0f;
}

__device__ __forceinline__ float load_in(const void* p, int64_t i, int dtype) {
  if (dtype == 0) return reinterpret_cast<const float*>(p)[i];
  const uint32_t bits = static_cast<uint32_t>(reinterpret_cast<const uint16_t*>(p)[i]) << 16;
  return __builtin_bit_cast(float, bits);
}

// One thread per output (grid-stride over rows and columns, so any M and N
// fit the grid's limits); k ascending, fp32 fused multiply-add. dtype 0/1
// (fp32/bf16), plus 16 when A is K-major (element (m, k) at A[k·M + m]).
__global__ void reference_kernel(const void* __restrict__ A, const void* __restrict__ B,
                                 float* __restrict__ C, int64_t M, int64_t N, int64_t K,
                                 int dtype) {
  const int dt = dtype & 15;
  const int64_t sr = (dtype & 16) ? 1 : K, sk = (dtype & 16) ? M : 1;
  const int64_t rstep = static_cast<int64_t>(gridDim.y) * blockDim.y;
  const int64_t cstep = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t row = static_cast<int64_t>(blockIdx.y) * blockDim.y + threadIdx.y; row < M;
       row += rstep)
    for (int64_t col = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; col < N;
         col += cstep) {
      float s = 0.0f;
      for (int64_t l = 0; l < K; ++l)
        s = fmaf(load_in(A, row * sr + l * sk, dt), load_in(B, l * N + col, dt), s);
      C[row * N + col] = s;
    }
}

// out[0] = max |C − R| bits, out[1] = max |R| bits (non-negative floats order
// like their bit patterns; a NaN difference wins the max).
__global__ void compare_kernel(const float* __restrict__ C, const float* __restrict__ R, int64_t n,
                               unsigned* __restrict__ out) {
  float md = 0.0f, mr = 0.0f;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride) {
    const float d = fabsf(C[i] - R[i]);
    md = (d > md || d != d) ? d : md;
    mr = fmaxf(mr, fabsf(R[i]));
  }
  unsigned ud = __builtin_bit_cast(unsigned, md), ur = __builtin_bit_cast(unsigned, mr);
  for (int off = 32; off > 0; off >>= 1) {
    ud = max(ud, static_cast<unsigned>(__shfl_xor(static_cast<int>(ud), off)));
    ur = max(ur, static_cast<unsigned>(__shfl_xor(static_cast<int>(ur), off)));
  }
  if ((threadIdx.x & 63) == 0) {
    atomicMax(&out[0], ud);
    atomicMax(&out[1], ur);
  }
}

__global__ void clear2_kernel(unsigned* out) {
  if (threadIdx.x < 2) out[threadIdx.x] = 0u;
}

}  // namespace

hipError_t launch_fill_zero(float* p, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = (n + 255) / 256;
  const unsigned g = static_cast<unsigned>(blocks < 65536 ? blocks : 65536);
  hipLaunchKernelGGL(fill_zero_kernel, dim3(g), dim3(256), 0, s, p, n);
  return hipGetLastError();
}

hipError_t launch_reference(const void* A, const void* B, float* C, int64_t M, int64_t N, int64_t K,
                            int dtype, hipStream_t s) {
  if (M <= 0 || N <= 0) return hipSuccess;  // an empty C: nothing to write
  const dim3 block(64, 4);
  // grid.y is limited to 65535 blocks; the kernel strides over what is left
  const dim3 grid(static_cast<unsigned>(std::min<int64_t>((N + 63) / 64, int64_t{1} << 20)),
                  static_cast<unsigned>(std::min<int64_t>((M + 3) / 4, 65535)));
  hipLaunchKernelGGL(reference_kernel, grid, block, 0, s, A, B, C, M, N, K, dtype);
  return hipGetLastError();
}

hipError_t launch_compare(const float* C, const float* R, int64_t n, unsigned* out, hipStream_t s) {
  hipLaunchKernelGGL(clear2_kernel, dim3(1), dim3(64), 0, s, out);
  const int64_t blocks = (n + 255) / 256;
  const unsigned g = static_cast<unsigned>(blocks < 4096 ? (blocks > 0 ? blocks : 1) : 4096);
  hipLaunchKernelGGL(compare_kernel, dim3(g), dim3(256), 0, s, C, R, n, out);
  return hipGetLastError();
}

}  // namespace gt
