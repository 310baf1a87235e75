// Lowered form of a configuration and the runtime's internal entry points.
#pragma once
#include <hip/hip_runtime.h>

#include "gemm_kernel.hpp"
#include "internal.h"

namespace gt {

struct Lowered {
  KArgs args;
  dim3 grid, block;
  size_t lds = 0;
  bool fast = false;
  LaunchFn fn = nullptr;
  Levels L;
};

// Validates (membership, J) and lowers; GT_OK or an error with message.
int lower(const gt_config& c, int64_t M, int64_t N, int64_t K, int dtype, const void* A,
          const void* B, void* C, Lowered* out);
int launch_lowered(const Lowered& lw, hipStream_t s);
// Spread of the timed runs of one measurement (each run between its own pair
// of events; the mean is first-to-last over the runs).
struct RunStats {
  double median_ms, min_ms, stdev_ms;
};
int measure(const gt_config& c, const void* A, const void* B, void* C, int64_t M, int64_t N,
            int64_t K, int dtype, hipStream_t s, int warmup, int runs, double abort_ms,
            double* mean_ms, double* first_ms, int* aborted, RunStats* stats);
int compare_on_gpu(const void* C, const void* R, int64_t n, hipStream_t s, double* rel);
// The comparison with a caller-chosen 2-word device buffer (cleared by a
// kernel, filled by the reduction, read back; synchronises the stream).
int compare_into(const void* C, const void* R, int64_t n, unsigned* buf, hipStream_t s,
                 double* rel);

}  // namespace gt
