// gt_compare_noalloc: the output comparison with its result words in a
// static device array instead of a buffer the library allocates, for callers
// that may not allocate device memory.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>
#include <string>

#include "internal.h"
#include "runtime.h"

// The comparison's two result words (max |C − R| and max |R| as ordered bit
// patterns) live in words 0 and 1; 64 words (256 bytes) in all. Every call on
// a GPU uses that GPU's copy: the comparison kernel's first launch clears the
// two words, and calls that overlap on one GPU race on them.
static __device__ __align__(256) unsigned scratch[64];

namespace gt {
namespace {

// Device address of `scratch` on each GPU (its own copy there), looked up
// once per device with that device current. In host code `scratch` names a
// host-side stand-in, never the device memory: only these pointers are passed
// to kernels and copies.
std::mutex g_mu;
unsigned* g_scratch_ptr[64] = {};

int scratch_of_current_device(unsigned** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    set_error(std::string("gt_compare_noalloc: hipGetDevice: ") + hipGetErrorString(e));
    return GT_EHIP;
  }
  if (dev < 0 || dev >= 64) {
    set_error("gt_compare_noalloc: device index out of range");
    return GT_EINVAL;
  }
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      set_error(std::string("gt_compare_noalloc: hipGetSymbolAddress: ") + hipGetErrorString(e));
      return GT_EHIP;
    }
    g_scratch_ptr[dev] = static_cast<unsigned*>(p);
  }
  *out = g_scratch_ptr[dev];
  return GT_OK;
}

}  // namespace
}  // namespace gt

extern "C" int gt_compare_noalloc(const void* C, const void* R, int64_t n, void* stream,
                                  double* rel) {
  if (!C || !R || !rel || n < 1) {
    gt::set_error("gt_compare_noalloc: bad argument");
    return GT_EINVAL;
  }
  unsigned* buf = nullptr;
  if (int rc = gt::scratch_of_current_device(&buf)) return rc;
  return gt::compare_into(C, R, n, buf, static_cast<hipStream_t>(stream), rel);
}
