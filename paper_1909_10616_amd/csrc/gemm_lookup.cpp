// Dispatch from (dtype, MFMA size, CPR, TM, TN) to the instantiation that
// the per-triple translation units provide.
#include "gemm_kernel.hpp"

namespace gt {

#define GT_DECL(dt, i, c) LaunchFn lookup_##dt##_##i##_##c(int, int);
#define GT_TRIPLES(X)                                                                     \
  X(0, 16, 0) X(0, 32, 0) X(1, 16, 0) X(1, 32, 0) X(0, 32, 2) X(0, 32, 4) X(0, 32, 8)     \
      X(0, 32, 16) X(0, 16, 4) X(0, 16, 8) X(0, 16, 16) X(1, 32, 2) X(1, 32, 4)          \
          X(1, 32, 8) X(1, 32, 16) X(1, 16, 4) X(1, 16, 8) X(1, 16, 16)
GT_TRIPLES(GT_DECL)
#undef GT_DECL

LaunchFn find_gemm_kernel(int dtype, int I, int cpr, int TM, int TN) {
#define GT_PICK(dt, i, c) \
  if (dtype == dt && I == i && cpr == c) return lookup_##dt##_##i##_##c(TM, TN);
  GT_TRIPLES(GT_PICK)
#undef GT_PICK
  return nullptr;
}

}  // namespace gt
