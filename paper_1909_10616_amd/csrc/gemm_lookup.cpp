// Dispatch from (dtype, MFMA size, CPR, layout, TM, TN) to the instantiation
// that the per-triple translation units provide.
#include "gemm_kernel.hpp"

namespace gt {

#define GT_DECL(dt, i, c, k) LaunchFn lookup_##dt##_##i##_##c##_##k(int, int);
#define GT_TRIPLES(X)                                                                          \
  X(0, 16, 0, 0) X(0, 32, 0, 0) X(1, 16, 0, 0) X(1, 32, 0, 0) X(0, 32, 2, 0) X(0, 32, 4, 0)    \
      X(0, 32, 8, 0) X(0, 32, 16, 0) X(0, 16, 4, 0) X(0, 16, 8, 0) X(0, 16, 16, 0)              \
          X(1, 32, 2, 0) X(1, 32, 4, 0) X(1, 32, 8, 0) X(1, 32, 16, 0) X(1, 16, 4, 0)           \
              X(1, 16, 8, 0) X(1, 16, 16, 0) X(0, 32, 2, 1) X(0, 32, 4, 1) X(0, 32, 8, 1)       \
                  X(0, 32, 16, 1) X(0, 16, 4, 1) X(0, 16, 8, 1) X(0, 16, 16, 1)
GT_TRIPLES(GT_DECL)
#undef GT_DECL

LaunchFn find_gemm_kernel(int dtype, int I, int cpr, int TM, int TN, bool akm) {
  const int k = akm ? 1 : 0;
#define GT_PICK(dt, i, c, kk) \
  if (dtype == dt && I == i && cpr == c && k == kk) return lookup_##dt##_##i##_##c##_##kk(TM, TN);
  GT_TRIPLES(GT_PICK)
#undef GT_PICK
  return nullptr;
}

}  // namespace gt
