// One translation unit of the kernel family: the (TM, TN) instantiations of a
// single (dtype, MFMA size, CPR) triple (CPR = 0: generic path), selected
// with -DGT_DT, -DGT_I and -DGT_CPR at compile time.
#include "gemm_kernel.hpp"

#if !defined(GT_DT) || !defined(GT_I) || !defined(GT_CPR)
#error "compile with -DGT_DT=<0|1> -DGT_I=<16|32> -DGT_CPR=<0|2|4|8|16>"
#endif

#define GT_CAT(a, b, c, d) a##_##b##_##c##_##d
#define GT_LOOKUP_NAME(a, b, c, d) GT_CAT(a, b, c, d)

namespace gt {

LaunchFn GT_LOOKUP_NAME(lookup, GT_DT, GT_I, GT_CPR)(int tm, int tn) {
#define GT_CASE(a, b) \
  if (tm == a && tn == b) return &launch_gemm<GT_DT, GT_I, a, b, GT_CPR>;
#if GT_I == 32
  GT_PAIRS_16(GT_CASE)
#else
  GT_PAIRS_64(GT_CASE)
#endif
#undef GT_CASE
  return nullptr;
}

}  // namespace gt
