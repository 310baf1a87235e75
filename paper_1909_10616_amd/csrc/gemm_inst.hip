// One translation unit of the kernel family: the (TM, TN) instantiations of a
// single (dtype, MFMA size, CPR) triple (CPR = 0: generic path), selected
// with -DGT_DT, -DGT_I and -DGT_CPR at compile time; -DGT_AKM=1 builds the
// K-major-A fast path of the triple instead.
#include "gemm_kernel.hpp"

#if !defined(GT_DT) || !defined(GT_I) || !defined(GT_CPR)
#error "compile with -DGT_DT=<0|1> -DGT_I=<16|32> -DGT_CPR=<0|2|4|8|16> [-DGT_AKM=1]"
#endif
#ifndef GT_AKM
#define GT_AKM 0
#endif

#define GT_CAT(a, b, c, d, e) a##_##b##_##c##_##d##_##e
#define GT_LOOKUP_NAME(a, b, c, d, e) GT_CAT(a, b, c, d, e)

namespace gt {

LaunchFn GT_LOOKUP_NAME(lookup, GT_DT, GT_I, GT_CPR, GT_AKM)(int tm, int tn) {
#define GT_CASE(a, b) \
  if (tm == a && tn == b) return &launch_gemm<GT_DT, GT_I, a, b, GT_CPR, GT_AKM != 0>;
#if GT_I == 32
  GT_PAIRS_16(GT_CASE)
#else
  GT_PAIRS_64(GT_CASE)
#endif
#undef GT_CASE
  return nullptr;
}

}  // namespace gt
