// One translation unit of the kernel family: the (TM, TN) instantiations of a
// single (dtype, MFMA size, path) triple, selected with -DGT_DT, -DGT_I and
// -DGT_FAST at compile time, exposed through one lookup function.
#include "gemm_kernel.hpp"

#if !defined(GT_DT) || !defined(GT_I) || !defined(GT_FAST)
#error "compile with -DGT_DT=<0|1> -DGT_I=<16|32> -DGT_FAST=<0|1>"
#endif

#define GT_CAT5(a, b, c, d, e) a##b##c##d##e
#define GT_NAME(a, b, c, d, e) GT_CAT5(a, b, c, d, e)
#if GT_DT == 0
#define GT_DTN f32
#else
#define GT_DTN bf16
#endif
#if GT_FAST
#define GT_PATH fast
#else
#define GT_PATH generic
#endif

namespace gt {

LaunchFn GT_NAME(lookup_, GT_DTN, _, GT_I, GT_NAME(_, GT_PATH, , , ))(int tm, int tn) {
#define GT_CASE(a, b) \
  if (tm == a && tn == b) return &launch_gemm<GT_DT, GT_I, a, b, GT_FAST != 0>;
#if GT_I == 32
  GT_PAIRS_16(GT_CASE)
#else
  GT_PAIRS_64(GT_CASE)
#endif
#undef GT_CASE
  return nullptr;
}

}  // namespace gt
