// Instantiations of the scaled FP8 GEMM with MX block scales and the single-pass dynamic
// rescale for
// A stored [M][K] and B stored [K][N].
#include "gemm4_kernel.h"

namespace scalify {

template <>
hipError_t launch_layout_mx_sp<false, false>(const GemmParams& p, int fa, int fb, int, hipStream_t s) {
  return by_formats<SpFamily<false, false, true>::template F>(p, fa, fb, s);
}

}  // namespace scalify
