// Instantiations of the scaled FP8 GEMM with the single-pass dynamic rescale (grid barrier on
// the amax statistic, cast in the same kernel) for
// A stored [M][K] and B stored [K][N].
#include "gemm4_kernel.h"

namespace scalify {

template <>
hipError_t launch_layout_sp<false, false>(const GemmParams& p, int fa, int fb, int, hipStream_t s) {
  return by_formats<SpFamily<false, false, false>::template F>(p, fa, fb, s);
}

}  // namespace scalify
