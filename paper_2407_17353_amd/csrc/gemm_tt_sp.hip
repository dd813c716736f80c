// Instantiations of the scaled FP8 GEMM with the single-pass dynamic rescale (grid barrier on
// the amax statistic, cast in the same kernel) for
// A stored [K][M] and B stored [N][K].
#include "gemm4_kernel.h"

namespace scalify {

template <>
hipError_t launch_layout_sp<true, true>(const GemmParams& p, int fa, int fb, int, hipStream_t s) {
  return by_formats<SpFamily<true, true, false>::template F>(p, fa, fb, s);
}

}  // namespace scalify
