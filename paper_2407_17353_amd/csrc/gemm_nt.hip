// Instantiations of the scaled FP8 GEMM for A stored [M][K] and B stored [N][K].
#include "gemm_kernel.h"

namespace scalify {

template <>
hipError_t launch_layout<false, true, false>(const GemmParams& p, int fa, int fb, int epi,
                                                 hipStream_t s) {
  return launch_formats<false, true, false>(p, fa, fb, epi, s);
}

}  // namespace scalify
