// Instantiations of the scaled FP8 GEMM for A stored [K][M] and B stored [K][N].
#include "gemm_kernel.h"

namespace scalify {

template <>
hipError_t launch_layout<true, false, false>(const GemmParams& p, int fa, int fb, int epi,
                                                 hipStream_t s) {
  return launch_formats<true, false, false>(p, fa, fb, epi, s);
}

}  // namespace scalify
