// Instantiations of the scaled FP8 GEMM with the fused residual add and
// activation epilogue, for A stored [K][M] and B stored [K][N].
#include "gemm_kernel.h"

namespace scalify {

template <>
hipError_t launch_layout<true, false, true>(const GemmParams& p, int fa, int fb, int epi,
                                                 hipStream_t s) {
  return launch_formats<true, false, true>(p, fa, fb, epi, s);
}

}  // namespace scalify
