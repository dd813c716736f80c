// Instantiations of the scaled FP8 GEMM with the fused residual add and
// activation epilogue, for A stored [K][M] and B stored [N][K].
#include "gemm_kernel.h"

namespace scalify {

template <>
hipError_t launch_layout<true, true, true>(const GemmParams& p, int fa, int fb, int epi,
                                                 hipStream_t s) {
  return launch_formats<true, true, true>(p, fa, fb, epi, s);
}

}  // namespace scalify
