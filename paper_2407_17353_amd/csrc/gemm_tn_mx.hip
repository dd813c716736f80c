// Instantiations of the scaled FP8 GEMM with MX block scales for A stored
// [K][M] and B stored [K][N].
#include "gemm_kernel.h"

namespace scalify {

template <>
hipError_t launch_layout_mx<true, false>(const GemmParams& p, int fa, int fb, int epi,
                                        hipStream_t s) {
  return launch_formats_mx<true, false>(p, fa, fb, epi, s);
}

}  // namespace scalify
