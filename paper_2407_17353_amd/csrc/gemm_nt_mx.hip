// Instantiations of the scaled FP8 GEMM with MX block scales and the direct cast for
// A stored [M][K] and B stored [N][K].
#include "gemm4_kernel.h"

namespace scalify {

template <>
hipError_t launch_layout_mx<false, true>(const GemmParams& p, int fa, int fb, int, hipStream_t s) {
  return by_formats<DirectFamily<false, true, true>::template F>(p, fa, fb, s);
}

}  // namespace scalify
