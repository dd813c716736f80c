// Instantiations of the scaled FP8 GEMM with the direct cast (output scale known before the
// GEMM: delayed or no rescale) for
// A stored [K][M] and B stored [N][K].
#include "gemm4_kernel.h"

namespace scalify {

template <>
hipError_t launch_layout_direct<true, true>(const GemmParams& p, int fa, int fb, int, hipStream_t s) {
  return by_formats<DirectFamily<true, true, false>::template F>(p, fa, fb, s);
}

}  // namespace scalify
