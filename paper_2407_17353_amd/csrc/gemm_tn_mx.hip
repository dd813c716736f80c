// Instantiations of the scaled FP8 GEMM with MX block scales (8 waves: direct cast, or fp32
// intermediate + cast kernel) for
// A stored [K][M] and B stored [K][N].
#include "gemm4_kernel.h"

namespace scalify {

template <>
hipError_t launch_layout_mx<true, false>(const GemmParams& p, int fa, int fb, int, hipStream_t s) {
  return by_formats<Mx8Family<true, false>::template F>(p, fa, fb, s);
}

}  // namespace scalify
