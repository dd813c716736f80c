// Instantiations of the scaled FP8 GEMM with the pre-cast intermediate (GEMM + cast kernel) for
// A stored [M][K] and B stored [N][K].
#include "gemm4_kernel.h"

namespace scalify {

template <>
hipError_t launch_layout<false, true, false>(const GemmParams& p, int fa, int fb, int, hipStream_t s) {
  return by_formats<PlainFamily<false, true, false>::template F>(p, fa, fb, s);
}

}  // namespace scalify
