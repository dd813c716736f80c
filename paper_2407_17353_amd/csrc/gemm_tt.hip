// Instantiations of the scaled FP8 GEMM with the pre-cast intermediate (GEMM + cast kernel) for
// A stored [K][M] and B stored [N][K].
#include "gemm4_kernel.h"

namespace scalify {

template <>
hipError_t launch_layout<true, true, false>(const GemmParams& p, int fa, int fb, int, hipStream_t s) {
  return by_formats<PlainFamily<true, true, false>::template F>(p, fa, fb, s);
}

}  // namespace scalify
