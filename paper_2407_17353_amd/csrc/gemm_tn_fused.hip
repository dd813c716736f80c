// Instantiations of the scaled FP8 GEMM with the fused residual add, activation and channel
// scales for
// A stored [K][M] and B stored [K][N].
#include "gemm4_kernel.h"

namespace scalify {

template <>
hipError_t launch_layout<true, false, true>(const GemmParams& p, int fa, int fb, int, hipStream_t s) {
  return by_formats<PlainFamily<true, false, true>::template F>(p, fa, fb, s);
}

}  // namespace scalify
