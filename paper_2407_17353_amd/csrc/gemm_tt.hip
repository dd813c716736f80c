// Instantiations of the scaled FP8 GEMM for A stored [K][M] and
// B stored [N][K].
#include "gemm_kernel.h"

namespace scalify {

template <int FA, int FB>
static hipError_t launch_fmt(const GemmParams& p, int epi, hipStream_t s) {
  const dim3 grid(p.tiles_m * p.tiles_n), block(NTHR);
  switch (epi) {
    case EPI_INTER16:
      hipLaunchKernelGGL((gemm_kernel<true, true, FA, FB, EPI_INTER16>), grid, block, 0, s, p);
      break;
    case EPI_INTER32:
      hipLaunchKernelGGL((gemm_kernel<true, true, FA, FB, EPI_INTER32>), grid, block, 0, s, p);
      break;
    default:
      hipLaunchKernelGGL((gemm_kernel<true, true, FA, FB, EPI_DIRECT>), grid, block, 0, s, p);
      break;
  }
  return hipGetLastError();
}

template <>
hipError_t launch_layout<true, true>(const GemmParams& p, int fa, int fb, int epi, hipStream_t s) {
  if (fa == kE4M3 && fb == kE4M3) return launch_fmt<kE4M3, kE4M3>(p, epi, s);
  if (fa == kE4M3 && fb == kE5M2) return launch_fmt<kE4M3, kE5M2>(p, epi, s);
  if (fa == kE5M2 && fb == kE4M3) return launch_fmt<kE5M2, kE4M3>(p, epi, s);
  return launch_fmt<kE5M2, kE5M2>(p, epi, s);
}

}  // namespace scalify
