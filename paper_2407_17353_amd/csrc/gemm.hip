// Dispatch of the scaled FP8 GEMM over the four storage orders of A and B.
#include "gemm_kernel.h"

namespace scalify {

hipError_t launch_gemm(const GemmParams& p, bool a_mn, bool b_kc, int fa, int fb, int epi,
                       bool fuse, hipStream_t s) {
  if (p.tiles_m * p.tiles_n == 0) return hipSuccess;
  if (p.mx_a) {
    if (!a_mn && b_kc) return launch_layout_mx<false, true>(p, fa, fb, epi, s);
    if (!a_mn && !b_kc) return launch_layout_mx<false, false>(p, fa, fb, epi, s);
    if (a_mn && b_kc) return launch_layout_mx<true, true>(p, fa, fb, epi, s);
    return launch_layout_mx<true, false>(p, fa, fb, epi, s);
  }
  if (fuse) {
    if (!a_mn && b_kc) return launch_layout<false, true, true>(p, fa, fb, epi, s);
    if (!a_mn && !b_kc) return launch_layout<false, false, true>(p, fa, fb, epi, s);
    if (a_mn && b_kc) return launch_layout<true, true, true>(p, fa, fb, epi, s);
    return launch_layout<true, false, true>(p, fa, fb, epi, s);
  }
  if (!a_mn && b_kc) return launch_layout<false, true, false>(p, fa, fb, epi, s);
  if (!a_mn && !b_kc) return launch_layout<false, false, false>(p, fa, fb, epi, s);
  if (a_mn && b_kc) return launch_layout<true, true, false>(p, fa, fb, epi, s);
  return launch_layout<true, false, false>(p, fa, fb, epi, s);
}

}  // namespace scalify
