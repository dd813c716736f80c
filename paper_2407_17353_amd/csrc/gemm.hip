// Dispatch of the scaled FP8 GEMM over the four storage orders of A and B.
#include "gemm4_kernel.h"

namespace scalify {

int gemm4_grid(int tiles) {
  constexpr int kMaxDevices = 64;
  static int cus[kMaxDevices];  // CUs per device, looked up once (a benign race)
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) dev = -1;
  int n = dev >= 0 ? cus[dev] : 0;
  if (n <= 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev < 0 ? 0 : dev) !=
            hipSuccess || n <= 0)
      n = 256;
    if (dev >= 0) cus[dev] = n;
  }
  return tiles < n ? tiles : n;
}

hipError_t launch_gemm(const GemmParams& p_in, bool a_mn, bool b_kc, int fa, int fb, int epi,
                       bool fuse, hipStream_t s) {
  if (p_in.tiles_m * p_in.tiles_n == 0) return hipSuccess;
  GemmParams p = p_in;
  p.epi = epi;
  if (p.mx_a) {
    if (mx_on_8_waves(a_mn, b_kc)) return launch_layout_mx<true, false>(p, fa, fb, epi, s);
    if (!p.single_pass) {
      if (!a_mn && b_kc) return launch_layout_mx<false, true>(p, fa, fb, epi, s);
      if (!a_mn && !b_kc) return launch_layout_mx<false, false>(p, fa, fb, epi, s);
      return launch_layout_mx<true, true>(p, fa, fb, epi, s);
    }
    if (!a_mn && b_kc) return launch_layout_mx_sp<false, true>(p, fa, fb, epi, s);
    if (!a_mn && !b_kc) return launch_layout_mx_sp<false, false>(p, fa, fb, epi, s);
    return launch_layout_mx_sp<true, true>(p, fa, fb, epi, s);
  }
  if (fuse) {
    if (!a_mn && b_kc) return launch_layout<false, true, true>(p, fa, fb, epi, s);
    if (!a_mn && !b_kc) return launch_layout<false, false, true>(p, fa, fb, epi, s);
    if (a_mn && b_kc) return launch_layout<true, true, true>(p, fa, fb, epi, s);
    return launch_layout<true, false, true>(p, fa, fb, epi, s);
  }
  if (epi == EPI_DIRECT) {
    if (!a_mn && b_kc) return launch_layout_direct<false, true>(p, fa, fb, epi, s);
    if (!a_mn && !b_kc) return launch_layout_direct<false, false>(p, fa, fb, epi, s);
    if (a_mn && b_kc) return launch_layout_direct<true, true>(p, fa, fb, epi, s);
    return launch_layout_direct<true, false>(p, fa, fb, epi, s);
  }
  if (p.single_pass) {
    if (!a_mn && b_kc) return launch_layout_sp<false, true>(p, fa, fb, epi, s);
    if (!a_mn && !b_kc) return launch_layout_sp<false, false>(p, fa, fb, epi, s);
    if (a_mn && b_kc) return launch_layout_sp<true, true>(p, fa, fb, epi, s);
    return launch_layout_sp<true, false>(p, fa, fb, epi, s);
  }
  if (!a_mn && b_kc) return launch_layout<false, true, false>(p, fa, fb, epi, s);
  if (!a_mn && !b_kc) return launch_layout<false, false, false>(p, fa, fb, epi, s);
  if (a_mn && b_kc) return launch_layout<true, true, false>(p, fa, fb, epi, s);
  return launch_layout<true, false, false>(p, fa, fb, epi, s);
}

// One thread per packed 32-bit word: word ((t * G + q) * 64 + 16 g + r)
// holds, lowest byte first, the bytes of rows 64 q + r + 16 i (i = 0..3) at
// k-block 4 t + g; rows and blocks outside the array read as 127 (factor 1).
__global__ __launch_bounds__(256) void mx_pack_kernel(const uint8_t* __restrict__ src, int rows,
                                                      int nblk, int ld, int groups, int words,
                                                      uint32_t* __restrict__ dst) {
  const int w = blockIdx.x * 256 + threadIdx.x;
  if (w >= words) return;
  const int lane = w & 63, q = (w >> 6) % groups, t = (w >> 6) / groups;
  const int blk = 4 * t + (lane >> 4);
  uint32_t v = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = 64 * q + 16 * i + (lane & 15);
    const uint32_t byte = (r < rows && blk < nblk) ? src[(int64_t)r * ld + blk] : 127u;
    v |= byte << (8 * i);
  }
  dst[w] = v;
}

hipError_t launch_mx_pack(const uint8_t* src, int rows, int K, int ld, uint8_t* dst,
                          hipStream_t s) {
  const int groups = (rows + 63) / 64, steps = (K + 127) / 128;
  const int words = steps * groups * 64;
  hipLaunchKernelGGL(mx_pack_kernel, dim3((words + 255) / 256), dim3(256), 0, s, src, rows,
                     (K + 31) / 32, ld, groups, words, (uint32_t*)dst);
  return hipGetLastError();
}

}  // namespace scalify
