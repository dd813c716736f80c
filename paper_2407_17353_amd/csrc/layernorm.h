// Internal interface of the scaled LayerNorm kernels (layernorm.hip).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace scalify {

// Rows of D <= 8192 values, row-major.
struct LnParams {
  const void* x;        // [R][ldx], format x_fmt
  int64_t ldx;
  int x_fmt;
  const void* dy;       // backward: [R][lddy], format dy_fmt
  int64_t lddy;
  int dy_fmt;
  const float* gamma;   // [D] or NULL (1)
  const float* beta;    // [D] or NULL (0)
  void* out;            // forward y / backward dx codes [R][ldo]
  int64_t ldo;
  float* pre_out;       // optional fp32 [R][D]: the values before the cast
  int64_t R;
  int D;
  float eps;
  int sat, target, mode;  // backward rescale: mode 1 = amax, 0 = none
  uint32_t* hdr;        // backward: workspace header
  float* partial;       // backward: per-row numbers [R][4], then [row tiles][2][stride]
  float* out_scale;
  float* amax_out;      // backward: optional amax of |dx|
  float* dgamma;        // backward: optional [D]
  float* dbeta;         // backward: optional [D]
};

constexpr int kLayerNormMaxD = 8192;

// Row stride of the backward's partial parameter gradients (16-float aligned).
__host__ __device__ inline int64_t layernorm_param_stride(int64_t D) { return (D + 15) / 16 * 16; }
// Backward workspace after the header, in floats: per-row numbers (4 R) and
// per-row-tile partial parameter gradients.
int64_t layernorm_ws_floats(int64_t R, int64_t D);
hipError_t launch_layernorm_fwd(const LnParams& p, int out_dtype, hipStream_t s);
hipError_t launch_layernorm_bwd(const LnParams& p, const float* s_dy, const float* s_x,
                                int out_dtype, hipStream_t s);

}  // namespace scalify
