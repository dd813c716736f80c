// Internal interface between the C ABI (scalify_abi.hip) and the kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace scalify {

// Workspace header, in 32-bit words at the start of every workspace:
//   [0] amax as fp32 bits (atomic max target; zeroed by the prologue)
//   [1] e_w, the scale exponent of the pre-cast value w (the exponent sum of
//       the input scales, or the scaled-add exponent with a residual):
//       snapshot taken by the prologue, so that an output scale aliasing an
//       input scale cannot race
//   [2] direct cast (delayed rescale, or none): its shift, data' = w * 2^-shift
//   [3] fused residual add: shift of acc into w's scale (e_a + e_b - e_w)
//   [4] fused residual add: shift of the residual (q - e_w)
//   [5] single pass: workgroups arrived at the grid barrier (zeroed by the prologue)
//   [6] single pass: barrier state, 0 running, 1 complete, 2 aborted (zeroed by the prologue)
//   [7] single pass: workgroups that wrote their held tile after an abort (zeroed by the prologue)
constexpr size_t kHeaderBytes = 256;

// Activation of the fused epilogue (values of scalify_activation).
enum Act : int { ACT_NONE = 0, ACT_RELU = 1, ACT_GELU_TANH = 2, ACT_SILU = 3 };

// What the GEMM writes: a pre-cast intermediate for the cast kernel that
// follows (16-bit rounding-preserving encoding for FP8 outputs, the fp32
// accumulator for FP16 outputs), or, when the output scale is known before
// the GEMM runs (delayed rescale), the output codes themselves.
enum Epi : int { EPI_INTER16 = 0, EPI_INTER32 = 1, EPI_DIRECT = 2 };

struct GemmParams {
  const uint8_t* a;
  const uint8_t* b;
  int64_t lda, ldb;
  uint32_t a_bytes, b_bytes;  // stored-matrix sizes (buffer range limits)
  int M, N, K;
  int tiles_m, tiles_n;
  int e_c;        // matmul scale rule exponent
  int sat;
  uint32_t* hdr;  // workspace header
  void* inter;    // pre-cast intermediate [M][ldw] (EPI_INTER16: u16, EPI_INTER32: f32)
  int64_t ldw;
  float* acc_out;  // optional raw accumulator [M][N]
  void* out;       // EPI_DIRECT: output codes [M][ldc] of format out_fmt
  int64_t ldc;
  int out_fmt;
  // Fused epilogue (FUSE kernels only): residual codes [M][ldr] (ldr = 0:
  // one row for every row) of format res_fmt or NULL, activation, and the
  // optional export of the pre-cast value w [M][N].
  const void* res;
  int64_t ldr;
  int res_fmt;
  int act;
  float* pre_out;
  // Channel scales (FUSE kernels only): powers of two per output row
  // (ch_a [M]) and per output column (ch_b [N]) multiplied into the
  // accumulator with the power-of-two product of the epilogue; NULL = 1.
  const float* ch_a;
  const float* ch_b;
  // MX block scales (MX kernels only), packed by launch_mx_pack: per 128-k
  // step and 64-row group (mx_groups_* = ceil(rows / 64) groups), 64 words,
  // word 16 g + r holding the bytes of rows r, r + 16, r + 32, r + 48 of the
  // group at k-block g of the step; byte sizes for the buffer range checks.
  const uint8_t* mx_a;
  const uint8_t* mx_b;
  int mx_groups_a, mx_groups_b;
  uint32_t mx_a_bytes, mx_b_bytes;
  // The persistent 4-wave kernel: workgroups (gemm4_grid), and the single
  // pass of the dynamic rescale (EPI_INTER16 / EPI_INTER32 kernels that hold
  // their last tile, meet at a grid barrier and cast): its rescale target,
  // the output scale and statistic it writes, and the barrier's wait budget
  // in ticks of the 100 MHz real-time counter.
  int grid;
  int epi;  // Epi of the launch (set by launch_gemm)
  int single_pass;
  int target;
  float* out_scale;
  float* amax_out;
  int64_t spin_ticks;
};

// Workgroups of the persistent 4-wave kernel for `tiles` output tiles: one
// per CU of the current device (its LDS holds one workgroup), at most one
// per tile.
int gemm4_grid(int tiles);

// Packed MX block scales (see GemmParams) from row-major bytes src[r * ld + b].
hipError_t launch_mx_pack(const uint8_t* src, int rows, int K, int ld, uint8_t* dst,
                          hipStream_t s);

// fuse: launch the kernels with the fused residual add / activation / pre_out
// epilogue (the plain kernels otherwise).
hipError_t launch_gemm(const GemmParams& p, bool a_mn, bool b_kc, int fa, int fb, int epi,
                       bool fuse, hipStream_t s);

// Prologue: hdr[0] = 0, hdr[1] = exponent(s0) + exponent(s1) (NULL = scale 1).
hipError_t launch_prologue(uint32_t* hdr, const float* s0, const float* s1, hipStream_t s);

// Prologue of the matmul: hdr[0] = hdr[5] = hdr[6] = hdr[7] = 0 and hdr[1] =
// e_w, the scale exponent of the pre-cast value: e_a + e_b, or with a
// residual of scale 2^q the scaled add exponent max(e_a + e_b + e_c, q)
// (sqrt(s_p^2 + s_r^2) rounded down), with hdr[3] = e_a + e_b - e_w and
// hdr[4] = q - e_w. Direct cast (output scale known before the GEMM): from
// the statistic *amax_in of an earlier call (delayed rescale; e_r =
// floor(log2 amax_in) - target, 0 when amax_in is 0, Inf or NaN) or with
// e_r = 0 (no rescale, amax_in NULL): writes *out_scale = 2^e_out, e_out =
// clamp(e_w + e_cc + e_r), and hdr[2] = e_out - e_w, where e_cc = e_c
// without a residual and 0 with one.
struct MatmulPrologue {
  const float* s0;
  const float* s1;
  const float* s_res;  // residual scale (NULL = 1)
  int residual;        // 1: scaled add of a residual
  int e_c;
  int direct;
  const float* amax_in;
  int target;
  float* out_scale;
};
hipError_t launch_matmul_prologue(uint32_t* hdr, const MatmulPrologue& q, hipStream_t s);

// *amax_out = amax recorded in hdr[0] (max |w|) times 2^-e_cc.
hipError_t launch_finalize_amax(const uint32_t* hdr, int e_c, float* amax_out, hipStream_t s);

// Cast of the GEMM intermediate [M][ldw] to out [M][ldc]; computes the
// rescale exponent from hdr and writes *out_scale (and *amax_out).
struct EpilogueParams {
  const void* inter;
  int64_t ldw;
  void* out;
  int64_t ldc;
  int M, N;
  int e_c, target, sat, mode;
  const uint32_t* hdr;
  float* out_scale;
  float* amax_out;
};
hipError_t launch_epilogue_cast(const EpilogueParams& p, int inter32, int out_dtype,
                                hipStream_t s);

// Elementwise rescale / cast / set_scaling of a contiguous array of n elements.
enum ScaleRule : int { RULE_AMAX = 0, RULE_KEEP = 1, RULE_FIXED = 2, RULE_COPY = 3 };
struct ElemParams {
  const void* in;
  void* out;
  int64_t n;
  int rule;          // RULE_AMAX: from hdr amax; RULE_KEEP: e_out = e_in; RULE_FIXED: e_out = e_fixed;
                     // RULE_COPY: shift 0 and the raw input scale value is copied
  int target, sat, e_fixed;
  const uint32_t* hdr;      // RULE_AMAX / RULE_KEEP (e_in snapshot); may be NULL otherwise
  const float* in_scale;    // read directly when hdr is NULL
  float* out_scale;
};
hipError_t launch_amax(const void* in, int in_dtype, int64_t n, uint32_t* hdr, hipStream_t s);
hipError_t launch_elementwise(const ElemParams& p, int in_dtype, int out_dtype, hipStream_t s);

}  // namespace scalify
