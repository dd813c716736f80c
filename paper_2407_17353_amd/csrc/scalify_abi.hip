// C ABI of the scaled-FP8 matmul library: argument validation on the host,
// the propagation rule table (exponent arithmetic only), workspace sizing and
// the launch sequence of each entry point. See include/scalify.h.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <stdlib.h>

#include <mutex>

#include "../../include/scalify.h"
#include "kernels.h"
#include "layernorm.h"

using namespace scalify;

namespace {

bool is_fp8(int32_t d) { return d == SCALIFY_E4M3 || d == SCALIFY_E5M2; }
bool is_out(int32_t d) { return d == SCALIFY_E4M3 || d == SCALIFY_E5M2 || d == SCALIFY_F16; }
bool is_any(int32_t d) { return d >= SCALIFY_E4M3 && d <= SCALIFY_F32; }
int64_t elem_bytes(int32_t d) { return d == SCALIFY_F32 ? 4 : (d == SCALIFY_F16 ? 2 : 1); }
bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }
int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

constexpr int64_t kMaxDim = (int64_t)1 << 30;

// Stored rows of a matrix and the byte extent of its storage.
int64_t stored_rows(const scalify_scaled_array* x) { return x->trans ? x->cols : x->rows; }
int64_t stored_cols(const scalify_scaled_array* x) { return x->trans ? x->rows : x->cols; }

scalify_status check_matrix(const scalify_scaled_array* x, int64_t ld_multiple) {
  if (x->rows < 0 || x->cols < 0 || x->rows > kMaxDim || x->cols > kMaxDim) return SCALIFY_ERR_SHAPE;
  if (x->trans != 0 && x->trans != 1) return SCALIFY_ERR_LAYOUT;
  if (x->rows == 0 || x->cols == 0) return SCALIFY_OK;
  if (x->data == nullptr) return SCALIFY_ERR_NULL;
  if (x->ld < stored_cols(x)) return SCALIFY_ERR_SHAPE;
  if (x->ld % ld_multiple != 0 || !aligned16(x->data)) return SCALIFY_ERR_ALIGN;
  return SCALIFY_OK;
}

// fused: the call fuses a residual add or an activation, or exports pre_out;
// its intermediate is then fp32 (exact for every pre-cast value, fp32
// subnormals included).
size_t matmul_ws(int64_t M, int64_t N, int32_t out_dtype, int32_t rescale, bool fused) {
  if (M < 0 || N < 0 || !is_out(out_dtype) || rescale < SCALIFY_RESCALE_NONE ||
      rescale > SCALIFY_RESCALE_DELAYED)
    return 0;
  // DELAYED and NONE: codes written by the GEMM (the output scale is known
  // before it runs)
  if (rescale != SCALIFY_RESCALE_AMAX) return kHeaderBytes;
  const size_t bytes = (out_dtype == SCALIFY_F16 || fused) ? 4u : 2u;
  return kHeaderBytes + (size_t)M * (size_t)round_up(N, 16) * bytes;
}

// The single pass of the dynamic rescale (GEMM, grid barrier on the
// statistic, cast: one kernel) where every workgroup of the persistent grid
// holds one tile (no intermediate at all: it is faster there), the GEMM +
// cast kernel pair otherwise (the earlier tiles' intermediate, cast by the
// 4 waves of a CU after the barrier, is slower than the cast kernel).
// SCALIFY_SINGLE_PASS=1 takes the single pass wherever it can run, 0 never.
bool single_pass_choice(int64_t tiles, int grid) {
  const char* v = getenv("SCALIFY_SINGLE_PASS");
  if (v && v[0] == '1' && v[1] == 0) return true;
  if (v && v[0] == '0' && v[1] == 0) return false;
  return tiles <= grid;
}

// The 4-wave kernel is persistent (one workgroup per CU walks its tiles)
// unless SCALIFY_PERSISTENT=0, which launches one workgroup per tile (and
// then no single pass, whose barrier needs the grid co-resident).
bool persistent_enabled() {
  const char* v = getenv("SCALIFY_PERSISTENT");
  return !(v && v[0] == '0' && v[1] == 0);
}

// Wait budget of the single pass's grid barrier, in ticks of the 100 MHz
// real-time counter: far beyond the arrival skew of a co-resident grid (at
// most one tile's main loop, about a microsecond per 128-deep k-step, plus
// its epilogue): 20 ms + 4 us per k-step. SCALIFY_SPIN_TICKS overrides it
// (0: a workgroup that is not the last to arrive gives up at once, which
// exercises the recovery of a grid that is not co-resident).
int64_t spin_ticks(int64_t K) {
  const char* v = getenv("SCALIFY_SPIN_TICKS");
  if (v && v[0]) return strtoll(v, nullptr, 10);
  return 2000000 + 400 * ((K + 127) / 128);
}

bool is_fused(const scalify_matmul_opts* o) {
  return o->residual != nullptr || o->activation != SCALIFY_ACT_NONE || o->pre_out != nullptr ||
         o->a_channel_scale != nullptr || o->b_channel_scale != nullptr;
}

bool has_mx(const scalify_matmul_opts* o) {
  return o->a_block_scale != nullptr || o->b_block_scale != nullptr;
}

// Calls whose pre-cast value may be any fp32 (fused epilogues, block
// scales) keep an fp32 intermediate.
bool f32_intermediate(const scalify_matmul_opts* o) { return is_fused(o) || has_mx(o); }

// Residual of the fused scaled add: M x N, row-major, ld = 0 (one row for
// every row) or ld >= N; the very same matrix as out, or disjoint from it.
scalify_status check_residual(const scalify_scaled_array* r, const scalify_scaled_array* out,
                              int64_t M, int64_t N) {
  if (!is_out(r->dtype)) return SCALIFY_ERR_DTYPE;
  if (r->rows != M || r->cols != N) return SCALIFY_ERR_SHAPE;
  if (r->trans != 0) return SCALIFY_ERR_LAYOUT;
  if (M == 0 || N == 0) return SCALIFY_OK;
  if (r->data == nullptr) return SCALIFY_ERR_NULL;
  if (r->ld != 0 && r->ld < N) return SCALIFY_ERR_SHAPE;
  if (r->ld % (r->dtype == SCALIFY_F16 ? 8 : 16) != 0 || !aligned16(r->data)) return SCALIFY_ERR_ALIGN;
  const uintptr_t r0 = (uintptr_t)r->data;
  const uintptr_t r1 = r0 + (uintptr_t)(((r->ld ? (M - 1) * r->ld : 0) + N) * elem_bytes(r->dtype));
  const uintptr_t o0 = (uintptr_t)out->data;
  const uintptr_t o1 = o0 + (uintptr_t)(((M - 1) * out->ld + N) * elem_bytes(out->dtype));
  const bool same = r->data == out->data && r->dtype == out->dtype && r->ld == out->ld;
  if (r0 < o1 && o0 < r1 && !same) return SCALIFY_ERR_LAYOUT;
  return SCALIFY_OK;
}

scalify_status check_elementwise(const scalify_scaled_array* in, const scalify_scaled_array* out) {
  if (!in || !out) return SCALIFY_ERR_NULL;
  if (!out->scale) return SCALIFY_ERR_NULL;
  if (!is_any(in->dtype) || !is_out(out->dtype)) return SCALIFY_ERR_DTYPE;
  if (in->rows < 0 || in->cols < 0 || in->rows > kMaxDim || in->cols > kMaxDim) return SCALIFY_ERR_SHAPE;
  if (in->rows != out->rows || in->cols != out->cols) return SCALIFY_ERR_SHAPE;
  if (in->trans != out->trans || (in->trans != 0 && in->trans != 1)) return SCALIFY_ERR_LAYOUT;
  const int64_t n = in->rows * in->cols;
  if (n == 0) return SCALIFY_OK;
  if (!in->data || !out->data) return SCALIFY_ERR_NULL;
  if (in->ld != stored_cols(in) || out->ld != stored_cols(out)) return SCALIFY_ERR_LAYOUT;
  if (!aligned16(in->data) || !aligned16(out->data)) return SCALIFY_ERR_ALIGN;
  // Aliasing: allowed only as the very same buffer with the same element size.
  const uintptr_t i0 = (uintptr_t)in->data, i1 = i0 + (uintptr_t)(n * elem_bytes(in->dtype));
  const uintptr_t o0 = (uintptr_t)out->data, o1 = o0 + (uintptr_t)(n * elem_bytes(out->dtype));
  if (i0 < o1 && o0 < i1 && !(i0 == o0 && elem_bytes(in->dtype) == elem_bytes(out->dtype)))
    return SCALIFY_ERR_LAYOUT;
  return SCALIFY_OK;
}

// A LayerNorm operand: R x D, row-major (trans = 0), 1 <= D <= 8192 when
// R > 0, rows 16-byte aligned (ld a multiple of 16 bytes), ld >= D.
scalify_status check_rows(const scalify_scaled_array* x, int64_t R, int64_t D) {
  if (x->rows != R || x->cols != D) return SCALIFY_ERR_SHAPE;
  if (x->trans != 0) return SCALIFY_ERR_LAYOUT;
  if (R == 0) return SCALIFY_OK;
  if (x->data == nullptr) return SCALIFY_ERR_NULL;
  if (x->ld < D) return SCALIFY_ERR_SHAPE;
  if ((x->ld * elem_bytes(x->dtype)) % 16 != 0 || !aligned16(x->data)) return SCALIFY_ERR_ALIGN;
  return SCALIFY_OK;
}

// An output may be the very same matrix as an input (same data, element
// size and ld: every row is read before it is written, by one workgroup),
// or must not overlap it.
bool rows_conflict(const scalify_scaled_array* a, const scalify_scaled_array* b, int64_t R,
                   int64_t D) {
  if (R == 0 || D == 0) return false;
  const uintptr_t a0 = (uintptr_t)a->data;
  const uintptr_t a1 = a0 + (uintptr_t)(((R - 1) * a->ld + D) * elem_bytes(a->dtype));
  const uintptr_t b0 = (uintptr_t)b->data;
  const uintptr_t b1 = b0 + (uintptr_t)(((R - 1) * b->ld + D) * elem_bytes(b->dtype));
  const bool same = a->data == b->data && elem_bytes(a->dtype) == elem_bytes(b->dtype) &&
                    a->ld == b->ld;
  return a0 < b1 && b0 < a1 && !same;
}

// ---- allocation-free matmul: its workspace is this file-scope device array
// (header + pre-cast intermediate), one copy per GPU the library runs on,
// held until the process ends. In host code `scratch` names a host-side
// stand-in; its device address, different on every GPU, comes from
// hipGetSymbolAddress with that GPU current and is the only form passed on.
constexpr size_t kNoallocScratchBytes = kHeaderBytes + ((size_t)32 << 20);
static __device__ __align__(256) uint8_t scratch[kNoallocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices];

// Device address of the current GPU's scratch array (looked up on the first
// call made with that GPU current, then kept).
scalify_status current_scratch(void** ptr) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return SCALIFY_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr)
      return SCALIFY_ERR_HIP;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return SCALIFY_OK;
}

size_t layernorm_bwd_ws(int64_t R, int64_t D) {
  if (R < 0 || D < 0 || D > kLayerNormMaxD || R > kMaxDim) return 0;
  return kHeaderBytes + (size_t)layernorm_ws_floats(R, D) * sizeof(float);
}

}  // namespace

extern "C" {

int64_t scalify_mx_packed_bytes(int64_t rows, int64_t K) {
  if (rows < 1 || K < 1) return 0;
  return 256 * ((K + 127) / 128) * ((rows + 63) / 64);
}

scalify_status scalify_mx_pack_block_scales(const uint8_t* src, int64_t rows, int64_t K,
                                            int64_t src_ld, uint8_t* dst, void* stream) {
  if (rows < 0 || K < 0 || rows > kMaxDim || K > kMaxDim) return SCALIFY_ERR_SHAPE;
  if (rows == 0 || K == 0) return SCALIFY_OK;
  if (!src || !dst) return SCALIFY_ERR_NULL;
  if (src_ld < (K + 31) / 32 || scalify_mx_packed_bytes(rows, K) >= ((int64_t)1 << 32) ||
      rows * src_ld >= ((int64_t)1 << 32))
    return SCALIFY_ERR_SHAPE;
  if ((uintptr_t)dst & 3u) return SCALIFY_ERR_ALIGN;
  return launch_mx_pack(src, (int)rows, (int)K, (int)src_ld, dst, (hipStream_t)stream) == hipSuccess
             ? SCALIFY_OK
             : SCALIFY_ERR_HIP;
}

int32_t scalify_matmul_scale_log2(int64_t K) {
  // Largest e with 2^e <= sqrt(K), i.e. 4^e <= K (integer arithmetic only).
  int32_t e = 0;
  if (K < 1) return 0;
  while (e < 31 && ((int64_t)1 << (2 * (e + 1))) <= K) ++e;
  return e;
}

size_t scalify_matmul_workspace_size(int64_t M, int64_t N, int32_t out_dtype, int32_t rescale) {
  return matmul_ws(M, N, out_dtype, rescale, false);
}

size_t scalify_matmul_workspace_size_opts(int64_t M, int64_t N, const scalify_matmul_opts* opts) {
  if (!opts) return 0;
  return matmul_ws(M, N, opts->out_dtype, opts->rescale, f32_intermediate(opts));
}

size_t scalify_rescale_workspace_size(int64_t n) { return n < 0 ? 0 : kHeaderBytes; }

const char* scalify_status_string(int32_t s) {
  switch (s) {
    case SCALIFY_OK: return "ok";
    case SCALIFY_ERR_NULL: return "null pointer";
    case SCALIFY_ERR_DTYPE: return "unsupported dtype";
    case SCALIFY_ERR_SHAPE: return "bad shape";
    case SCALIFY_ERR_LAYOUT: return "unsupported layout or aliasing";
    case SCALIFY_ERR_ALIGN: return "misaligned pointer or leading dimension";
    case SCALIFY_ERR_WORKSPACE: return "workspace missing or too small";
    case SCALIFY_ERR_VALUE: return "scalar argument out of range";
    case SCALIFY_ERR_HIP: return "HIP launch failed";
    default: return "unknown status";
  }
}

scalify_status scalify_matmul(const scalify_scaled_array* a, const scalify_scaled_array* b,
                              scalify_scaled_array* out, const scalify_matmul_opts* opts,
                              void* workspace, size_t workspace_bytes, void* stream) {
  if (!a || !b || !out || !opts) return SCALIFY_ERR_NULL;
  if (!out->scale) return SCALIFY_ERR_NULL;
  if (!is_fp8(a->dtype) || !is_fp8(b->dtype) || !is_out(opts->out_dtype) ||
      out->dtype != opts->out_dtype)
    return SCALIFY_ERR_DTYPE;
  if (opts->rescale < SCALIFY_RESCALE_NONE || opts->rescale > SCALIFY_RESCALE_DELAYED)
    return SCALIFY_ERR_VALUE;
  if (opts->rescale == SCALIFY_RESCALE_DELAYED && !opts->amax_in) return SCALIFY_ERR_NULL;
  if (opts->target_log2 < -1000 || opts->target_log2 > 1000) return SCALIFY_ERR_VALUE;
  if (opts->activation < SCALIFY_ACT_NONE || opts->activation > SCALIFY_ACT_SILU)
    return SCALIFY_ERR_VALUE;
  if (out->trans != 0) return SCALIFY_ERR_LAYOUT;
  const int64_t M = a->rows, K = a->cols, N = b->cols;
  if (b->rows != K || out->rows != M || out->cols != N) return SCALIFY_ERR_SHAPE;
  scalify_status st;
  if ((st = check_matrix(a, 16)) != SCALIFY_OK) return st;
  if ((st = check_matrix(b, 16)) != SCALIFY_OK) return st;
  if ((st = check_matrix(out, out->dtype == SCALIFY_F16 ? 8 : 16)) != SCALIFY_OK) return st;
  const scalify_scaled_array* res = opts->residual;
  if (res && (st = check_residual(res, out, M, N)) != SCALIFY_OK) return st;
  if (!aligned16(opts->b_channel_scale) || ((uintptr_t)opts->a_channel_scale & 3u))
    return SCALIFY_ERR_ALIGN;
  const bool fused = is_fused(opts);
  const bool mx = has_mx(opts);
  const int64_t mx_a_bytes = scalify_mx_packed_bytes(M, K), mx_b_bytes = scalify_mx_packed_bytes(N, K);
  if (mx) {
    // an array of no bytes (M, N or K zero) may be NULL
    if ((!opts->a_block_scale && M * K > 0) || (!opts->b_block_scale && N * K > 0))
      return SCALIFY_ERR_NULL;
    if (fused) return SCALIFY_ERR_VALUE;
    if (((uintptr_t)opts->a_block_scale | (uintptr_t)opts->b_block_scale) & 3u)
      return SCALIFY_ERR_ALIGN;
    if (mx_a_bytes >= ((int64_t)1 << 32) || mx_b_bytes >= ((int64_t)1 << 32)) return SCALIFY_ERR_SHAPE;
  }
  // 32-bit byte offsets inside the GEMM kernel, including the range-checked
  // reads of up to one tile past the last stored row.
  if (M && K && (stored_rows(a) + 256) * a->ld + 256 >= ((int64_t)1 << 32)) return SCALIFY_ERR_SHAPE;
  if (K && N && (stored_rows(b) + 256) * b->ld + 256 >= ((int64_t)1 << 32)) return SCALIFY_ERR_SHAPE;
  const size_t need = matmul_ws(M, N, opts->out_dtype, opts->rescale, fused || mx);
  if (!workspace || workspace_bytes < need || ((uintptr_t)workspace & 255u))
    return SCALIFY_ERR_WORKSPACE;

  hipStream_t s = (hipStream_t)stream;
  uint32_t* hdr = (uint32_t*)workspace;
  const int e_c = scalify_matmul_scale_log2(K);
  const bool amax_mode = opts->rescale == SCALIFY_RESCALE_AMAX;
  const bool delayed = opts->rescale == SCALIFY_RESCALE_DELAYED;
  // Delayed or no rescale: the output scale is known before the GEMM runs
  // (from the statistic of an earlier call, or the propagated scale itself),
  // so the GEMM casts straight to codes (no intermediate). Dynamic rescale:
  // the GEMM writes a pre-cast intermediate: 16-bit for FP8 outputs of the
  // plain epilogue, fp32 for FP16 outputs, for fused epilogues and with
  // block scales (whose accumulators may be fp32 subnormals, which the
  // 16-bit encoding does not keep exactly); the single pass keeps each
  // workgroup's last tile out of it and casts in the same kernel.
  const int epi = !amax_mode ? EPI_DIRECT
                             : ((opts->out_dtype == SCALIFY_F16 || fused || mx) ? EPI_INTER32
                                                                                 : EPI_INTER16);
  const bool tn_mx = mx && a->trans != 0 && b->trans == 0;  // 8-wave kernel
  // (the 4-wave block-scaled kernel casts only in the single pass)
  const bool persistent = persistent_enabled();
  const int64_t tiles = ((M + 255) / 256) * ((N + 255) / 256);
  const int grid = persistent ? gemm4_grid((int)tiles) : (int)tiles;
  const bool single_pass =
      amax_mode && !fused && !tn_mx && persistent && single_pass_choice(tiles, grid);
  // Exponent offset of the statistic: the matmul data is acc * 2^-e_c; with
  // a residual the statistic is taken over w itself.
  const int e_cc = res ? 0 : e_c;

  MatmulPrologue pq = {};
  pq.s0 = a->scale;
  pq.s1 = b->scale;
  pq.s_res = res ? res->scale : nullptr;
  pq.residual = res ? 1 : 0;
  pq.e_c = e_c;
  pq.direct = epi == EPI_DIRECT ? 1 : 0;
  pq.amax_in = delayed ? opts->amax_in : nullptr;
  pq.target = opts->target_log2;
  pq.out_scale = out->scale;
  if (launch_matmul_prologue(hdr, pq, s) != hipSuccess) return SCALIFY_ERR_HIP;

  GemmParams p = {};
  p.a = (const uint8_t*)a->data;
  p.b = (const uint8_t*)b->data;
  p.lda = a->ld;
  p.ldb = b->ld;
  p.M = (int)M;
  p.N = (int)N;
  p.K = (int)K;
  p.tiles_m = (int)((M + 255) / 256);
  p.tiles_n = (int)((N + 255) / 256);
  p.a_bytes = (uint32_t)(stored_rows(a) * a->ld);
  p.b_bytes = (uint32_t)(stored_rows(b) * b->ld);
  p.e_c = e_c;
  p.sat = opts->saturate != 0;
  p.hdr = hdr;
  p.inter = (uint8_t*)workspace + kHeaderBytes;
  p.ldw = round_up(N, 16);
  p.acc_out = opts->acc_out;
  p.out = out->data;
  p.ldc = out->ld;
  p.out_fmt = opts->out_dtype;
  p.res = res && M > 0 && N > 0 ? res->data : nullptr;
  p.ldr = res ? res->ld : 0;
  p.res_fmt = res ? res->dtype : 0;
  p.act = opts->activation;
  p.pre_out = opts->pre_out;
  p.ch_a = opts->a_channel_scale;
  p.ch_b = opts->b_channel_scale;
  // (the block-scale kernels run whenever the product has terms: K > 0)
  p.mx_a = mx && K > 0 ? opts->a_block_scale : nullptr;
  p.mx_b = mx && K > 0 ? opts->b_block_scale : nullptr;
  p.mx_groups_a = (int)((M + 63) / 64);
  p.mx_groups_b = (int)((N + 63) / 64);
  p.mx_a_bytes = (uint32_t)mx_a_bytes;
  p.mx_b_bytes = (uint32_t)mx_b_bytes;
  p.grid = grid;
  p.single_pass = single_pass ? 1 : 0;
  p.target = opts->target_log2;
  p.out_scale = out->scale;
  p.amax_out = opts->amax_out;
  p.spin_ticks = spin_ticks(K);
  hipEvent_t* ev = (hipEvent_t*)opts->events;
  if (ev && ev[0] && hipEventRecord(ev[0], s) != hipSuccess) return SCALIFY_ERR_HIP;
  if (M > 0 && N > 0) {
    if (launch_gemm(p, a->trans != 0, b->trans != 0, a->dtype, b->dtype, epi, fused, s) !=
        hipSuccess)
      return SCALIFY_ERR_HIP;
  }
  if (ev && ev[1] && hipEventRecord(ev[1], s) != hipSuccess) return SCALIFY_ERR_HIP;
  if (epi == EPI_DIRECT) {
    // The statistic this call records (for the next one, when delayed).
    if (opts->amax_out && launch_finalize_amax(hdr, e_cc, opts->amax_out, s) != hipSuccess)
      return SCALIFY_ERR_HIP;
  } else if (single_pass) {
    // The GEMM has cast the output and written its scale and statistic; with
    // nothing to compute (an empty output) they are written here.
    if (M == 0 || N == 0) {
      EpilogueParams q = {};
      q.M = 0;
      q.N = (int)N;
      q.e_c = e_cc;
      q.target = opts->target_log2;
      q.mode = 1;
      q.hdr = hdr;
      q.out_scale = out->scale;
      q.amax_out = opts->amax_out;
      if (launch_epilogue_cast(q, epi == EPI_INTER32, opts->out_dtype, s) != hipSuccess)
        return SCALIFY_ERR_HIP;
    }
  } else {
    // Second pass of the two-kernel dynamic rescale: global amax -> rescale
    // exponent -> output scale, and the cast of the intermediate.
    EpilogueParams q = {};
    q.inter = p.inter;
    q.ldw = p.ldw;
    q.out = out->data;
    q.ldc = out->ld;
    q.M = N > 0 ? (int)M : 0;
    q.N = (int)N;
    q.e_c = e_cc;
    q.target = opts->target_log2;
    q.sat = p.sat;
    q.mode = 1;
    q.hdr = hdr;
    q.out_scale = out->scale;
    q.amax_out = opts->amax_out;
    if (launch_epilogue_cast(q, epi == EPI_INTER32, opts->out_dtype, s) != hipSuccess)
      return SCALIFY_ERR_HIP;
  }
  if (ev && ev[2] && hipEventRecord(ev[2], s) != hipSuccess) return SCALIFY_ERR_HIP;
  return SCALIFY_OK;
}

scalify_status scalify_matmul_noalloc(const scalify_scaled_array* a,
                                      const scalify_scaled_array* b, scalify_scaled_array* out,
                                      const scalify_matmul_opts* opts, void* stream) {
  if (!a || !b || !out || !opts) return SCALIFY_ERR_NULL;
  // A workspace larger than the array is refused before anything is enqueued
  // (scalify_matmul checks the other arguments first and returns their error).
  void* ws = nullptr;
  const scalify_status st = current_scratch(&ws);
  if (st != SCALIFY_OK) return st;
  return scalify_matmul(a, b, out, opts, ws, kNoallocScratchBytes, stream);
}

scalify_status scalify_rescale(const scalify_scaled_array* in, scalify_scaled_array* out,
                               int32_t mode, int32_t target_log2, int32_t saturate,
                               void* workspace, size_t workspace_bytes, void* stream) {
  scalify_status st = check_elementwise(in, out);
  if (st != SCALIFY_OK) return st;
  if (mode != SCALIFY_RESCALE_NONE && mode != SCALIFY_RESCALE_AMAX) return SCALIFY_ERR_VALUE;
  if (target_log2 < -1000 || target_log2 > 1000) return SCALIFY_ERR_VALUE;
  if (!workspace || workspace_bytes < kHeaderBytes || ((uintptr_t)workspace & 255u))
    return SCALIFY_ERR_WORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  uint32_t* hdr = (uint32_t*)workspace;
  const int64_t n = in->rows * in->cols;
  if (launch_prologue(hdr, in->scale, nullptr, s) != hipSuccess) return SCALIFY_ERR_HIP;
  if (mode == SCALIFY_RESCALE_AMAX && n > 0)
    if (launch_amax(in->data, in->dtype, n, hdr, s) != hipSuccess) return SCALIFY_ERR_HIP;
  ElemParams p = {};
  p.in = in->data;
  p.out = out->data;
  p.n = n;
  p.rule = mode == SCALIFY_RESCALE_AMAX ? RULE_AMAX : RULE_KEEP;
  p.target = target_log2;
  p.sat = saturate != 0;
  p.hdr = hdr;
  p.in_scale = in->scale;
  p.out_scale = out->scale;
  if (launch_elementwise(p, in->dtype, out->dtype, s) != hipSuccess) return SCALIFY_ERR_HIP;
  return SCALIFY_OK;
}

scalify_status scalify_cast(const scalify_scaled_array* in, scalify_scaled_array* out,
                            int32_t saturate, void* stream) {
  scalify_status st = check_elementwise(in, out);
  if (st != SCALIFY_OK) return st;
  ElemParams p = {};
  p.in = in->data;
  p.out = out->data;
  p.n = in->rows * in->cols;
  p.rule = RULE_COPY;
  p.sat = saturate != 0;
  p.in_scale = in->scale;
  p.out_scale = out->scale;
  if (launch_elementwise(p, in->dtype, out->dtype, (hipStream_t)stream) != hipSuccess)
    return SCALIFY_ERR_HIP;
  return SCALIFY_OK;
}

scalify_status scalify_set_scaling(const scalify_scaled_array* in, scalify_scaled_array* out,
                                   int32_t new_scale_log2, int32_t saturate, void* stream) {
  scalify_status st = check_elementwise(in, out);
  if (st != SCALIFY_OK) return st;
  if (new_scale_log2 < -127 || new_scale_log2 > 127) return SCALIFY_ERR_VALUE;
  if (in->scale != nullptr && in->scale == out->scale) return SCALIFY_ERR_LAYOUT;
  ElemParams p = {};
  p.in = in->data;
  p.out = out->data;
  p.n = in->rows * in->cols;
  p.rule = RULE_FIXED;
  p.e_fixed = new_scale_log2;
  p.sat = saturate != 0;
  p.in_scale = in->scale;
  p.out_scale = out->scale;
  if (launch_elementwise(p, in->dtype, out->dtype, (hipStream_t)stream) != hipSuccess)
    return SCALIFY_ERR_HIP;
  return SCALIFY_OK;
}

scalify_status scalify_layernorm_fwd(const scalify_scaled_array* x, const float* gamma,
                                     const float* beta, float eps, scalify_scaled_array* out,
                                     int32_t saturate, float* pre_out, void* stream) {
  if (!x || !out) return SCALIFY_ERR_NULL;
  if (!out->scale) return SCALIFY_ERR_NULL;
  if (!is_any(x->dtype) || !is_out(out->dtype)) return SCALIFY_ERR_DTYPE;
  const int64_t R = x->rows, D = x->cols;
  if (R < 0 || D < 0 || R > kMaxDim) return SCALIFY_ERR_SHAPE;
  if (R > 0 && (D < 1 || D > kLayerNormMaxD)) return SCALIFY_ERR_SHAPE;
  if (!(eps >= 0.0f) || !(eps < 3.0e38f)) return SCALIFY_ERR_VALUE;
  if (!aligned16(gamma) || !aligned16(beta) || !aligned16(pre_out)) return SCALIFY_ERR_ALIGN;
  scalify_status st;
  if ((st = check_rows(x, R, D)) != SCALIFY_OK) return st;
  if ((st = check_rows(out, R, D)) != SCALIFY_OK) return st;
  if (rows_conflict(x, out, R, D)) return SCALIFY_ERR_LAYOUT;
  LnParams p = {};
  p.x = x->data;
  p.ldx = x->ld;
  p.x_fmt = x->dtype;
  p.gamma = gamma;
  p.beta = beta;
  p.out = out->data;
  p.ldo = out->ld;
  p.pre_out = pre_out;
  p.R = R;
  p.D = (int)D;
  p.eps = eps;
  p.sat = saturate != 0;
  p.out_scale = out->scale;
  if (launch_layernorm_fwd(p, out->dtype, (hipStream_t)stream) != hipSuccess)
    return SCALIFY_ERR_HIP;
  return SCALIFY_OK;
}

size_t scalify_layernorm_bwd_workspace_size(int64_t R, int64_t D) { return layernorm_bwd_ws(R, D); }

scalify_status scalify_layernorm_bwd(const scalify_scaled_array* dy, const scalify_scaled_array* x,
                                     const float* gamma, float eps, scalify_scaled_array* dx,
                                     float* dgamma, float* dbeta, int32_t rescale,
                                     int32_t target_log2, int32_t saturate, float* amax_out,
                                     float* pre_out, void* workspace, size_t workspace_bytes,
                                     void* stream) {
  if (!dy || !x || !dx) return SCALIFY_ERR_NULL;
  if (!dx->scale) return SCALIFY_ERR_NULL;
  if (!is_any(dy->dtype) || !is_any(x->dtype) || !is_out(dx->dtype)) return SCALIFY_ERR_DTYPE;
  if (rescale != SCALIFY_RESCALE_NONE && rescale != SCALIFY_RESCALE_AMAX) return SCALIFY_ERR_VALUE;
  if (target_log2 < -1000 || target_log2 > 1000) return SCALIFY_ERR_VALUE;
  if (!(eps >= 0.0f) || !(eps < 3.0e38f)) return SCALIFY_ERR_VALUE;
  const int64_t R = x->rows, D = x->cols;
  if (R < 0 || D < 0 || R > kMaxDim) return SCALIFY_ERR_SHAPE;
  if (R > 0 && (D < 1 || D > kLayerNormMaxD)) return SCALIFY_ERR_SHAPE;
  if (!aligned16(gamma) || !aligned16(dgamma) || !aligned16(dbeta) || !aligned16(pre_out))
    return SCALIFY_ERR_ALIGN;
  scalify_status st;
  if ((st = check_rows(x, R, D)) != SCALIFY_OK) return st;
  if ((st = check_rows(dy, R, D)) != SCALIFY_OK) return st;
  if ((st = check_rows(dx, R, D)) != SCALIFY_OK) return st;
  if (rows_conflict(dx, dy, R, D) || rows_conflict(dx, x, R, D)) return SCALIFY_ERR_LAYOUT;
  const size_t need = layernorm_bwd_ws(R, D);
  if (!workspace || workspace_bytes < need || ((uintptr_t)workspace & 255u))
    return SCALIFY_ERR_WORKSPACE;
  LnParams p = {};
  p.x = x->data;
  p.ldx = x->ld;
  p.x_fmt = x->dtype;
  p.dy = dy->data;
  p.lddy = dy->ld;
  p.dy_fmt = dy->dtype;
  p.gamma = gamma;
  p.out = dx->data;
  p.ldo = dx->ld;
  p.pre_out = pre_out;
  p.R = R;
  p.D = (int)D;
  p.eps = eps;
  p.sat = saturate != 0;
  p.target = target_log2;
  p.mode = rescale == SCALIFY_RESCALE_AMAX ? 1 : 0;
  p.hdr = (uint32_t*)workspace;
  p.partial = (float*)((uint8_t*)workspace + kHeaderBytes);
  p.out_scale = dx->scale;
  p.amax_out = amax_out;
  p.dgamma = dgamma;
  p.dbeta = dbeta;
  if (launch_layernorm_bwd(p, dy->scale, x->scale, dx->dtype, (hipStream_t)stream) != hipSuccess)
    return SCALIFY_ERR_HIP;
  return SCALIFY_OK;
}

}  // extern "C"
