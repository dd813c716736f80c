/*
 * scalify.h - C ABI of the MI355X (gfx950) scaled-FP8 matmul library.
 *
 * Implements the hot path of Scalify's scale propagation (Balanca et al.,
 * "Scalify: scale propagation for efficient low-precision LLM training",
 * arXiv 2407.17353):
 *   - a ScaledArray is a pair (data X_d, scale X_s) with X = X_d * X_s, where
 *     X_s is a power of two held in one fp32 (Section 2; Section 3.1,
 *     Algorithm 2);
 *   - the scaled matmul propagates the output scale s_a * s_b * c with
 *     c = sqrt(K) rounded DOWN to a power of two, dividing the data by c
 *     (Section 3.2, Algorithm 3: static rule from scales and shapes under the
 *     independent-Gaussian assumption; scales rounded down);
 *   - dynamic rescaling: statistic of the data -> power of two (rounded down)
 *     -> rebalance_scale (Section 3.3, Algorithm 4); the statistic is amax;
 *   - set_scaling and get_data_and_scale (Section 3.1);
 *   - casts act on the data component only (Appendix A, cast operators);
 *   - the scaled add and activation rules, fused into the matmul epilogue
 *     (Section 3.2, Algorithm 3; Appendix C.1), and the scaled LayerNorm with
 *     the dynamic rescale of its input gradient (Appendix C.2, Section 4);
 *   - FP8 formats E4M3 / E5M2 (Section 1, Appendix A; OCP encodings on gfx950)
 *     and FP16 (E5M10) outputs.
 *
 * Conventions for every entry point
 *   - All data and scale pointers are DEVICE pointers owned by the caller.
 *     The library allocates nothing and keeps no state between calls;
 *     concurrent calls are safe when they use distinct workspaces.
 *   - Work is enqueued on `stream` (a hipStream_t passed as void*, NULL = the
 *     default stream). No call synchronises the host or reads a scale back.
 *   - Argument errors are detected on the host before any launch; they return
 *     a status and leave every output untouched. A failed launch returns
 *     SCALIFY_ERR_HIP.
 *   - Numeric specials are not errors: NaN inputs give NaN outputs, amax
 *     ignores NaN, Inf amax or zero amax keep the propagated scale.
 *   - Preconditions not checked by the kernels: input scales are finite
 *     powers of two within the E8M0 range [2^-127, 2^127]. A NULL input scale
 *     means scale 1 (get_data_and_scale of an unscaled array, Section 3.1).
 */
#ifndef SCALIFY_H
#define SCALIFY_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    SCALIFY_OK = 0,
    SCALIFY_ERR_NULL = 1,      /* a required pointer is NULL */
    SCALIFY_ERR_DTYPE = 2,     /* unsupported data type or combination */
    SCALIFY_ERR_SHAPE = 3,     /* inconsistent or negative sizes */
    SCALIFY_ERR_LAYOUT = 4,    /* unsupported storage layout or aliasing */
    SCALIFY_ERR_ALIGN = 5,     /* data pointer or leading dimension not 16-byte aligned */
    SCALIFY_ERR_WORKSPACE = 6, /* workspace missing or too small */
    SCALIFY_ERR_VALUE = 7,     /* scalar argument out of range */
    SCALIFY_ERR_HIP = 8        /* a HIP launch failed */
} scalify_status;

typedef enum {
    SCALIFY_E4M3 = 0, /* OCP FP8 E4M3: bias 7, max 448, no Inf, NaN = S.1111.111 */
    SCALIFY_E5M2 = 1, /* OCP FP8 E5M2: bias 15, max 57344, Inf and NaN */
    SCALIFY_F16 = 2,  /* IEEE binary16 (E5M10) */
    SCALIFY_F32 = 3   /* IEEE binary32 (inputs of rescale / cast / set_scaling only) */
} scalify_dtype;

typedef enum {
    SCALIFY_RESCALE_NONE = 0,   /* static propagation rule only */
    SCALIFY_RESCALE_AMAX = 1,   /* dynamic power-of-two rescale from this call's amax */
    SCALIFY_RESCALE_DELAYED = 2 /* delayed rescale: from the amax an earlier call recorded */
} scalify_rescale_mode;

/* Activation applied by the matmul epilogue (Appendix C.1): f(x) = x * g(x)
 * with a gate g -> 0 at -inf and -> 1 at +inf; on a ScaledArray the scale
 * is kept and the data becomes X_d * g(X_d * X_s). */
typedef enum {
    SCALIFY_ACT_NONE = 0,
    SCALIFY_ACT_RELU = 1,      /* g = 1 for x > 0, else 0 */
    SCALIFY_ACT_GELU_TANH = 2, /* g = (1 + tanh(sqrt(2/pi) (x + 0.044715 x^3))) / 2 */
    SCALIFY_ACT_SILU = 3       /* g = 1 / (1 + exp(-x)) (swish) */
} scalify_activation;

/* A ScaledArray (Section 2, Section 3.1): value = decode(data) * (*scale).
 * Logical shape rows x cols.
 *   trans = 0: element (r, c) is stored at data[r * ld + c]  (ld >= cols)
 *   trans = 1: element (r, c) is stored at data[c * ld + r]  (ld >= rows)
 * The storage must hold every stored row in full: (stored rows) * ld
 * elements. `scale` points to ONE fp32 power of two on the device; NULL is
 * allowed for inputs (scale 1) and is an error for outputs. */
typedef struct {
    void* data;
    float* scale;
    int32_t dtype; /* scalify_dtype */
    int32_t trans;
    int64_t rows;
    int64_t cols;
    int64_t ld; /* in elements */
} scalify_scaled_array;

typedef struct {
    int32_t out_dtype;   /* SCALIFY_E4M3 | SCALIFY_E5M2 | SCALIFY_F16 */
    int32_t rescale;     /* scalify_rescale_mode */
    int32_t target_log2; /* t: AMAX puts the rescaled amax in [2^t, 2^(t+1)); default 0 */
    int32_t saturate;    /* 1: overflow and +-Inf -> +-max; 0: E4M3 -> NaN, E5M2/F16 -> +-Inf */
    float* acc_out;      /* optional device [M][N] fp32: the raw accumulator sum_k a_ik b_kj */
    float* amax_out;     /* optional device fp32: amax of acc * 2^-e_c over non-NaN elements
                            (with a fused add or activation: of the data the statistic is
                            gathered over, see scalify_matmul) */
    void** events;       /* optional host array of 3 hipEvent_t recorded on the stream: before
                            the GEMM kernel, after it, and after the epilogue cast (DELAYED:
                            after the amax write-back) -- timing of the fused GEMM without
                            host synchronisation; NULL = none, and a NULL entry skips
                            that record */
    const float* amax_in; /* DELAYED only (required there): device fp32 statistic recorded by
                            an earlier call (its amax_out); may be the same memory as
                            amax_out, it is read before this call writes its own */
    const scalify_scaled_array* residual; /* optional: R added to the product by the scaled
                            add rule before the activation (see scalify_matmul); E4M3, E5M2 or
                            F16, rows = M, cols = N, trans = 0, 16-byte aligned, ld a multiple
                            of 16 elements (8 for F16) and >= N, or ld = 0: one row added to
                            every row (a bias). It may be the very same matrix as out (same
                            data, dtype and ld) but must not otherwise overlap it. NULL = none */
    int32_t activation;  /* scalify_activation applied after the add; NONE = 0 */
    float* pre_out;      /* optional validation output: device fp32 [M][N], the value w the
                            rescale and cast see (after the add and the activation), whose
                            true value is w * 2^e_w (e_w as in scalify_matmul) */
    const float* a_channel_scale; /* optional channel scales of a (Section 2: a scale
                            broadcastable to the data; channel scaling): device fp32 [M],
                            one power of two (exponent in [-149, 127]) per row of the logical
                            a, i.e. per output row, on top of *a.scale; NULL = none */
    const float* b_channel_scale; /* optional: device fp32 [N], one power of two per column
                            of the logical b (per output column), on top of *b.scale,
                            16-byte aligned; NULL = none */
    const uint8_t* a_block_scale; /* optional MX block scales of a (Section 2: block
                            scaling formats such as MX as scales broadcastable to the
                            data): P, one E8M0 byte P[i][k / 32] (value 2^(byte - 127))
                            per 32 k of each row i of the logical a, scaling a[i,k] on
                            top of *a.scale, in the packed order that
                            scalify_mx_pack_block_scales writes (rows = M); device,
                            4-byte aligned; given together with b_block_scale;
                            NULL = none */
    const uint8_t* b_block_scale; /* Q, one byte Q[j][k / 32] per 32 k of each column j
                            of the logical b, packed likewise (rows = N); NULL = none */
} scalify_matmul_opts;

/* Bytes of the packed form of an MX block-scale array with `rows` rows (rows
 * of a, or columns of b) for depth K: 256 * ceil(K / 128) * ceil(rows / 64).
 * Returns 0 when rows or K is below 1. */
int64_t scalify_mx_packed_bytes(int64_t rows, int64_t K);

/* Pack MX block-scale bytes from the natural row-major order, src[r * src_ld
 * + b] for row r < rows and block b < ceil(K / 32) (src_ld >= ceil(K / 32)),
 * into the order the block-scaled matmul reads: for 128-k step t, 64-row
 * group q, k-block g in 0..3 and row r in 0..15 of the group's four 16-row
 * blocks, the 4 bytes of rows 64 q + r, + 16, + 32, + 48 at block 4 t + g
 * are the 32-bit word at byte offset ((t * ceil(rows / 64) + q) * 64 + 16 g
 * + r) * 4 of dst (lowest byte first). Blocks past ceil(K / 32) and rows
 * past `rows` are written as 127 (a factor of 1; they meet zero data).
 * dst: device, scalify_mx_packed_bytes(rows, K) bytes, 4-byte aligned,
 * not overlapping src. Pure data movement; enqueued on `stream`. Weights'
 * scales are packed once; an activation's producer can write this order
 * directly. Errors: SCALIFY_ERR_NULL (NULL src or dst with rows, K > 0),
 * SCALIFY_ERR_SHAPE (negative sizes, src_ld < ceil(K / 32), more than 2^32
 * bytes), SCALIFY_ERR_ALIGN (dst), SCALIFY_ERR_HIP. */
scalify_status scalify_mx_pack_block_scales(const uint8_t* src, int64_t rows, int64_t K,
                                            int64_t src_ld, uint8_t* dst, void* stream);

/* Exponent e_c of the matmul scale rule (Section 3.2, Algorithm 3): the
 * largest e with 2^e <= sqrt(K) (sqrt(K) rounded down to a power of two),
 * computed with integers. Returns 0 for K < 1. Host only. */
int32_t scalify_matmul_scale_log2(int64_t K);

/* Bytes of device workspace scalify_matmul needs for an M x N output with
 * the given output type and rescale mode: a 256-byte header plus, for AMAX,
 * the pre-cast intermediate (M rows of N rounded up to 16 elements; 2 bytes
 * per element for FP8 outputs, 4 for FP16). DELAYED and NONE, whose output
 * scale is known before the GEMM runs, need the header only. Returns 0 for
 * invalid arguments. */
size_t scalify_matmul_workspace_size(int64_t M, int64_t N, int32_t out_dtype, int32_t rescale);

/* Workspace bytes of a scalify_matmul call with these options: as above, but
 * an AMAX call that fuses a residual add or an activation, has channel or MX
 * block scales, or asks for pre_out, keeps an fp32 intermediate (4 bytes per
 * element for every output type).
 * Returns 0 for invalid arguments or a NULL opts. */
size_t scalify_matmul_workspace_size_opts(int64_t M, int64_t N, const scalify_matmul_opts* opts);

/* Scaled matmul on ScaledArray operands (Section 3.2, Algorithm 3; FP8
 * matmul with mixed input formats and higher-precision accumulation,
 * Appendix A), with the dynamic or delayed rescale (Section 3.3) fused:
 *   acc   = sum_k dec(a)[i,k] * dec(b)[k,j]        fp32 accumulation (MFMA)
 *   e_c   = scalify_matmul_scale_log2(K)
 *   AMAX: e_r = floor(log2 amax(acc * 2^-e_c)) - target_log2
 *         (0 when that amax is 0 or +Inf or every element is NaN)
 *   DELAYED: e_r = floor(log2 |*opts.amax_in|) - target_log2, the statistic
 *         of an earlier call (0 when it is 0, Inf or NaN); this call's amax
 *         (of acc * 2^-e_c) goes to opts.amax_out for the next call. Values
 *         the stale scale pushes past the format's range saturate (or
 *         overflow when saturate = 0). The GEMM writes the codes directly:
 *         no intermediate, no second pass over the output.
 *   NONE: e_r = 0 (the GEMM writes the codes directly, as for DELAYED)
 *   e_out = clamp(e_a + e_b + e_c + e_r, -127, 127)        (E8M0 range)
 *   out.data  = RNE(acc * 2^(e_a + e_b - e_out)) in out.dtype (saturating
 *               when opts.saturate), *out.scale = 2^e_out
 * so that dec(out) * s_out = s_a * s_b * acc up to the final rounding.
 *
 * Channel scales (opts.a_channel_scale = c, opts.b_channel_scale = d): a[i,k]
 * = dec(a)[i,k] * s_a * c[i], b[k,j] = dec(b)[k,j] * s_b * d[j]. The output
 * keeps one scalar scale: the channel factors go into the data as one
 * power-of-two product of acc (exact unless it leaves the fp32 range),
 * w = fl32(acc * c[i] * d[j]) in place of acc below (with a residual, the
 * product term is fl32(acc * 2^(e_a+e_b-e_w) * c[i] * d[j])); such a call
 * keeps an fp32 intermediate like a fused one.
 *
 * MX block scales (opts.a_block_scale = P, opts.b_block_scale = Q, both or
 * neither, each packed by scalify_mx_pack_block_scales): a[i,k] = dec(a)[i,k] * s_a * 2^(P[i][k/32] - 127), b[k,j] =
 * dec(b)[k,j] * s_b * 2^(Q[j][k/32] - 127): the matrix cores apply the block
 * factors to the products, acc = sum_k dec(a)[i,k] dec(b)[k,j]
 * 2^(P[i][k/32] + Q[j][k/32] - 254), and everything below acts on that acc
 * (the output keeps one scalar scale). The byte 0xFF (E8M0's NaN) is not a
 * scale: results of a call that uses one are unspecified. Block factors
 * that push products or partial sums out of fp32's normal range give what
 * the matrix cores give there (Inf, or subnormals and zeros). Such a call
 * keeps an fp32 intermediate; it cannot be combined with a residual, an
 * activation, pre_out or channel scales (SCALIFY_ERR_VALUE); one of the two
 * arrays alone is SCALIFY_ERR_NULL (an array of no bytes, M * K or N * K
 * zero, may be NULL), a pointer not 4-byte aligned SCALIFY_ERR_ALIGN.
 *
 * Fused scaled add and activation (opts.residual, opts.activation): the
 * epilogue first forms w, whose true value is w * 2^e_w, then rescales and
 * casts w in place of acc:
 *   no residual: w = acc, e_w = e_a + e_b, statistic over w * 2^-e_c;
 *   residual R (scale 2^q): scaled add (Algorithm 3) of the product, whose
 *     propagated scale is 2^(e_a+e_b+e_c), and R: the output scale is
 *     sqrt(s_p^2 + s_r^2) rounded down to a power of two, i.e. e_w =
 *     max(e_a + e_b + e_c, q); w = fl32(acc * 2^(e_a+e_b-e_w) + dec(R) * 2^(q-e_w))
 *     (one rounding of the sum), statistic over w;
 *   activation (Appendix C.1, after the add): w = fl32(w * g(w * 2^e_w)),
 *     scale unchanged; relu is exact, gelu and silu are evaluated in fp32
 *     (within a few ulp of the exact gate).
 *   Then e_out = clamp(e_w + (e_c, or 0 with a residual) + e_r) with e_r from
 *   the statistic of w (AMAX) or from amax_in (DELAYED), and
 *   out.data = RNE(w * 2^(e_w - e_out)); amax_out is that statistic.
 *
 * a: M x K, b: K x N, out: M x N. a and b are E4M3 or E5M2 in any mix and
 * either storage order (trans 0/1). out.trans must be 0 and out.dtype must
 * equal opts->out_dtype. All data pointers 16-byte aligned, every ld a
 * multiple of 16 elements (8 for an FP16 out). workspace: device memory of
 * at least scalify_matmul_workspace_size_opts(M, N, opts) bytes (for a call
 * with nothing fused: scalify_matmul_workspace_size(M, N, ...)), 256-byte aligned,
 * not shared with a concurrent call. Determinism: reruns are bit-identical.
 * M, N or K may be 0 (K = 0 gives an all-zero output).
 *
 * AMAX without a fused epilogue, on an output of at most one 256 x 256 tile
 * per compute unit, runs as one GEMM kernel (the single pass): its
 * workgroups hold their output tile in the matrix cores' accumulators, meet
 * at a grid barrier on the amax statistic, and cast; the output scale and
 * amax_out are written by that kernel. Larger outputs take the GEMM + cast
 * kernel pair (faster there). The barrier's wait is bounded: if the grid is
 * not co-resident on the GPU (other work occupies its compute units), the
 * workgroups fall back to casting from the intermediate after the wait, with
 * the same result, later. Environment (read at each call):
 * SCALIFY_SINGLE_PASS=1 takes the single pass at any size, =0 never (it
 * does not cover block-scaled calls with a.trans = 1 and b.trans = 0);
 * SCALIFY_SPIN_TICKS=<n> sets the barrier's wait in ticks of the
 * GPU's 100 MHz counter (default 20 ms plus 4 us per 128 of K; 0 exercises
 * the fallback). SCALIFY_PERSISTENT=0 launches one workgroup per tile (and no
 * single pass) instead of the persistent grid. */
scalify_status scalify_matmul(const scalify_scaled_array* a, const scalify_scaled_array* b,
                              scalify_scaled_array* out, const scalify_matmul_opts* opts,
                              void* workspace, size_t workspace_bytes, void* stream);

/* scalify_matmul for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same computation, arguments and statuses, with the workspace taken
 * from a static array of the library instead of the caller. The library
 * holds one such array of 256 + 32 MiB bytes on every GPU it runs on, from
 * the first call with that GPU current until the process ends; this call
 * allocates nothing itself. A call whose workspace size
 * (scalify_matmul_workspace_size_opts) exceeds 256 + 32 MiB returns
 * SCALIFY_ERR_WORKSPACE and enqueues nothing: DELAYED and NONE calls fit at
 * any size (header only); AMAX calls fit while M x round_up(N, 16) x (2 for
 * FP8 outputs, 4 for FP16 outputs and fused / channel / block-scaled calls)
 * <= 32 MiB, e.g. 4096 x 4096 FP8 outputs. Every call on one GPU shares its
 * array: calls that may overlap on one GPU (other streams, other host
 * threads) race and must be ordered by the caller. `stream` must belong to
 * the current GPU. The array keeps the last call's contents; each call
 * clears what it needs cleared. SCALIFY_ERR_HIP also when the array's
 * address cannot be obtained. */
scalify_status scalify_matmul_noalloc(const scalify_scaled_array* a,
                                      const scalify_scaled_array* b, scalify_scaled_array* out,
                                      const scalify_matmul_opts* opts, void* stream);

/* Bytes of device workspace scalify_rescale needs (a 256-byte header). */
size_t scalify_rescale_workspace_size(int64_t n);

/* Dynamic rescale of a ScaledArray (Section 3.3, Algorithm 4: statistic,
 * power of two rounded down, rebalance_scale), with a cast when out.dtype
 * differs from in.dtype:
 *   AMAX: e_r = floor(log2 amax(dec(in))) - target_log2 (0 for amax 0 / +Inf /
 *         all NaN); NONE: e_r = 0
 *   e_out = clamp(e_in + e_r, -127, 127); out.data = RNE(dec(in) * 2^(e_in - e_out))
 * in.dtype: any scalify_dtype; out.dtype: E4M3, E5M2 or F16. in and out have
 * the same shape and trans and are stored contiguously (ld = cols, or rows
 * when trans = 1). out may alias in only when both have the same element
 * size; out.scale may alias in.scale. workspace >= 256 bytes. */
scalify_status scalify_rescale(const scalify_scaled_array* in, scalify_scaled_array* out,
                               int32_t mode, int32_t target_log2, int32_t saturate,
                               void* workspace, size_t workspace_bytes, void* stream);

/* Cast of the data component only; the scale is copied (Appendix A cast
 * operators): out.data = RNE(dec(in)), *out.scale = *in.scale (1 if NULL).
 * Same layout rules as scalify_rescale. */
scalify_status scalify_cast(const scalify_scaled_array* in, scalify_scaled_array* out,
                            int32_t saturate, void* stream);

/* set_scaling (Section 3.1): the output gets scale 2^new_scale_log2 and the
 * data is rescaled by the ratio of the old and new scales:
 *   out.data = RNE(dec(in) * 2^(e_in - new_scale_log2)), *out.scale = 2^new_scale_log2.
 * new_scale_log2 in [-127, 127]. out.scale must not alias in.scale. Same
 * layout rules as scalify_rescale. */
scalify_status scalify_set_scaling(const scalify_scaled_array* in, scalify_scaled_array* out,
                                   int32_t new_scale_log2, int32_t saturate, void* stream);

/* Scaled LayerNorm forward (Appendix C.2): a mean-variance normalization is
 * invariant to the scale of its input up to its eps, so it normalizes the
 * data component and gives the output scale 1. Per row r of x (R x D):
 *   mean = sum_j x_d[r,j] / D,  std = sqrt(sum_j (x_d[r,j] - mean)^2 / D),
 *   y = (x_d - mean) / (std + eps) * gamma + beta,
 *   out.data = RNE(y) in out.dtype (saturating when saturate), *out.scale = 1.
 * x.dtype: any scalify_dtype (x.scale is not read); out.dtype: E4M3, E5M2 or
 * F16. Both R x D, row-major (trans = 0), rows 16-byte aligned (ld a
 * multiple of 16 bytes, ld >= D), 1 <= D <= 8192 (any D when R = 0). gamma,
 * beta: device fp32 [D], NULL = 1 and 0. eps >= 0 (ERR_VALUE otherwise). out
 * may be the very same matrix as x (same data, element size and ld) but must
 * not otherwise overlap it. pre_out: optional device fp32 [R][D] receiving y
 * before the cast (validation). The statistics are fp32 sums in a fixed
 * order: reruns are bit-identical. Rows of 2049 .. 4096 FP16 / FP8 elements
 * are read from HBM once (the backward's statistics too);
 * SCALIFY_LN_SINGLE_READ=0 (read at each call) selects the multi-pass
 * kernels instead, with the same results bit for bit. */
scalify_status scalify_layernorm_fwd(const scalify_scaled_array* x, const float* gamma,
                                     const float* beta, float eps, scalify_scaled_array* out,
                                     int32_t saturate, float* pre_out, void* stream);

/* Bytes of device workspace scalify_layernorm_bwd needs: a 256-byte header
 * plus min(R, 1024) x 2 x D fp32 partial parameter gradients. 0 for invalid
 * sizes (D > 8192). */
size_t scalify_layernorm_bwd_workspace_size(int64_t R, int64_t D);

/* Input gradient of scalify_layernorm_fwd with its dynamic rescale (the
 * LayerNorm backward rescale of the paper's experiments, Section 4, with the
 * rebalance of Section 3.3). The forward is a function of the data x_d =
 * X / X_s, so for an upstream gradient dY = dy_d * s_dy the input gradient is
 * the ScaledArray (dx, s_dy / s_x) with, per row (c = x_d - mean,
 * s = std + eps, xhat = c / s, g = dy_d * gamma):
 *   dx = (g - mean(g) - (c / std) mean(g * xhat)) / s   (last term 0 when std = 0).
 * AMAX: e_r = floor(log2 amax |dx|) - target_log2 (0 for amax 0 / Inf / all
 * NaN); NONE: e_r = 0. e_out = clamp(e(s_dy) - e(s_x) + e_r, -127, 127),
 * dx.data = RNE(dx * 2^(e(s_dy) - e(s_x) - e_out)), *dx.scale = 2^e_out.
 * dgamma[j] = sum_r dy_d[r,j] xhat[r,j] and dbeta[j] = sum_r dy_d[r,j]
 * (optional device fp32 [D]; their true values are these times s_dy);
 * amax_out: optional device fp32, the amax of |dx|; pre_out: optional device
 * fp32 [R][D], dx before the rescale (validation). dy and x: any
 * scalify_dtype, R x D with the layout rules of scalify_layernorm_fwd; dx:
 * E4M3, E5M2 or F16, the same layout, may be the very same matrix as dy or x
 * but must not otherwise overlap them. workspace: at least
 * scalify_layernorm_bwd_workspace_size(R, D) bytes, 256-byte aligned, not
 * shared with a concurrent call. Deterministic (fixed-order sums). */
scalify_status scalify_layernorm_bwd(const scalify_scaled_array* dy, const scalify_scaled_array* x,
                                     const float* gamma, float eps, scalify_scaled_array* dx,
                                     float* dgamma, float* dbeta, int32_t rescale,
                                     int32_t target_log2, int32_t saturate, float* amax_out,
                                     float* pre_out, void* workspace, size_t workspace_bytes,
                                     void* stream);

/* Human-readable name of a status code (static string). */
const char* scalify_status_string(int32_t status);

#ifdef __cplusplus
}
#endif

#endif /* SCALIFY_H */
