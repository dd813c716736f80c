/*
 * CPU oracle for the Scalify scaled matmul path (arXiv 2407.17353).
 *
 * TEST INFRASTRUCTURE ONLY. Only tests/, __graft_entry__.smoke() and the
 * cpu_baseline leg of bench.py may load this library. The product path
 * (the HIP library) never calls it and shares no code with it.
 *
 * Plain, slow, obviously correct. Every number format is decoded by a table
 * built from its closed-form definition; every cast is an exact nearest
 * search over the sorted list of representable values; every matmul sums
 * products in fp64 in ascending k and rounds once to fp32.
 *
 * What each function follows in the paper:
 *   - ScaledArray X = X_d * X_s with a power-of-two scale simulated in fp32
 *     (Section 2, "Scaled array representation and quantization").
 *   - Two-stage quantization: unit-scale the data, round the scale to a power
 *     of two and correct q(X_d) (Section 2).
 *   - Matmul scale propagation under the independent-Gaussian assumption,
 *     with power-of-two rounding down of the scale (Section 3.2 and
 *     Algorithm 3).
 *   - Dynamic rescaling: statistic -> power of two -> rebalance_scale
 *     (Section 3.3, Algorithm 4), statistic = amax.
 *   - set_scaling / get_data_and_scale (Section 3.1).
 *   - FP8 E4M3 / E5M2 and FP16 formats (Section 1, Appendix A), OCP variants.
 *   - Scales broadcast beyond a scalar (Section 2): per-channel powers of two
 *     and E8M0 block scales of the MX formats.
 *
 * Readings of the paper where it is silent are listed in the design notes
 * of the repository; the ones used here are restated next to the code.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>

enum { OR_E4M3 = 0, OR_E5M2 = 1, OR_F16 = 2, OR_F32 = 3 };
enum { OR_RESCALE_NONE = 0, OR_RESCALE_AMAX = 1, OR_RESCALE_DELAYED = 2 };

/* ------------------------------------------------------------------------ */
/* Number formats: closed-form decode (OCP FP8 E4M3 / E5M2, IEEE binary16).  */
/* ------------------------------------------------------------------------ */

/* E4M3 (OCP "fn"): s|eeee|mmm, bias 7, no infinities, NaN = s.1111.111. */
double or_decode_e4m3(uint32_t c)
{
    int s = (c >> 7) & 1, e = (c >> 3) & 15, m = c & 7;
    double v;
    if (e == 15 && m == 7) return s ? -NAN : NAN;   /* the sign bit of a NaN is kept */
    if (e == 0) v = m * ldexp(1.0, -9);               /* subnormal: m/8 * 2^-6 */
    else v = (1.0 + m / 8.0) * ldexp(1.0, e - 7);
    return s ? -v : v;
}

/* E5M2: s|eeeee|mm, bias 15, IEEE-like: e=31 is Inf (m=0) or NaN. */
double or_decode_e5m2(uint32_t c)
{
    int s = (c >> 7) & 1, e = (c >> 2) & 31, m = c & 3;
    double v;
    if (e == 31) return m ? (s ? -NAN : NAN) : (s ? -INFINITY : INFINITY);
    if (e == 0) v = m * ldexp(1.0, -16);              /* subnormal: m/4 * 2^-14 */
    else v = (1.0 + m / 4.0) * ldexp(1.0, e - 15);
    return s ? -v : v;
}

/* IEEE binary16: s|eeeee|mmmmmmmmmm, bias 15. */
double or_decode_f16(uint32_t h)
{
    int s = (h >> 15) & 1, e = (h >> 10) & 31, m = h & 1023;
    double v;
    if (e == 31) return m ? (s ? -NAN : NAN) : (s ? -INFINITY : INFINITY);
    if (e == 0) v = m * ldexp(1.0, -24);
    else v = (1.0 + m / 1024.0) * ldexp(1.0, e - 15);
    return s ? -v : v;
}

double or_decode(int fmt, uint32_t code)
{
    switch (fmt) {
    case OR_E4M3: return or_decode_e4m3(code & 0xFF);
    case OR_E5M2: return or_decode_e5m2(code & 0xFF);
    case OR_F16:  return or_decode_f16(code & 0xFFFF);
    default: { float f; uint32_t u = code; memcpy(&f, &u, 4); return (double)f; }
    }
}

void or_decode_table8(int fmt, double* out256)
{
    for (uint32_t c = 0; c < 256; ++c) out256[c] = or_decode(fmt, c);
}

/* ------------------------------------------------------------------------ */
/* Cast: exact nearest search, ties to the even code.                        */
/* ------------------------------------------------------------------------ */

/* Sorted non-negative finite values of a format with their codes. The list is
 * extended by one "virtual" value: the next value above the largest finite
 * one, as if the exponent range were unbounded. Rounding to it means the
 * input overflowed. Its code is max_code + 1, so the even-code tie rule
 * applies to it like to any other candidate. */
typedef struct {
    int n;              /* number of entries incl. the virtual one */
    double* val;        /* ascending */
    uint32_t* code;
    uint32_t max_code;  /* largest finite positive code */
    uint32_t nan_code;  /* canonical positive NaN */
    uint32_t inf_code;  /* positive infinity, 0 if the format has none */
    int sign_shift;     /* 7 for FP8, 15 for FP16 */
} or_grid;

static or_grid g_grid[3];
static int g_grid_ready = 0;

static void grid_build(or_grid* g, int fmt)
{
    uint32_t ncodes = (fmt == OR_F16) ? 0x8000u : 0x80u;   /* positive half */
    g->val = (double*)malloc(sizeof(double) * (ncodes + 1));
    g->code = (uint32_t*)malloc(sizeof(uint32_t) * (ncodes + 1));
    g->n = 0;
    g->max_code = 0;
    /* Positive codes decode to non-decreasing values in code order for all
     * three formats; collect the finite ones. */
    for (uint32_t c = 0; c < ncodes; ++c) {
        double v = or_decode(fmt, c);
        if (!isfinite(v)) continue;
        g->val[g->n] = v;
        g->code[g->n] = c;
        g->n++;
        g->max_code = c;
    }
    /* Virtual overflow value: max + one unit in the last place at max. */
    {
        double vmax = g->val[g->n - 1];
        double prev = g->val[g->n - 2];
        /* ulp at max equals the spacing of the top binade; the value below
         * max is in the same binade for all three formats. */
        g->val[g->n] = vmax + (vmax - prev);
        g->code[g->n] = g->max_code + 1;
        g->n++;
    }
    if (fmt == OR_E4M3) { g->nan_code = 0x7F; g->inf_code = 0; g->sign_shift = 7; }
    else if (fmt == OR_E5M2) { g->nan_code = 0x7F; g->inf_code = 0x7C; g->sign_shift = 7; }
    else { g->nan_code = 0x7E00; g->inf_code = 0x7C00; g->sign_shift = 15; }
}

static void grids_init(void)
{
    if (g_grid_ready) return;
    /* Built once, before any parallel region uses it. */
    grid_build(&g_grid[OR_E4M3], OR_E4M3);
    grid_build(&g_grid[OR_E5M2], OR_E5M2);
    grid_build(&g_grid[OR_F16], OR_F16);
    g_grid_ready = 1;
}

void or_init(void) { grids_init(); }

/* Round the exact value of x (an fp32) to format fmt.
 * NaN -> canonical NaN with the sign of x. +-Inf and overflow: saturate to
 * +-max when sat != 0; otherwise E4M3 gives NaN, E5M2 and FP16 give +-Inf.
 * Subnormals of the target are kept; -0 stays -0. */
uint32_t or_cast(int fmt, int sat, float x)
{
    const or_grid* g;
    uint32_t sign;
    double a;
    int lo, hi;
    grids_init();
    g = &g_grid[fmt];
    sign = signbit(x) ? (1u << g->sign_shift) : 0u;
    if (isnan(x)) return g->nan_code | sign;
    if (isinf(x)) {
        if (sat) return g->max_code | sign;
        return (g->inf_code ? g->inf_code : g->nan_code) | sign;
    }
    a = fabs((double)x);
    /* Largest index lo with val[lo] <= a (val[0] = 0). */
    lo = 0; hi = g->n - 1;
    if (a >= g->val[hi]) {
        lo = hi;
    } else {
        while (hi - lo > 1) {
            int mid = (lo + hi) / 2;
            if (g->val[mid] <= a) lo = mid; else hi = mid;
        }
    }
    {
        int pick;
        if (g->val[lo] == a || lo == g->n - 1) {
            pick = lo;
        } else {
            /* Bracketed by val[lo] < a < val[lo+1]; the midpoint of two
             * grid values is exact in fp64, so this comparison is exact. */
            double mid = 0.5 * (g->val[lo] + g->val[lo + 1]);
            if (a < mid) pick = lo;
            else if (a > mid) pick = lo + 1;
            else pick = (g->code[lo] & 1u) ? lo + 1 : lo;   /* tie: even code */
        }
        if (pick == g->n - 1) {   /* rounded to the virtual value: overflow */
            if (sat) return g->max_code | sign;
            return (g->inf_code ? g->inf_code : g->nan_code) | sign;
        }
        return g->code[pick] | sign;
    }
}

void or_cast_array(int fmt, int sat, const float* x, int64_t n, void* out)
{
    int64_t i;
    grids_init();
    if (fmt == OR_F16) {
        uint16_t* o = (uint16_t*)out;
        #pragma omp parallel for schedule(static)
        for (i = 0; i < n; ++i) o[i] = (uint16_t)or_cast(fmt, sat, x[i]);
    } else {
        uint8_t* o = (uint8_t*)out;
        #pragma omp parallel for schedule(static)
        for (i = 0; i < n; ++i) o[i] = (uint8_t)or_cast(fmt, sat, x[i]);
    }
}

/* ------------------------------------------------------------------------ */
/* Power-of-two helpers (Section 2: the scale is always 2^k, E8M0).          */
/* ------------------------------------------------------------------------ */

/* floor(log2 |x|) for finite nonzero x, from frexp: x = f * 2^e, f in [0.5,1). */
int32_t or_floor_log2(double x)
{
    int e;
    frexp(fabs(x), &e);
    return e - 1;
}

/* Exponent of a power-of-two scale. Returns 0 and sets *ok = 0 if s is not a
 * finite positive power of two (a precondition violation). */
int32_t or_scale_exponent(float s, int* ok)
{
    int e;
    double f;
    if (!(s > 0.0f) || !isfinite(s)) { *ok = 0; return 0; }
    f = frexp((double)s, &e);
    *ok = (f == 0.5);
    return e - 1;
}

/* Matmul scale rule (Section 3.2, Algorithm 3): under the independent
 * unit-Gaussian assumption Var(sum_k a_k b_k) = K, so the output is divided
 * by sqrt(K); that constant is rounded DOWN to a power of two, as the paper
 * does for every scale. Result: the largest e with 2^e <= sqrt(K), i.e. with
 * 4^e <= K. Integer search, no floating-point sqrt. */
int32_t or_matmul_scale_log2(int64_t K)
{
    int32_t e = 0;
    if (K < 1) return 0;
    while (e < 31 && ((int64_t)1 << (2 * (e + 1))) <= K) e++;
    return e;
}

/* E8M0 range of a scale exponent (Section 2: 8-bit power-of-two scale). */
static int32_t clamp_e8m0(int32_t e)
{
    if (e < -127) return -127;
    if (e > 127) return 127;
    return e;
}

/* ------------------------------------------------------------------------ */
/* FP8 dot_general with fp64 accumulation.                                   */
/* ------------------------------------------------------------------------ */

/* Element (i,k) of A and (k,j) of B under the storage convention:
 * trans = 0: stored [rows][ld]; trans = 1: stored transposed [cols][ld]. */
#define A_AT(i, k) (ta ? A[(int64_t)(k) * lda + (i)] : A[(int64_t)(i) * lda + (k)])
#define B_AT(k, j) (tb ? B[(int64_t)(j) * ldb + (k)] : B[(int64_t)(k) * ldb + (j)])

/* acc[i*N+j] = fp32( sum_{k=0}^{K-1} dec(A[i,k]) * dec(B[k,j]) ), summed in
 * fp64 in ascending k. Rows are independent; OpenMP splits rows only. */
void or_matmul_acc(const uint8_t* A, int fa, int ta, int64_t lda,
                   const uint8_t* B, int fb, int tb, int64_t ldb,
                   int64_t M, int64_t N, int64_t K, float* acc)
{
    double da[256], db[256];
    int64_t i;
    or_decode_table8(fa, da);
    or_decode_table8(fb, db);
    #pragma omp parallel for schedule(dynamic, 1)
    for (i = 0; i < M; ++i) {
        int64_t j, k;
        for (j = 0; j < N; ++j) {
            double s = 0.0;
            for (k = 0; k < K; ++k) s += da[A_AT(i, k)] * db[B_AT(k, j)];
            acc[i * N + j] = (float)s;
        }
    }
}

/* The same sum for a list of (i, j) pairs, plus two norms of the product
 * terms that set the accumulator tolerance: l2 = sqrt(sum_k (a_ik b_kj)^2)
 * and l1 = sum_k |a_ik b_kj| (the magnitude a dot product's rounding error
 * is classically bounded against). Non-finite terms are left out of both. */
void or_matmul_acc_at(const uint8_t* A, int fa, int ta, int64_t lda,
                      const uint8_t* B, int fb, int tb, int64_t ldb,
                      int64_t K, const int64_t* ii, const int64_t* jj, int64_t n,
                      float* acc, double* term_l2, double* term_l1)
{
    double da[256], db[256];
    int64_t p;
    or_decode_table8(fa, da);
    or_decode_table8(fb, db);
    #pragma omp parallel for schedule(static)
    for (p = 0; p < n; ++p) {
        int64_t i = ii[p], j = jj[p], k;
        double s = 0.0, q = 0.0, a1 = 0.0;
        for (k = 0; k < K; ++k) {
            double t = da[A_AT(i, k)] * db[B_AT(k, j)];
            s += t;
            if (isfinite(t)) { q += t * t; a1 += fabs(t); }
        }
        acc[p] = (float)s;
        if (term_l2) term_l2[p] = sqrt(q);
        if (term_l1) term_l1[p] = a1;
    }
}

/* MX block scales (Section 2: a scale broadcastable to the data covers
 * block formats such as OCP MX, whose scales are E8M0). Row i of A and
 * column j of B carry one E8M0 byte per 32 consecutive k: the element
 * A[i,k] stands for dec(A[i,k]) * 2^(sa[i*ld + k/32] - 127), B[k,j] for
 * dec(B[k,j]) * 2^(sb[j*ld + k/32] - 127), on top of the scalar scales.
 * 0xFF (the NaN encoding of E8M0) is not a scale: returns 1 if any byte
 * that a product uses holds it, else 0. Entries k/32 >= ceil(K/32) of a row
 * are never read. The sum is that of or_matmul_acc with each exact product
 * multiplied by its two block factors (exact in fp64: both are powers of
 * two and the product of two FP8 values has at most 8 significant bits). */
static int mx_block_ok(const uint8_t* s, int64_t rows, int64_t ld, int64_t nb)
{
    int64_t r, b;
    for (r = 0; r < rows; ++r)
        for (b = 0; b < nb; ++b)
            if (s[r * ld + b] == 0xFF) return 0;
    return 1;
}

int or_matmul_acc_mx(const uint8_t* A, int fa, int ta, int64_t lda,
                     const uint8_t* B, int fb, int tb, int64_t ldb,
                     int64_t M, int64_t N, int64_t K,
                     const uint8_t* sa, const uint8_t* sb, int64_t lds, float* acc)
{
    double da[256], db[256];
    int64_t i, nb = (K + 31) / 32;
    if (!mx_block_ok(sa, M, lds, nb) || !mx_block_ok(sb, N, lds, nb)) return 1;
    or_decode_table8(fa, da);
    or_decode_table8(fb, db);
    #pragma omp parallel for schedule(dynamic, 1)
    for (i = 0; i < M; ++i) {
        int64_t j, k;
        for (j = 0; j < N; ++j) {
            double s = 0.0;
            for (k = 0; k < K; ++k) {
                const int e = (int)sa[i * lds + k / 32] - 127 + (int)sb[j * lds + k / 32] - 127;
                s += ldexp(da[A_AT(i, k)] * db[B_AT(k, j)], e);
            }
            acc[i * N + j] = (float)s;
        }
    }
    return 0;
}

/* The same at listed positions (i, j), with the l1 norm of the scaled
 * product terms (non-finite terms left out), as or_matmul_acc_at. */
int or_matmul_acc_mx_at(const uint8_t* A, int fa, int ta, int64_t lda,
                        const uint8_t* B, int fb, int tb, int64_t ldb, int64_t K,
                        const uint8_t* sa, const uint8_t* sb, int64_t lds,
                        const int64_t* ii, const int64_t* jj, int64_t n,
                        float* acc, double* term_l1)
{
    double da[256], db[256];
    int64_t p, nb = (K + 31) / 32, bad = 0;
    or_decode_table8(fa, da);
    or_decode_table8(fb, db);
    for (p = 0; p < n; ++p) {
        int64_t b;
        for (b = 0; b < nb; ++b)
            if (sa[ii[p] * lds + b] == 0xFF || sb[jj[p] * lds + b] == 0xFF) bad = 1;
    }
    if (bad) return 1;
    #pragma omp parallel for schedule(static)
    for (p = 0; p < n; ++p) {
        int64_t i = ii[p], j = jj[p], k;
        double s = 0.0, a1 = 0.0;
        for (k = 0; k < K; ++k) {
            const int e = (int)sa[i * lds + k / 32] - 127 + (int)sb[j * lds + k / 32] - 127;
            const double t = ldexp(da[A_AT(i, k)] * db[B_AT(k, j)], e);
            s += t;
            if (isfinite(t)) a1 += fabs(t);
        }
        acc[p] = (float)s;
        term_l1[p] = a1;
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Dynamic rescale (Section 3.3) and the matmul epilogue.                    */
/* ------------------------------------------------------------------------ */

/* amax = max |x| over non-NaN elements; *any = 0 if every element is NaN. */
float or_amax(const float* x, int64_t n, int* any)
{
    float m = 0.0f;
    int64_t i;
    *any = 0;
    for (i = 0; i < n; ++i) {
        float a = fabsf(x[i]);
        if (isnan(a)) continue;
        *any = 1;
        if (a > m) m = a;
    }
    return m;
}

/* Rescale exponent e_r from the statistic: the power of two is rounded down
 * (floor(log2 amax)), then shifted by the target t, so that the rescaled
 * amax lies in [2^t, 2^(t+1)). No rescale (0) when there is nothing to
 * measure: amax 0, +Inf, or no non-NaN element. */
int32_t or_rescale_exponent(float amax, int any, int32_t t)
{
    if (!any || amax == 0.0f || isinf(amax)) return 0;
    return or_floor_log2((double)amax) - t;
}

/* Shared tail of the matmul epilogue and of rescale: given fp32 values v
 * whose true value is v * 2^e_in, choose the output scale exponent and cast.
 *   mode NONE: e_want = e_in;  mode AMAX: e_want = e_in + e_r(amax of v);
 *   mode DELAYED: e_want = e_in + e_r(stat_in), stat_in from an earlier call.
 *   e_out = clamp(e_want) to the E8M0 range;  data' = ldexp(v, e_in - e_out).
 * One power-of-two shift of the exact fp32 value, then one rounding. */
static int32_t finish(const float* v, int64_t n, int32_t e_in, int mode, int32_t t,
                      int sat, int out_fmt, void* out, float* amax_out, float stat_in)
{
    int any;
    float amax = or_amax(v, n, &any);
    int32_t e_r = 0;
    if (mode == OR_RESCALE_AMAX) e_r = or_rescale_exponent(amax, any, t);
    /* DELAYED: the statistic recorded by an earlier call; a NaN one counts
     * as "nothing measured", like an all-NaN tensor in AMAX mode. */
    if (mode == OR_RESCALE_DELAYED) e_r = or_rescale_exponent(stat_in, !isnan(stat_in), t);
    int32_t e_out = clamp_e8m0(e_in + e_r);
    int32_t shift = e_in - e_out;
    int64_t i;
    grids_init();
    if (amax_out) *amax_out = amax;
    #pragma omp parallel for schedule(static)
    for (i = 0; i < n; ++i) {
        float d = ldexpf(v[i], shift);
        uint32_t c = or_cast(out_fmt, sat, d);
        if (out_fmt == OR_F16) ((uint16_t*)out)[i] = (uint16_t)c;
        else ((uint8_t*)out)[i] = (uint8_t)c;
    }
    return e_out;
}

int32_t or_finish_pre(const float* w, int64_t n, int32_t e_w, int32_t e_cc, int mode, int32_t t,
                      float stat_in, int sat, int out_fmt, void* out, float* amax_out);

/* Epilogue of the scaled matmul (Section 3.2 propagation + Section 3.3
 * dynamic rescale + stage-2 cast of Section 2), applied to an fp32
 * accumulator acc[n] (n = M*N).
 *   e_c  = matmul scale rule for K; the propagated data is acc * 2^-e_c, a
 *   power-of-two division of the accumulator, with value
 *   data * 2^(e_a + e_b + e_c).
 * That data is never rounded to fp32 on its own: where acc * 2^-e_c would
 * be an fp32 subnormal, rounding it first and then shifting it again by the
 * rescale would round twice. The statistic is therefore taken on acc, with
 * e_c subtracted from its exponent (floor(log2(amax * 2^-e_c)) =
 * floor(log2 amax) - e_c exactly), and each code is the cast of acc after
 * one power-of-two shift to the output scale: or_finish_pre with the
 * pre-cast value w = acc, e_w = e_a + e_b and the statistic offset e_c.
 * Returns 0 on success, -1 on a non-power-of-two input scale.
 * Outputs: codes, *e_out (output scale = 2^e_out), *amax (of acc*2^-e_c,
 * rounded once to fp32). */
static int matmul_epilogue_impl(const float* acc, int64_t n, float s_a, float s_b, int64_t K,
                                int mode, int32_t t, int sat, int out_fmt,
                                void* out, int32_t* e_out, float* amax, float stat_in)
{
    int ok_a = 1, ok_b = 1;
    int32_t e_a = or_scale_exponent(s_a, &ok_a);
    int32_t e_b = or_scale_exponent(s_b, &ok_b);
    int32_t e_c = or_matmul_scale_log2(K);
    if (!ok_a || !ok_b) return -1;
    *e_out = or_finish_pre(acc, n, e_a + e_b, e_c, mode, t, stat_in, sat, out_fmt, out, amax);
    return 0;
}

int or_matmul_epilogue(const float* acc, int64_t n, float s_a, float s_b, int64_t K,
                       int mode, int32_t t, int sat, int out_fmt,
                       void* out, int32_t* e_out, float* amax)
{
    if (mode != OR_RESCALE_NONE && mode != OR_RESCALE_AMAX) return -2;
    return matmul_epilogue_impl(acc, n, s_a, s_b, K, mode, t, sat, out_fmt, out, e_out, amax, 0.0f);
}

/* Delayed rescaling (Section 3.3): as the epilogue above, with the rescale
 * exponent taken from amax_in, the statistic an earlier call recorded
 * (e_r = floor(log2 amax_in) - t; 0 when amax_in is 0, +Inf or NaN). The
 * amax this call measures is returned in *amax for the next call. */
int or_matmul_epilogue_delayed(const float* acc, int64_t n, float s_a, float s_b, int64_t K,
                               float amax_in, int32_t t, int sat, int out_fmt,
                               void* out, int32_t* e_out, float* amax)
{
    return matmul_epilogue_impl(acc, n, s_a, s_b, K, OR_RESCALE_DELAYED, t, sat, out_fmt,
                                out, e_out, amax, amax_in);
}

/* Full scaled matmul: accumulate then epilogue. acc_out may be NULL. */
int or_matmul(const uint8_t* A, int fa, int ta, int64_t lda, float s_a,
              const uint8_t* B, int fb, int tb, int64_t ldb, float s_b,
              int64_t M, int64_t N, int64_t K,
              int mode, int32_t t, int sat, int out_fmt,
              void* out, int32_t* e_out, float* amax, float* acc_out)
{
    float* acc = acc_out ? acc_out : (float*)malloc(sizeof(float) * (size_t)(M * N > 0 ? M * N : 1));
    int rc;
    or_matmul_acc(A, fa, ta, lda, B, fb, tb, ldb, M, N, K, acc);
    rc = or_matmul_epilogue(acc, M * N, s_a, s_b, K, mode, t, sat, out_fmt, out, e_out, amax);
    if (!acc_out) free(acc);
    return rc;
}

/* Decode an array of codes (or fp32 bits) of format fmt to fp32. FP8 and
 * FP16 values are exact in fp32. */
static void decode_to_f32(int fmt, const void* in, int64_t n, float* out)
{
    int64_t i;
    for (i = 0; i < n; ++i) {
        uint32_t c;
        if (fmt == OR_F32) { memcpy(&out[i], (const float*)in + i, 4); continue; }
        c = (fmt == OR_F16) ? ((const uint16_t*)in)[i] : ((const uint8_t*)in)[i];
        out[i] = (float)or_decode(fmt, c);
    }
}

/* Dynamic rescale of a ScaledArray (Section 3.3 with rebalance_scale, plus
 * the cast when the output format differs): value = dec(in) * s_in.
 * AMAX: e_r from the amax of dec(in); s_out = s_in * 2^e_r (clamped);
 * data' = dec(in) * 2^-(e_out - e_in). NONE: scale kept, data cast. */
int or_rescale(int in_fmt, const void* in, int64_t n, float s_in,
               int mode, int32_t t, int sat, int out_fmt,
               void* out, int32_t* e_out, float* amax)
{
    int ok = 1;
    int32_t e_in = or_scale_exponent(s_in, &ok);
    float* v;
    if (!ok) return -1;
    v = (float*)malloc(sizeof(float) * (size_t)(n > 0 ? n : 1));
    decode_to_f32(in_fmt, in, n, v);
    *e_out = finish(v, n, e_in, mode, t, sat, out_fmt, out, amax, 0.0f);
    free(v);
    return 0;
}

/* set_scaling (Section 3.1): the output gets scale 2^e_new; the data is
 * rescaled by the ratio of the old and new scales, then cast. */
int or_set_scaling(int in_fmt, const void* in, int64_t n, float s_in,
                   int32_t e_new, int sat, int out_fmt, void* out)
{
    int ok = 1;
    int32_t e_in = or_scale_exponent(s_in, &ok);
    float* v;
    int64_t i;
    if (!ok || e_new < -127 || e_new > 127) return -1;
    v = (float*)malloc(sizeof(float) * (size_t)(n > 0 ? n : 1));
    decode_to_f32(in_fmt, in, n, v);
    for (i = 0; i < n; ++i) {
        uint32_t c = or_cast(out_fmt, sat, ldexpf(v[i], e_in - e_new));
        if (out_fmt == OR_F16) ((uint16_t*)out)[i] = (uint16_t)c;
        else ((uint8_t*)out)[i] = (uint8_t)c;
    }
    free(v);
    return 0;
}

/* Cast operator on the data only (Appendix A: casts act on data, the scale
 * is unchanged). */
void or_cast_data(int in_fmt, const void* in, int64_t n, int sat, int out_fmt, void* out)
{
    float* v = (float*)malloc(sizeof(float) * (size_t)(n > 0 ? n : 1));
    int64_t i;
    decode_to_f32(in_fmt, in, n, v);
    for (i = 0; i < n; ++i) {
        uint32_t c = or_cast(out_fmt, sat, v[i]);
        if (out_fmt == OR_F16) ((uint16_t*)out)[i] = (uint16_t)c;
        else ((uint8_t*)out)[i] = (uint8_t)c;
    }
    free(v);
}

/* ------------------------------------------------------------------------ */
/* Scaled add and activation applied to the matmul output, before the        */
/* rescale and cast (add rule: Section 3.2 / Algorithm 3; activation rule:  */
/* Appendix C.1).                                                            */
/* ------------------------------------------------------------------------ */

enum { OR_ACT_NONE = 0, OR_ACT_RELU = 1, OR_ACT_GELU_TANH = 2, OR_ACT_SILU = 3 };

/* Gating function g of an activation written f(x) = x * g(x), with g -> 0 at
 * -inf and g -> 1 at +inf (Appendix C.1), evaluated in fp64:
 *   relu: g = 1 for x > 0, else 0;
 *   gelu, tanh form: g = (1 + tanh(u)) / 2 with u = sqrt(2/pi) (x + 0.044715 x^3),
 *     evaluated as the equal 1 / (1 + exp(-2u)): 1 + tanh(u) cancels for
 *     u << 0, where the gate would lose all its digits;
 *   silu (swish): g = 1 / (1 + exp(-x)).
 * Any other act: g = 1 (identity). */
double or_gate(int act, double x)
{
    switch (act) {
    case OR_ACT_RELU:
        return x > 0.0 ? 1.0 : 0.0;
    case OR_ACT_GELU_TANH: {
        double u = sqrt(2.0 / M_PI) * (x + 0.044715 * x * x * x);
        return 1.0 / (1.0 + exp(-2.0 * u));
    }
    case OR_ACT_SILU:
        return 1.0 / (1.0 + exp(-x));
    default:
        return 1.0;
    }
}

/* Output scale exponent of the scaled add (Algorithm 3): for independent
 * unit-scaled operands the sum's standard deviation is sqrt(s_1^2 + s_2^2);
 * like every scale it is rounded down to a power of two. */
int32_t or_add_scale_log2(int32_t e1, int32_t e2)
{
    return or_floor_log2(sqrt(ldexp(1.0, 2 * e1) + ldexp(1.0, 2 * e2)));
}

/* Pre-cast value w[i] of the fused matmul epilogue, whose true value is
 * w * 2^(*e_w); the data whose statistic the rescale gathers is
 * w * 2^-(*e_cc).
 *   - no residual: w = acc (true value acc * 2^(e_a+e_b)), e_cc = e_c: the
 *     matmul's propagated data is acc * 2^-e_c (Section 3.2);
 *   - residual R (codes res[i*res_ld + j], format res_fmt, scale s_res = 2^q;
 *     res_ld = 0 repeats one row): scaled add of the matmul output
 *     (scale 2^(e_a+e_b+e_c)) and R, e_w = add-rule exponent, e_cc = 0,
 *     w = fl32(fl32(acc * 2^(e_a+e_b-e_w)) + fl32(r * 2^(q-e_w))): each
 *     power-of-two product exact unless it underflows, one rounding of the sum;
 *   - activation act (after the add, scale unchanged, Appendix C.1):
 *     w = fl32(w * g(w * 2^e_w)).
 * y64[i] (optional) receives the unrounded fp64 value before that last
 * rounding (w itself without an activation).
 * Returns 0, or -1 on a scale that is not a finite power of two. */
int or_fused_pre_ch(const float* acc, int64_t M, int64_t N, float s_a, float s_b,
                    const float* ch_a, const float* ch_b, int64_t K,
                    const void* res, int res_fmt, int64_t res_ld, float s_res, int act,
                    float* w, double* y64, int32_t* e_w_out, int32_t* e_cc_out);

int or_fused_pre(const float* acc, int64_t M, int64_t N, float s_a, float s_b, int64_t K,
                 const void* res, int res_fmt, int64_t res_ld, float s_res, int act,
                 float* w, double* y64, int32_t* e_w_out, int32_t* e_cc_out)
{
    return or_fused_pre_ch(acc, M, N, s_a, s_b, NULL, NULL, K, res, res_fmt, res_ld, s_res, act,
                           w, y64, e_w_out, e_cc_out);
}

/* or_fused_pre with channel scales (Section 2: a scale broadcastable to the
 * data; channel scaling): A = A_d * s_a * ch_a[i] (ch_a: one power of two per
 * row of A, i.e. per output row; NULL = all 1), B = B_d * s_b * ch_b[j] (one
 * per column of B, i.e. per output column). The output keeps one scalar
 * scale: the channel factors go into the data, as one power-of-two product
 * of acc (exact unless it leaves the fp32 range):
 *   no residual: w = fl32(acc * ch_a[i] * ch_b[j]);
 *   residual: the product term is fl32(acc * 2^(e_a+e_b-e_w) * ch_a[i] * ch_b[j])
 *     (one power-of-two product) before the scaled add. */
int or_fused_pre_ch(const float* acc, int64_t M, int64_t N, float s_a, float s_b,
                    const float* ch_a, const float* ch_b, int64_t K,
                    const void* res, int res_fmt, int64_t res_ld, float s_res, int act,
                    float* w, double* y64, int32_t* e_w_out, int32_t* e_cc_out)
{
    int ok_a = 1, ok_b = 1, ok_r = 1, ok_ch = 1;
    int32_t e_a = or_scale_exponent(s_a, &ok_a);
    int32_t e_b = or_scale_exponent(s_b, &ok_b);
    int32_t e_c = or_matmul_scale_log2(K);
    int32_t q = res ? or_scale_exponent(s_res, &ok_r) : 0;
    int32_t e_w, e_cc;
    int64_t i, j;
    if (!ok_a || !ok_b || !ok_r) return -1;
    for (i = 0; ch_a && i < M; ++i) {
        int ok = 1;
        (void)or_scale_exponent(ch_a[i], &ok);
        ok_ch &= ok;
    }
    for (j = 0; ch_b && j < N; ++j) {
        int ok = 1;
        (void)or_scale_exponent(ch_b[j], &ok);
        ok_ch &= ok;
    }
    if (!ok_ch) return -1;
    if (res) {
        e_w = or_add_scale_log2(e_a + e_b + e_c, q);
        e_cc = 0;
    } else {
        e_w = e_a + e_b;
        e_cc = e_c;
    }
    for (i = 0; i < M; ++i) {
        for (j = 0; j < N; ++j) {
            int64_t k = i * N + j;
            double y;
            float v = acc[k];
            int32_t e_ch = (ch_a ? or_scale_exponent(ch_a[i], &ok_ch) : 0) +
                           (ch_b ? or_scale_exponent(ch_b[j], &ok_ch) : 0);
            if (res) {
                int64_t rk = i * res_ld + j;
                uint32_t c = res_fmt == OR_F16 ? ((const uint16_t*)res)[rk]
                                               : ((const uint8_t*)res)[rk];
                float r = (float)or_decode(res_fmt, c);
                v = (float)((double)ldexpf(v, e_a + e_b - e_w + e_ch) + (double)ldexpf(r, q - e_w));
            } else if (e_ch != 0) {
                v = ldexpf(v, e_ch);
            }
            y = (double)v;
            if (act != OR_ACT_NONE) y = (double)v * or_gate(act, ldexp((double)v, e_w));
            if (y64) y64[k] = y;
            w[k] = (float)y;
        }
    }
    *e_w_out = e_w;
    *e_cc_out = e_cc;
    return 0;
}

/* Rescale and cast of pre-cast values w (true value w * 2^e_w; statistic
 * over the data w * 2^-e_cc), Section 3.3 and stage 2 of Section 2:
 *   amax = max |w| over non-NaN elements (reported as amax * 2^-e_cc);
 *   AMAX: e_r = floor(log2 amax) - e_cc - t (0 for 0, +Inf, all NaN);
 *   DELAYED: e_r from stat_in as in finish(); NONE: e_r = 0;
 *   e_out = clamp(e_w + e_cc + e_r); codes = cast(w * 2^(e_w - e_out)),
 * one power-of-two shift of w, then one rounding. Returns e_out. */
int32_t or_finish_pre(const float* w, int64_t n, int32_t e_w, int32_t e_cc, int mode, int32_t t,
                      float stat_in, int sat, int out_fmt, void* out, float* amax_out)
{
    int any;
    float amax = or_amax(w, n, &any);
    int32_t e_r = 0, e_out, shift;
    int64_t i;
    if (mode == OR_RESCALE_AMAX && any && amax != 0.0f && !isinf(amax))
        e_r = or_floor_log2((double)amax) - e_cc - t;
    if (mode == OR_RESCALE_DELAYED) e_r = or_rescale_exponent(stat_in, !isnan(stat_in), t);
    e_out = clamp_e8m0(e_w + e_cc + e_r);
    shift = e_w - e_out;
    grids_init();
    if (amax_out) *amax_out = ldexpf(amax, -e_cc);
    #pragma omp parallel for schedule(static)
    for (i = 0; i < n; ++i) {
        uint32_t c = or_cast(out_fmt, sat, ldexpf(w[i], shift));
        if (out_fmt == OR_F16) ((uint16_t*)out)[i] = (uint16_t)c;
        else ((uint8_t*)out)[i] = (uint8_t)c;
    }
    return e_out;
}

/* ------------------------------------------------------------------------ */
/* Scaled LayerNorm (Appendix C.2; the custom LayerNorm of the experiments,  */
/* with the dynamic rescale of its input gradient, Section 4).               */
/* ------------------------------------------------------------------------ */

/* Forward on the data component, one row of D values x (true value x * X_s):
 * the normalization is scale invariant up to eps, so it normalizes X_d and
 * gives the output scale 1:
 *   mu = mean(x), sigma = sqrt(mean((x - mu)^2)), xhat = (x - mu) / (sigma + eps),
 *   y = xhat * gamma + beta   (gamma NULL = 1, beta NULL = 0).
 * fp64 throughout; y64 (optional) gets y, mu_out / sigma_out (optional) the
 * row statistics. Rows are independent. */
void or_layernorm_fwd_pre(int in_fmt, const void* x, int64_t R, int64_t D, const float* gamma,
                          const float* beta, double eps, double* y64, double* mu_out,
                          double* sigma_out)
{
    int64_t r;
    double* v = (double*)malloc(sizeof(double) * (size_t)(D > 0 ? D : 1));
    for (r = 0; r < R; ++r) {
        double mu = 0.0, var = 0.0, sigma, den;
        int64_t j;
        for (j = 0; j < D; ++j) {
            int64_t k = r * D + j;
            if (in_fmt == OR_F32) v[j] = (double)((const float*)x)[k];
            else if (in_fmt == OR_F16) v[j] = or_decode(OR_F16, ((const uint16_t*)x)[k]);
            else v[j] = or_decode(in_fmt, ((const uint8_t*)x)[k]);
            mu += v[j];
        }
        mu /= (double)D;
        for (j = 0; j < D; ++j) var += (v[j] - mu) * (v[j] - mu);
        var /= (double)D;
        sigma = sqrt(var);
        den = sigma + eps;
        for (j = 0; j < D; ++j) {
            double xh = (v[j] - mu) / den;
            double y = xh * (gamma ? (double)gamma[j] : 1.0) + (beta ? (double)beta[j] : 0.0);
            if (y64) y64[r * D + j] = y;
        }
        if (mu_out) mu_out[r] = mu;
        if (sigma_out) sigma_out[r] = sigma;
    }
    free(v);
}

/* Backward of the forward above with respect to the data component, for an
 * upstream gradient whose true value is dy * s_dy. With c = x - mu,
 * s = sigma + eps, xhat = c / s and g = dy * gamma:
 *   dL/dx_d = (1/s) (g - mean(g) - (c / sigma) mean(g * xhat)) * s_dy
 * (the last term is 0 for a constant row, sigma = 0, where its limit is 0
 * for eps > 0). As x = X_d * X_s, dL/dX = dL/dx_d / X_s: the gradient is the
 * ScaledArray (dx, s_dy / X_s) with
 *   dx = (1/s) (g - mean(g) - (c / sigma) mean(g * xhat)),
 * which the dynamic rescale then rebalances (Section 4: the rescale of the
 * LayerNorm input gradient). Also the parameter gradients, in units of s_dy:
 *   dgamma_j = sum_r dy[r,j] * xhat[r,j],   dbeta_j = sum_r dy[r,j].
 * fp64 throughout; every output is optional. */
void or_layernorm_bwd_pre(int dy_fmt, const void* dy, int x_fmt, const void* x, int64_t R,
                          int64_t D, const float* gamma, double eps, double* dx64,
                          double* dgamma, double* dbeta)
{
    int64_t r, j;
    double* v = (double*)malloc(sizeof(double) * (size_t)(D > 0 ? D : 1));
    double* g = (double*)malloc(sizeof(double) * (size_t)(D > 0 ? D : 1));
    double* d = (double*)malloc(sizeof(double) * (size_t)(D > 0 ? D : 1));
    if (dgamma) for (j = 0; j < D; ++j) dgamma[j] = 0.0;
    if (dbeta) for (j = 0; j < D; ++j) dbeta[j] = 0.0;
    for (r = 0; r < R; ++r) {
        double mu = 0.0, var = 0.0, sigma, s, mg = 0.0, mgx = 0.0;
        for (j = 0; j < D; ++j) {
            int64_t k = r * D + j;
            if (x_fmt == OR_F32) v[j] = (double)((const float*)x)[k];
            else if (x_fmt == OR_F16) v[j] = or_decode(OR_F16, ((const uint16_t*)x)[k]);
            else v[j] = or_decode(x_fmt, ((const uint8_t*)x)[k]);
            if (dy_fmt == OR_F32) d[j] = (double)((const float*)dy)[k];
            else if (dy_fmt == OR_F16) d[j] = or_decode(OR_F16, ((const uint16_t*)dy)[k]);
            else d[j] = or_decode(dy_fmt, ((const uint8_t*)dy)[k]);
            mu += v[j];
        }
        mu /= (double)D;
        for (j = 0; j < D; ++j) var += (v[j] - mu) * (v[j] - mu);
        var /= (double)D;
        sigma = sqrt(var);
        s = sigma + eps;
        for (j = 0; j < D; ++j) {
            double xh = (v[j] - mu) / s;
            g[j] = d[j] * (gamma ? (double)gamma[j] : 1.0);
            mg += g[j];
            mgx += g[j] * xh;
            if (dgamma) dgamma[j] += d[j] * xh;
            if (dbeta) dbeta[j] += d[j];
        }
        mg /= (double)D;
        mgx /= (double)D;
        for (j = 0; j < D; ++j) {
            double t = sigma > 0.0 ? ((v[j] - mu) / sigma) * mgx : 0.0;
            if (dx64) dx64[r * D + j] = (g[j] - mg - t) / s;
        }
    }
    free(v);
    free(g);
    free(d);
}
