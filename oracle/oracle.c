/*
 * CPU oracle for the fused W8A8 quantized linear.
 *
 * TEST INFRASTRUCTURE ONLY. Only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg load this library. The HIP library never links, loads or calls it,
 * and the two share no source, header, table or helper.
 *
 * What it computes, as plain loops in the order the definitions give:
 *   - orc_quantize_rows: symmetric absmax int8 quantization of every row of a
 *     K-contiguous bf16 matrix. Applied per output channel to W [N,K] and per token to
 *     X [M,K] (Section 3, "The quantization recipe (reused)": per-channel int8 weights,
 *     per-token dynamic int8 activations; "The fused kernel": the per-token scales are
 *     computed online).
 *   - orc_gemm_acc: the exact integer product acc[m][n] = sum_k Xq[m][k] * Wq[n][k]
 *     (Section 3, "The fused kernel": int8 x int8 -> int32 accumulation).
 *   - orc_epilogue: per-token scale times per-channel scale applied to the int32
 *     accumulator, plus the bias, written as bf16 (Section 3, "The fused kernel": the
 *     epilogue works directly on the accumulator and emits the dequantized result).
 *   - orc_epilogue_f64: diagnostic only; the same dequantization in double, rounded
 *     once to bf16, to show how far the float32 epilogue is from the exact value.
 *   - orc_quantize_rows_ex: the same row rule applied to transformed values
 *     v[k] = T(x[k]) * c[k]: T the identity or the exact (erf) GELU, c an optional
 *     per-K-channel multiplier. The multiplier is the runtime half of SmoothQuant
 *     (Section 3, "The quantization recipe (reused)": SmoothQuant with alpha = 0.5):
 *     X is divided per input channel by the smoothing factor, W multiplied by it, so
 *     the product is unchanged. GELU in front of the quantizer is the activation that
 *     feeds the MLP down-projection of the DiT (Section 3, "Target architecture").
 *   - orc_col_absmax, orc_smooth_factors: offline calibration of the smoothing
 *     factors, s[k] = max|X[:,k]|^alpha / max|W[:,k]|^(1 - alpha), the published
 *     SmoothQuant rule the recipe names.
 *
 * The paper leaves the following open; these readings are fixed here and bind the GPU
 * path too:
 *   - scale s = a / 127 with a = max_k |v[k]|; the codes are
 *     q = clamp(rne(v * (127 / a)), -127, 127): one correctly rounded division per row
 *     for 127/a, one float32 multiply per element, round half to even, symmetric clamp
 *     (-128 is never produced);
 *   - a row with a == 0, or whose 127/a overflows float32, is a zero row: s = 0, q = 0;
 *   - scales are float32 arrays;
 *   - epilogue: y = bf16_rne(fmaf((float)acc, sx[m] * sw[n], b[n])), b = +0 when there
 *     is no bias, (float)acc rounded to nearest even;
 *   - inputs must be finite (the paper's gate is "no NaNs"); a non-finite input is
 *     rejected with an error code;
 *   - transformed rows: t = GELU(x) is the double-precision value
 *     0.5 * x * erfc(-x / sqrt(2)) rounded once to float32 (the GPU computes its own
 *     float32 GELU, equal to this within a few units in the last place); v = t * c[k]
 *     is one float32 multiply; a = max |v|, and the row rule above applies to v;
 *   - smoothing factors: alpha = 0.5 gives s = sqrtf(ax) / sqrtf(aw) (each operation
 *     correctly rounded float32, so both sides agree bit for bit); any other alpha
 *     gives the double-precision value ax^alpha / aw^(1 - alpha) rounded to float32;
 *     a channel with ax or aw zero, or a factor that is zero or not finite, gets
 *     s = 1 (left unsmoothed); the runtime multiplier is s_inv = 1.0f / s.
 *
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fopenmp (no implicit FMA contraction, so
 * every float operation is exactly the one written).
 */
#include <fenv.h>
#include <math.h>
#include <stdint.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

#define ORC_OK 0
#define ORC_ERR_NONFINITE 1
#define ORC_ERR_ROUNDING_MODE 2
#define ORC_ERR_INT32_OVERFLOW 3
#define ORC_ERR_ARG 4

/* bf16 is the upper half of an IEEE binary32: widening is a 16-bit shift, exact. */
static float bf16_bits_to_f32(uint16_t h)
{
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

/* Round a binary32 to bf16, round-to-nearest, ties to even, from the definition: keep
 * the upper 16 bits and add one unit in their last place when the discarded lower 16
 * bits are more than half a unit, or exactly half and the kept part is odd. A carry out
 * of the mantissa moves to the next binade (and from the largest finite value to
 * infinity), as rounding requires. NaN stays NaN (quiet bit set). */
static uint16_t f32_to_bf16_rne(float f)
{
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu) != 0u)
        return (uint16_t)((u >> 16) | 0x0040u);
    uint32_t kept = u >> 16;
    uint32_t dropped = u & 0xFFFFu;
    if (dropped > 0x8000u || (dropped == 0x8000u && (kept & 1u)))
        kept += 1u;
    return (uint16_t)kept;
}

uint16_t orc_f32_to_bf16(float f) { return f32_to_bf16_rne(f); }

void orc_f32_to_bf16_array(const float *f, int64_t n, uint16_t *out)
{
    for (int64_t i = 0; i < n; ++i)
        out[i] = f32_to_bf16_rne(f[i]);
}

float orc_bf16_to_f32(uint16_t h) { return bf16_bits_to_f32(h); }

static void set_threads(int nthreads)
{
#ifdef _OPENMP
    if (nthreads > 0)
        omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
}

int orc_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Exact (to double precision) GELU: x * Phi(x), written with erfc so that the left
 * tail keeps its relative accuracy (1 + erf(z) would cancel for z << 0). */
static double gelu_f64(double x)
{
    return 0.5 * x * erfc(-x / sqrt(2.0));
}

void orc_gelu_f64_array(const double *x, int64_t n, double *out)
{
    for (int64_t i = 0; i < n; ++i)
        out[i] = gelu_f64(x[i]);
}

#define ORC_ACT_NONE 0
#define ORC_ACT_GELU 1

/* The value the row rule sees for element k: T(x) as float32, times c[k] if given. */
static float transformed(uint16_t h, int act, const float *colmul, int64_t k)
{
    float t = bf16_bits_to_f32(h);
    if (act == ORC_ACT_GELU)
        t = (float)gelu_f64((double)t);
    if (colmul)
        t = t * colmul[k];          /* one float32 multiply */
    return t;
}

/* Per-row symmetric absmax quantization (Section 3, "The quantization recipe
 * (reused)") of the transformed values v[k] = T(x[k]) * c[k]. x: [rows, K] bf16 bits,
 * row-major. act: 0 identity, 1 GELU. colmul: [K] or NULL. q: [rows, K] int8.
 * scale: [rows]. */
int orc_quantize_rows_ex(const uint16_t *x, int64_t rows, int64_t K, int act,
                         const float *colmul, int8_t *q, float *scale, int nthreads)
{
    if (rows < 0 || K < 0 || (act != ORC_ACT_NONE && act != ORC_ACT_GELU))
        return ORC_ERR_ARG;
    if (fegetround() != FE_TONEAREST)
        return ORC_ERR_ROUNDING_MODE;
    int err = ORC_OK;
    set_threads(nthreads);
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < rows; ++r) {
        const uint16_t *row = x + r * K;
        int8_t *qrow = q + r * K;
        /* a = max_k |v[k]|; for the identity transform v is the bf16 value, exact. */
        float a = 0.0f;
        int finite = 1;
        for (int64_t k = 0; k < K; ++k) {
            if (!isfinite(bf16_bits_to_f32(row[k])))
                finite = 0;
            float v = transformed(row[k], act, colmul, k);
            if (!isfinite(v))
                finite = 0;
            float av = fabsf(v);
            if (av > a)
                a = av;
        }
        if (!finite) {
#pragma omp atomic write
            err = ORC_ERR_NONFINITE;
            continue;
        }
        float inv = 127.0f / a;     /* reciprocal step, correctly rounded */
        float s = a / 127.0f;       /* dequantization scale, correctly rounded */
        if (!(a > 0.0f) || !isfinite(inv)) {
            scale[r] = 0.0f;
            for (int64_t k = 0; k < K; ++k)
                qrow[k] = 0;
            continue;
        }
        scale[r] = s;
        for (int64_t k = 0; k < K; ++k) {
            float p = transformed(row[k], act, colmul, k) * inv;   /* one float32 multiply */
            float n = nearbyintf(p);                               /* ties to even */
            if (n > 127.0f)
                n = 127.0f;
            if (n < -127.0f)
                n = -127.0f;
            qrow[k] = (int8_t)n;
        }
    }
    return err;
}

/* The plain rule: identity transform, no multiplier. */
int orc_quantize_rows(const uint16_t *v, int64_t rows, int64_t K, int8_t *q,
                      float *scale, int nthreads)
{
    return orc_quantize_rows_ex(v, rows, K, ORC_ACT_NONE, NULL, q, scale, nthreads);
}

/* Calibration: amax[k] = max over rows of |T(x[r][k])| (float32, T as above). */
int orc_col_absmax(const uint16_t *x, int64_t rows, int64_t K, int act, float *amax)
{
    if (rows < 0 || K < 0 || (act != ORC_ACT_NONE && act != ORC_ACT_GELU))
        return ORC_ERR_ARG;
    for (int64_t k = 0; k < K; ++k)
        amax[k] = 0.0f;
    for (int64_t r = 0; r < rows; ++r) {
        for (int64_t k = 0; k < K; ++k) {
            if (!isfinite(bf16_bits_to_f32(x[r * K + k])))
                return ORC_ERR_NONFINITE;
            float v = fabsf(transformed(x[r * K + k], act, NULL, k));
            if (v > amax[k])
                amax[k] = v;
        }
    }
    return ORC_OK;
}

/* SmoothQuant factors from calibrated per-channel maxima of X and of W. */
int orc_smooth_factors(const float *ax, const float *aw, int64_t K, float alpha,
                       float *s, float *s_inv)
{
    if (K < 0 || !(alpha >= 0.0f && alpha <= 1.0f))
        return ORC_ERR_ARG;
    for (int64_t k = 0; k < K; ++k) {
        float a = ax[k], b = aw[k];
        float f = 1.0f;
        if (a > 0.0f && b > 0.0f && isfinite(a) && isfinite(b)) {
            if (alpha == 0.5f)
                f = sqrtf(a) / sqrtf(b);
            else
                f = (float)(pow((double)a, (double)alpha) / pow((double)b, 1.0 - (double)alpha));
            if (!(f > 0.0f) || !isfinite(f))
                f = 1.0f;
        }
        s[k] = f;
        s_inv[k] = 1.0f / f;
    }
    return ORC_OK;
}

/* Exact integer product (Section 3, "The fused kernel": int8 x int8 -> int32).
 * xq: [M,K], wq: [N,K] (both K-contiguous), acc: [M,N] row-major. */
int orc_gemm_acc(const int8_t *xq, const int8_t *wq, int64_t M, int64_t N, int64_t K,
                 int32_t *acc, int nthreads)
{
    if (M < 0 || N < 0 || K < 0)
        return ORC_ERR_ARG;
    int err = ORC_OK;
    set_threads(nthreads);
#pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; ++m) {
        for (int64_t n = 0; n < N; ++n) {
            int64_t sum = 0;
            for (int64_t k = 0; k < K; ++k)
                sum += (int64_t)xq[m * K + k] * (int64_t)wq[n * K + k];
            if (sum > INT32_MAX || sum < INT32_MIN) {
#pragma omp atomic write
                err = ORC_ERR_INT32_OVERFLOW;
            }
            acc[m * N + n] = (int32_t)sum;
        }
    }
    return err;
}

/* Epilogue (Section 3, "The fused kernel": per-token scale x per-channel scale on the
 * accumulator, plus bias, dequantized output). bias may be NULL (no bias). */
int orc_epilogue(const int32_t *acc, const float *sx, const float *sw,
                 const uint16_t *bias, int64_t M, int64_t N, uint16_t *y, int nthreads)
{
    if (M < 0 || N < 0)
        return ORC_ERR_ARG;
    if (fegetround() != FE_TONEAREST)
        return ORC_ERR_ROUNDING_MODE;
    set_threads(nthreads);
#pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; ++m) {
        for (int64_t n = 0; n < N; ++n) {
            float b = bias ? bf16_bits_to_f32(bias[n]) : 0.0f;
            float s = sx[m] * sw[n];
            float y32 = fmaf((float)acc[m * N + n], s, b);
            y[m * N + n] = f32_to_bf16_rne(y32);
        }
    }
    return ORC_OK;
}

/* Round a double to bf16 once, nearest-even: the quantum of the binade of |d| (never
 * finer than the subnormal quantum 2^-133) is 2^(e-7); d / quantum is an exact power-
 * of-two scaling, rounded to an integer with ties to even. Overflow goes to infinity. */
static uint16_t f64_to_bf16_rne(double d)
{
    if (isnan(d))
        return 0x7FC0u;
    if (d == 0.0 || isinf(d))
        return f32_to_bf16_rne((float)d);
    int ex;
    frexp(d, &ex);                 /* |d| = f * 2^ex, f in [0.5, 1) */
    int e = ex - 1;                /* 2^e <= |d| < 2^(e+1) */
    if (e < -126)
        e = -126;
    double quantum = ldexp(1.0, e - 7);
    double r = nearbyint(d / quantum) * quantum;
    if (fabs(r) >= ldexp(1.0, 128))
        return (uint16_t)(r > 0 ? 0x7F80u : 0xFF80u);
    return f32_to_bf16_rne((float)r); /* r is a bf16 value: exact in float */
}

uint16_t orc_f64_to_bf16(double d) { return f64_to_bf16_rne(d); }

void orc_f64_to_bf16_array(const double *d, int64_t n, uint16_t *out)
{
    for (int64_t i = 0; i < n; ++i)
        out[i] = f64_to_bf16_rne(d[i]);
}

/* Diagnostic epilogue in double: acc * sx * sw + b with one final rounding to bf16. */
int orc_epilogue_f64(const int32_t *acc, const float *sx, const float *sw,
                     const uint16_t *bias, int64_t M, int64_t N, uint16_t *y,
                     int nthreads)
{
    if (M < 0 || N < 0)
        return ORC_ERR_ARG;
    set_threads(nthreads);
#pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; ++m) {
        for (int64_t n = 0; n < N; ++n) {
            double b = bias ? (double)bf16_bits_to_f32(bias[n]) : 0.0;
            double v = (double)acc[m * N + n] * (double)sx[m] * (double)sw[n] + b;
            y[m * N + n] = f64_to_bf16_rne(v);
        }
    }
    return ORC_OK;
}

/* The whole linear for already-quantized weights: quantize X per token, take the
 * integer product, apply the epilogue. xq/sx/acc are caller-provided scratch. */
int orc_linear(const uint16_t *x, const int8_t *wq, const float *sw,
               const uint16_t *bias, int64_t M, int64_t N, int64_t K, int8_t *xq,
               float *sx, int32_t *acc, uint16_t *y, int nthreads)
{
    int e = orc_quantize_rows(x, M, K, xq, sx, nthreads);
    if (e)
        return e;
    e = orc_gemm_acc(xq, wq, M, N, K, acc, nthreads);
    if (e)
        return e;
    return orc_epilogue(acc, sx, sw, bias, M, N, y, nthreads);
}
