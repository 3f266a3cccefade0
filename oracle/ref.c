/*
 * CPU oracle for SiFAR's one-shot all-reduce (test infrastructure only).
 *
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * may load this library. It shares no code, header or constant with the GPU
 * library; it is the plain definition of what the GPU path must compute,
 * written for a reader to check by eye against the paper:
 *
 *  - Reduction (Sec. 4.2, the one-shot pull-and-reduce listing; Sec. 3.1,
 *    "Oneshot"): every rank's partial is added into one result, peer after
 *    peer in ascending rank order. The element type of the payload is bf16 and
 *    the accumulator is fp32 (the paper leaves both unstated; 4-8 KB per token
 *    at batch 1 in Sec. 3.2 implies 2-byte elements). Each add is an IEEE
 *    binary32 add rounded to nearest-even with subnormals kept; the fp32 sum
 *    is then rounded once more, to bf16, to nearest-even.
 *  - Speculation, validation, retries and dual buffering never change this
 *    value (Sec. 3.5 and 4.1: a mis-speculated reduction is simply re-run).
 *  - Residual-add + RMSNorm epilogue: the paper is silent on it. It is defined
 *    here as the unfused chain of plain bf16 operations, computed in fp64 and
 *    rounded once to bf16 (see oracle_residual_rmsnorm).
 *
 * Build: gcc -O2 -fno-fast-math -ffp-contract=off -fPIC -shared ref.c -lm
 * No vector intrinsics, no reassociation; bf16 values are decoded and encoded
 * from sign, exponent and significand, never by reinterpreting float bits.
 */
#include <fenv.h>
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <xmmintrin.h>

/* ---- bf16 <-> real number, by definition ------------------------------- */
/* bf16: 1 sign bit, 8 exponent bits (bias 127), 7 fraction bits. Normal
 * values (1 + f/128) * 2^(e-127); subnormal values (f/128) * 2^-126. */

double oracle_bf16_value(uint16_t b)
{
    int sign = (b >> 15) & 1;
    int e = (b >> 7) & 0xFF;
    int f = b & 0x7F;
    double v;
    if (e == 0xFF)
        v = (f == 0) ? INFINITY : NAN;
    else if (e == 0)
        v = ldexp((double)f, -133);             /* (f/128) * 2^-126 */
    else
        v = ldexp((double)(128 + f), e - 134);  /* (1+f/128) * 2^(e-127) */
    return sign ? -v : v;
}

/* Encode a real that is exactly a finite bf16 value (or an infinity). */
static uint16_t encode_exact(double r, int sign)
{
    uint16_t s = (uint16_t)(sign << 15);
    if (isinf(r))
        return s | 0x7F80;
    if (r == 0.0)
        return s;
    if (r < ldexp(1.0, -126)) {                 /* subnormal: r = f * 2^-133 */
        double f = ldexp(r, 133);
        return s | (uint16_t)f;
    }
    int e2;
    double m = frexp(r, &e2);                   /* r = m * 2^e2, m in [0.5,1) */
    int biased = e2 - 1 + 127;                  /* r = (2m) * 2^(e2-1) */
    int f = (int)ldexp(2.0 * m - 1.0, 7);
    return s | (uint16_t)(biased << 7) | (uint16_t)f;
}

/* Round a real (given as a double) to the nearest bf16, ties to even.
 * NaN maps to a quiet NaN of the same sign (NaN payloads are outside the
 * contract: only "a NaN in gives a NaN out" is specified). */
uint16_t oracle_bf16_round(double x)
{
    int sign = signbit(x) ? 1 : 0;
    if (isnan(x))
        return (uint16_t)((sign << 15) | 0x7FC0);
    double ax = fabs(x);
    if (isinf(ax) || ax >= ldexp(1.0, 128))
        return encode_exact(INFINITY, sign);
    if (ax == 0.0)
        return encode_exact(0.0, sign);
    /* The spacing of bf16 values around ax: 8 significant bits for normal
     * numbers, a fixed 2^-133 in the subnormal range. */
    int e2;
    (void)frexp(ax, &e2);                       /* ax in [2^(e2-1), 2^e2) */
    int ulp_exp = e2 - 8;
    if (ulp_exp < -133)
        ulp_exp = -133;
    double q = ldexp(ax, -ulp_exp);             /* exact: scaling by 2^k */
    q = nearbyint(q);                           /* FE_TONEAREST: ties to even */
    double r = ldexp(q, ulp_exp);
    if (r >= ldexp(1.0, 128))
        r = INFINITY;
    return encode_exact(r, sign);
}

/* Element-wise versions of the two conversions, for bulk checks. */
void oracle_bf16_round_array(const double *x, size_t count, uint16_t *out)
{
    for (size_t i = 0; i < count; ++i)
        out[i] = oracle_bf16_round(x[i]);
}

void oracle_bf16_value_array(const uint16_t *b, size_t count, double *out)
{
    for (size_t i = 0; i < count; ++i)
        out[i] = oracle_bf16_value(b[i]);
}

/* ---- the reduction --------------------------------------------------------
 * out[i] = bf16( (((x_0[i] + x_1[i]) + x_2[i]) + ...) + x_{N-1}[i] ),
 * each '+' an fp32 add; x_r[i] = x[r * rank_stride + i].
 * The accumulator starts from rank 0's value, not from +0, so an all -0 input
 * sums to -0 (Sec. 4.2's listing leaves the initial value unstated). */
void oracle_reduce(const uint16_t *x, int nranks, size_t rank_stride, size_t count,
                   uint16_t *out)
{
    for (size_t i = 0; i < count; ++i) {
        float acc = (float)oracle_bf16_value(x[i]);
        for (int r = 1; r < nranks; ++r) {
            float v = (float)oracle_bf16_value(x[(size_t)r * rank_stride + i]);
            acc = acc + v;
        }
        out[i] = oracle_bf16_round((double)acc);
    }
}

/* ---- residual-add + RMSNorm epilogue (paper silent; fp64 reading) ----------
 * For each token t (row of `hidden` elements):
 *   res'[h] = bf16( a[h] + res[h] )                      (stored back into res)
 *   ms      = (sum_h res'[h]^2) / hidden                 (h ascending, fp64)
 *   y[h]    = bf16( res'[h] * w[h] / sqrt(ms + eps) )
 * a is the all-reduce output (already bf16). All arithmetic is fp64 with one
 * rounding to bf16 per stored value. */
void oracle_residual_rmsnorm(const uint16_t *a, uint16_t *res, const uint16_t *w,
                             int tokens, int hidden, double eps, uint16_t *y)
{
    for (int t = 0; t < tokens; ++t) {
        const uint16_t *at = a + (size_t)t * hidden;
        uint16_t *rt = res + (size_t)t * hidden;
        uint16_t *yt = y + (size_t)t * hidden;
        double ss = 0.0;
        for (int h = 0; h < hidden; ++h) {
            rt[h] = oracle_bf16_round(oracle_bf16_value(at[h]) + oracle_bf16_value(rt[h]));
            double v = oracle_bf16_value(rt[h]);
            ss += v * v;
        }
        double inv = 1.0 / sqrt(ss / (double)hidden + eps);
        for (int h = 0; h < hidden; ++h)
            yt[h] = oracle_bf16_round(oracle_bf16_value(rt[h]) * inv *
                                      oracle_bf16_value(w[h]));
    }
}

/* The floating-point environment this oracle assumes: round to nearest, no
 * flush-to-zero, no denormals-are-zero. Returns 1 when it holds. */
int oracle_fp_env_ok(void)
{
    unsigned csr = _mm_getcsr();
    int ftz = (csr >> 15) & 1, daz = (csr >> 6) & 1;
    return fegetround() == FE_TONEAREST && !ftz && !daz;
}
