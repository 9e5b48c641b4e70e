/*
 * Storage-format rounding for the LeapQuant CPU oracle.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; only the test-suite, the smoke check and the CPU-baseline
 * leg of the benchmark use it.
 *
 * The paper fixes three narrow storage formats for the decode path
 * (Sec. 4.1 "Implementation"): FP16 Compensator Tokens, an FP16 buffer of
 * window records, FP32 smoothing scales; the per-step BF16 state is one of its
 * baselines (Sec. 4.1 "Baselines").  The FP8 (OCP E4M3FN) code format is the
 * 8-bit floating-point alternative to INT8 codes.  Every conversion here is
 * written from the definition of the format: the value is rounded to the
 * nearest representable number, ties to the one whose last fraction bit is 0.
 *
 *   binary16 : 10 fraction bits, minimum normal exponent -14, max 65504
 *   bfloat16 :  7 fraction bits, minimum normal exponent -126
 *   E4M3FN   :  3 fraction bits, minimum normal exponent -6, max 448,
 *               no infinities, S.1111.111 is NaN (callers saturate first)
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

/* Round a >= 0 (finite) to the grid of a binary format with `mbits` fraction
 * bits whose smallest normal exponent is `emin`.  Below 2^emin the grid is the
 * subnormal grid 2^(emin-mbits).  a/spacing and the product back are exact
 * power-of-two scalings, so the only rounding is the one rint() performs in the
 * default round-to-nearest-even mode. */
static double round_to_grid(double a, int mbits, int emin)
{
    if (a == 0.0) return 0.0;
    int e;
    frexp(a, &e);            /* a = f * 2^e, f in [0.5, 1): floor(log2 a) = e-1 */
    int E = e - 1;
    if (E < emin) E = emin;
    double spacing = ldexp(1.0, E - mbits);
    return rint(a / spacing) * spacing;
}

/* ---------------- binary16 ---------------- */

uint16_t lqo_f32_to_f16(float x)
{
    uint32_t bits;
    memcpy(&bits, &x, 4);
    uint16_t sign = (uint16_t)((bits >> 16) & 0x8000u);
    if (isnan(x)) return (uint16_t)(sign | 0x7e00u);
    double a = fabs((double)x);
    if (isinf(x)) return (uint16_t)(sign | 0x7c00u);
    double r = round_to_grid(a, 10, -14);
    if (r >= 65536.0) return (uint16_t)(sign | 0x7c00u);          /* overflow -> inf */
    if (r < ldexp(1.0, -14)) {                                    /* subnormal or zero */
        return (uint16_t)(sign | (uint16_t)ldexp(r, 24));         /* count of 2^-24 */
    }
    int e;
    double f = frexp(r, &e);                                      /* r = f*2^e */
    int E = e - 1;                                                /* r in [2^E, 2^(E+1)) */
    uint16_t frac = (uint16_t)((f * 2.0 - 1.0) * 1024.0);
    return (uint16_t)(sign | (uint16_t)((E + 15) << 10) | frac);
}

float lqo_f16_to_f32(uint16_t h)
{
    int s = (h >> 15) & 1, E = (h >> 10) & 31, m = h & 1023;
    double v;
    if (E == 31) v = m ? NAN : INFINITY;
    else if (E == 0) v = ldexp((double)m, -24);
    else v = ldexp(1.0 + m / 1024.0, E - 15);
    return (float)(s ? -v : v);
}

/* ---------------- bfloat16 ---------------- */

uint16_t lqo_f32_to_bf16(float x)
{
    uint32_t bits;
    memcpy(&bits, &x, 4);
    uint16_t sign = (uint16_t)((bits >> 16) & 0x8000u);
    if (isnan(x)) return (uint16_t)(sign | 0x7fc0u);
    if (isinf(x)) return (uint16_t)(sign | 0x7f80u);
    double a = fabs((double)x);
    double r = round_to_grid(a, 7, -126);
    if (r >= ldexp(1.0, 128)) return (uint16_t)(sign | 0x7f80u);
    float rf = (float)r;                       /* exact: r has <= 8 significant bits */
    uint32_t rb;
    memcpy(&rb, &rf, 4);
    return (uint16_t)(sign | (uint16_t)(rb >> 16));
}

float lqo_bf16_to_f32(uint16_t b)
{
    uint32_t bits = (uint32_t)b << 16;
    float f;
    memcpy(&f, &bits, 4);
    return f;
}

/* ---------------- OCP FP8 E4M3FN ---------------- */

/* Encode with round-to-nearest-even.  The caller clamps to [-448, 448]; any
 * larger magnitude saturates to 448 here as well. */
uint8_t lqo_f32_to_e4m3(float x)
{
    uint8_t sign = signbit(x) ? 0x80u : 0x00u;
    if (isnan(x)) return (uint8_t)(sign | 0x7fu);
    double a = fabs((double)x);
    if (a > 448.0) a = 448.0;
    double r = round_to_grid(a, 3, -6);
    if (r > 448.0) r = 448.0;
    if (r < ldexp(1.0, -6)) return (uint8_t)(sign | (uint8_t)ldexp(r, 9));  /* count of 2^-9 */
    int e;
    double f = frexp(r, &e);
    int E = e - 1;
    uint8_t frac = (uint8_t)((f * 2.0 - 1.0) * 8.0);
    return (uint8_t)(sign | (uint8_t)((E + 7) << 3) | frac);
}

float lqo_e4m3_to_f32(uint8_t b)
{
    int s = (b >> 7) & 1, E = (b >> 3) & 15, m = b & 7;
    double v;
    if (E == 15 && m == 7) v = NAN;
    else if (E == 0) v = ldexp((double)m, -9);
    else v = ldexp(1.0 + m / 8.0, E - 7);
    return (float)(s ? -v : v);
}

/* Bulk helpers for the Python wrapper. */
void lqo_f32_to_f16_n(const float *x, uint16_t *y, long n)
{
    for (long i = 0; i < n; ++i) y[i] = lqo_f32_to_f16(x[i]);
}
void lqo_f32_to_bf16_n(const float *x, uint16_t *y, long n)
{
    for (long i = 0; i < n; ++i) y[i] = lqo_f32_to_bf16(x[i]);
}
void lqo_f32_to_e4m3_n(const float *x, uint8_t *y, long n)
{
    for (long i = 0; i < n; ++i) y[i] = lqo_f32_to_e4m3(x[i]);
}
void lqo_e4m3_to_f32_n(const uint8_t *x, float *y, long n)
{
    for (long i = 0; i < n; ++i) y[i] = lqo_e4m3_to_f32(x[i]);
}
