/*
 * Memory and undefined-behaviour check of the CPU oracle (test infrastructure).
 *
 * Built with AddressSanitizer and UndefinedBehaviorSanitizer (and leak
 * checking) by tests/test_sanitizers.py, once per arithmetic of the oracle
 * (OQ_REAL double and float).  It includes the oracle's source so that its
 * internal types are visible, and drives every routine over the whole
 * configuration space on small ragged shapes: both gates, every code format,
 * the three update rules, windows of 1, 3 and 8 tokens, 0 and 3 Compensator
 * Tokens, smoothing on and off, exact and FP16 records, quantized and exact
 * windows.  It checks only that every output is finite and that the storage
 * format conversions round-trip over all their codes; the arithmetic itself
 * is pinned by the Python tests.
 */
#include "../../oracle/lq_oracle.c"

#include <stdio.h>

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;

/* splitmix64 (Steele, Lea and Flood, 2014), mapped to [-1, 1) */
static double urand(void)
{
    uint64_t z = (rng_state += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    z ^= z >> 31;
    return (double)(z >> 11) * (2.0 / 9007199254740992.0) - 1.0;
}

static int failures = 0;

static void check_finite(const char *what, const double *x, size_t n)
{
    for (size_t i = 0; i < n; ++i)
        if (!isfinite(x[i])) {
            fprintf(stderr, "non-finite %s[%zu]\n", what, i);
            ++failures;
            return;
        }
}

static void unit_rows(float *x, int rows, int d)
{
    for (int r = 0; r < rows; ++r) {
        double s = 0;
        for (int i = 0; i < d; ++i) {
            x[(size_t)r * d + i] = (float)urand();
            s += (double)x[(size_t)r * d + i] * x[(size_t)r * d + i];
        }
        for (int i = 0; i < d; ++i) x[(size_t)r * d + i] = (float)(x[(size_t)r * d + i] / sqrt(s));
    }
}

static void run_case(int dk, int dv, int gate, int code, int rule, int W, int r, int smooth,
                     int quantize, int round_records)
{
    const lqo_cfg cfg = {dk, dv, W, r, 3, gate, code, smooth, quantize, round_records, rule};
    const int tiles = 2, T = 2 * W + 1, g = gate ? dk : 1, n_snap = n_snap_of(&cfg, T);
    const size_t TS = (size_t)tiles * T, D = (size_t)dk * dv;
    float *q = malloc(sizeof(float) * TS * dk), *k = malloc(sizeof(float) * TS * dk);
    float *b = rule == 2 ? malloc(sizeof(float) * TS * dk) : NULL;
    float *v = malloc(sizeof(float) * TS * dv), *alpha = malloc(sizeof(float) * TS * g);
    float *beta = malloc(sizeof(float) * TS);
    double *S0 = malloc(sizeof(double) * tiles * D);
    unit_rows(q, (int)TS, dk);
    unit_rows(k, (int)TS, dk);
    if (b) unit_rows(b, (int)TS, dk);
    for (size_t i = 0; i < TS * dv; ++i) v[i] = (float)urand();
    for (size_t i = 0; i < TS * g; ++i) alpha[i] = (float)(0.9 + 0.1 * fabs(urand()));
    for (size_t i = 0; i < TS; ++i) beta[i] = (float)(0.5 + 0.5 * fabs(urand()));
    for (size_t i = 0; i < tiles * D; ++i) S0[i] = urand() * (i % 17 == 0 ? 20.0 : 1.0);
    const lqo_inputs in = {q, k, v, alpha, beta, b};

    const size_t cb = code_bytes(&cfg), rr = r ? r : 1;
    lqo_outputs out = {0};
    out.Z = malloc(cb * tiles * n_snap * D);
    out.delta = malloc(sizeof(float) * tiles * n_snap * dv);
    out.c = malloc(sizeof(float) * tiles * n_snap * dk);
    out.Kt = malloc(sizeof(double) * tiles * n_snap * rr * dk);
    out.Ut = malloc(sizeof(double) * tiles * n_snap * rr * dv);
    out.S_final = malloc(sizeof(double) * tiles * D);
    out.rec_a = malloc(sizeof(double) * tiles * W * g);
    out.rec_k = malloc(sizeof(double) * tiles * W * dk);
    out.rec_u = malloc(sizeof(double) * tiles * W * dv);
    out.rec_len = malloc(sizeof(int32_t) * tiles);
    out.hist_a = malloc(sizeof(double) * TS * g);
    out.hist_k = malloc(sizeof(double) * TS * dk);
    out.hist_u = malloc(sizeof(double) * TS * dv);
    double *o = malloc(sizeof(double) * TS * dv);

    OQ(run_dense)(&cfg, tiles, T, S0, &in, o, &out, 2);
    check_finite("run_dense o", o, TS * dv);
    check_finite("run_dense S_final", out.S_final, tiles * D);
    check_finite("run_dense hist_k", out.hist_k, TS * dk);
    OQ(run_readout)(&cfg, tiles, T, S0, &in, o, &out, 2);
    check_finite("run_readout o", o, TS * dv);
    for (int mode = 0; mode < 3; ++mode) {
        OQ(run_baseline)(&cfg, tiles, T, S0, &in, o, out.S_final, mode, 2);
        check_finite("run_baseline o", o, TS * dv);
    }
    double drift[2 * 64], odrift[2 * 64];
    OQ(run_drift)(&cfg, tiles, T, 2, S0, &in, drift, odrift, 2);
    check_finite("run_drift", drift, (size_t)tiles * (T / 2));

    /* the single-token entry points on tile 0 */
    uint8_t *Z = malloc(cb * D);
    float *delta = malloc(sizeof(float) * dv), *c = malloc(sizeof(float) * dk);
    double *Kt = calloc(rr * dk, sizeof(double)), *Ut = calloc(rr * dv, sizeof(double));
    double *S = malloc(sizeof(double) * D), *Sd = malloc(sizeof(double) * D);
    double *ra = malloc(sizeof(double) * W * g), *rk = malloc(sizeof(double) * W * dk);
    double *ru = malloc(sizeof(double) * W * dv), *o1 = malloc(sizeof(double) * dv);
    OQ(quantize)(&cfg, S0, Z, delta, c, Kt, Ut);
    OQ(dequantize)(&cfg, Z, delta, c, Kt, Ut, Sd);
    check_finite("dequantize", Sd, D);
    memcpy(S, Sd, sizeof(double) * D);
    for (int s = 0; s < W; ++s) {
        OQ(readout_step)(&cfg, Z, delta, c, Kt, Ut, Sd, ra, rk, ru, s, q + (size_t)s * dk,
                         k + (size_t)s * dk, b ? b + (size_t)s * dk : NULL, v + (size_t)s * dv,
                         alpha + (size_t)s * g, beta[s], o1, ra + (size_t)s * g, rk + (size_t)s * dk,
                         ru + (size_t)s * dv);
        check_finite("readout_step", o1, dv);
        OQ(window_step)(&cfg, S, q + (size_t)s * dk, k + (size_t)s * dk, b ? b + (size_t)s * dk : NULL,
                        v + (size_t)s * dv, alpha + (size_t)s * g, beta[s], o1, ra + (size_t)s * g,
                        rk + (size_t)s * dk, ru + (size_t)s * dv);
        OQ(recurrent_step)(&cfg, Sd, q + (size_t)s * dk, k + (size_t)s * dk,
                           b ? b + (size_t)s * dk : NULL, v + (size_t)s * dv, alpha + (size_t)s * g,
                           beta[s], o1, s % 3);
    }
    OQ(dequantize)(&cfg, Z, delta, c, Kt, Ut, Sd);
    OQ(reconstruct)(&cfg, Z, delta, c, Kt, Ut, Sd, ra, rk, ru, W, S);
    check_finite("reconstruct", S, D);

    free(Z); free(delta); free(c); free(Kt); free(Ut); free(S); free(Sd);
    free(ra); free(rk); free(ru); free(o1);
    free(out.Z); free(out.delta); free(out.c); free(out.Kt); free(out.Ut); free(out.S_final);
    free(out.rec_a); free(out.rec_k); free(out.rec_u); free(out.rec_len);
    free(out.hist_a); free(out.hist_k); free(out.hist_u); free(o);
    free(q); free(k); free(b); free(v); free(alpha); free(beta); free(S0);
}

static void check_formats(void)
{
    for (uint32_t h = 0; h < 65536; ++h) {
        const float x = lqo_f16_to_f32((uint16_t)h);
        if (x == x && lqo_f32_to_f16(x) != h && !(x == 0.0f)) {
            fprintf(stderr, "f16 round trip %04x\n", h);
            ++failures;
        }
        const float y = lqo_bf16_to_f32((uint16_t)h);
        if (y == y && lqo_f32_to_bf16(y) != h) {
            fprintf(stderr, "bf16 round trip %04x\n", h);
            ++failures;
        }
    }
    for (uint32_t e = 0; e < 256; ++e) {
        const float x = lqo_e4m3_to_f32((uint8_t)e);
        if (x == x && x != 0.0f && lqo_f32_to_e4m3(x) != e) {
            fprintf(stderr, "e4m3 round trip %02x\n", e);
            ++failures;
        }
    }
    /* every conversion over a spread of fp32 bit patterns, specials included */
    for (uint64_t i = 0; i < (1ull << 32); i += 65537) {
        const uint32_t u = (uint32_t)i;
        float x;
        memcpy(&x, &u, sizeof(x));
        (void)lqo_f32_to_f16(x);
        (void)lqo_f32_to_bf16(x);
        (void)lqo_f32_to_e4m3(x);
    }
}

int main(void)
{
    check_formats();
    for (int gate = 0; gate < 2; ++gate)
        for (int code = 0; code < 5; ++code)
            for (int rule = 0; rule < 3; ++rule)
                for (int wi = 0; wi < 3; ++wi) {
                    const int W = wi == 0 ? 1 : wi == 1 ? 3 : 8;
                    const int r = code == 4 ? 0 : (wi % 2) * 3;
                    const int smooth = code == 4 ? 0 : (rule + wi) % 2;
                    run_case(16, 24, gate, code, rule, W, r, smooth, 1, (gate + wi) % 2);
                    if (wi == 1) run_case(16, 24, gate, code, rule, W, r, smooth, 0, 1);
                }
    run_case(128, 128, 1, 0, 0, 4, 8, 1, 1, 1);
    if (failures) {
        fprintf(stderr, "%d failures\n", failures);
        return 1;
    }
    printf("oracle sanitizer check ok\n");
    return 0;
}
