/*
 * LeapQuant CPU oracle: a plain, slow, obviously-correct statement of what the
 * 8-bit recurrent-state decode path computes.
 *
 * TEST INFRASTRUCTURE ONLY.  The product library never links, loads or calls
 * this code; only the tests, the smoke check and the CPU-baseline leg of the
 * benchmark do.  It shares no code, header, table or constant with the HIP
 * path.
 *
 * The file is compiled twice: with OQ_REAL=double (the oracle proper, prefix
 * lqo64_) and with OQ_REAL=float (an fp32 twin used only by self-checks and
 * diagnostics, prefix lqo32_).  Interface arrays are always double / float /
 * byte; only the internal arithmetic type changes.
 *
 * Notation follows the paper.  One (request, head) tile has a state
 * S in R^{dk x dv}, stored row-major as S[k*dv + v]; outputs o = S^T q.
 *
 *   O1  recurrence, Sec. 3.1 Eq. (general) with the GDN / KDA rows of the
 *       instance table (App. A): A = D_t S, u = v - A^T k, S = A + beta k u^T,
 *       o = S^T q.  The rows with b_t = 0 (linear attention, RetNet, Mamba2,
 *       GLA / RWKV6 / HGRN2) drop the read: u = v (cfg->rule = 1).  Because the read vector is b = alpha k (GDN) or alpha.k
 *       (KDA) and D_t is diagonal, S_{t-1}^T b = (D_t S_{t-1})^T k.  With
 *       cfg->rule = 2 the read vector is an input of its own, u = v - S_{t-1}^T b
 *       (the general form, App. A; the erase sub-step of RWKV7, whose read
 *       vector a.kappa is not the decay times the write key).
 *   O2  quantizer: Compensator Tokens (Sec. 3.3, Eqs. (compensator),
 *       (compensator-rank-r)), fitted by power iteration (Sec. 4.1), then
 *       residual smoothing (Sec. 3.4) and per-value-channel symmetric INT8
 *       (App. B.3) or E4M3 codes.
 *   O3  per-window method, dense form (Sec. 3.2, Eqs. (record), (window)):
 *       the state is carried densely inside a window, records are buffered in
 *       FP16, and the state is re-quantized only at the window end.
 *   O4  per-window method, readout form (App. B.2 Eq. (readout), App. B.3
 *       Eq. (smooth-readout)) and window-end reconstruction (Sec. 3.4
 *       Eq. (smooth)): outputs from the fixed quantized base plus records,
 *       never forming a dk x dv intermediate.
 *   O5  baselines: O1 with the state rounded to fp32 or bf16 after each step
 *       (Sec. 4.1 "Baselines").
 *
 * Readings of points the paper leaves open are listed where they are used:
 * power-iteration start vector and deflation, where the FP16 rounding of the
 * compensators happens, the smoothing floor, zero columns, tie rounding.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifndef OQ_REAL
#define OQ_REAL double
#endif
#ifndef OQ
#define OQ(n) lqo64_##n
#endif
typedef OQ_REAL real;

/* storage formats (lq_formats.c) */
uint16_t lqo_f32_to_f16(float x);
float lqo_f16_to_f32(uint16_t h);
uint16_t lqo_f32_to_bf16(float x);
float lqo_bf16_to_f32(uint16_t b);
uint8_t lqo_f32_to_e4m3(float x);
float lqo_e4m3_to_f32(uint8_t b);

typedef struct {
    int32_t dk, dv;
    int32_t window;        /* W: records buffered before the state is re-quantized */
    int32_t n_comp;        /* r: Compensator Tokens */
    int32_t power_iters;   /* power-iteration sweeps per token */
    int32_t gate;          /* 0: scalar decay (GDN); 1: per-key-channel decay (KDA) */
    int32_t code;          /* 0: INT8; 1: FP8 E4M3FN; 2: INT4; 3: INT6 codes; 4: BF16 state
                            * (the window end rounds the state to BF16: unit scales,
                            * no smoothing, no Compensator Tokens) */
    int32_t smooth;        /* 1: residual smoothing; 0: c = 1 */
    int32_t quantize;      /* 1: quantize at window ends; 0: keep the state exact */
    int32_t round_records; /* 1: FP16 records (alpha, write key, correction); 0: exact */
    int32_t rule;          /* 0: delta rule (b_t = D_t k_t); 1: additive (b_t = 0);
                            * 2: general, b_t given with the token */
} lqo_cfg;

enum { LQO_STATE_EXACT = 0, LQO_STATE_F32 = 1, LQO_STATE_BF16 = 2 };

/* Value of x after rounding to binary16, decided in fp32 like any fp32 producer. */
static real f16v(real x) { return (real)lqo_f16_to_f32(lqo_f32_to_f16((float)x)); }
static real rec_round(const lqo_cfg *cfg, real x) { return cfg->round_records ? f16v(x) : x; }

/* Codes are held one per byte here (the packing of 4- and 6-bit codes is a
 * storage layout, not arithmetic): integer codes as two's-complement bytes,
 * E4M3 codes as their bit pattern; the BF16 state as two bytes per entry. */
static size_t code_bytes(const lqo_cfg *cfg) { return cfg->code == 4 ? 2 : 1; }

static real code_value(const lqo_cfg *cfg, const uint8_t *Z, size_t i)
{
    if (cfg->code == 4) return (real)lqo_bf16_to_f32(((const uint16_t *)Z)[i]);
    if (cfg->code == 1) return (real)lqo_e4m3_to_f32(Z[i]);
    return (real)(int8_t)Z[i];
}

/* Largest code magnitude: 2^(b-1) - 1 for b-bit symmetric integers, 448 for E4M3. */
static float code_qmax(const lqo_cfg *cfg)
{
    switch (cfg->code) {
    case 1: return 448.0f;
    case 2: return 7.0f;
    case 3: return 31.0f;
    default: return 127.0f;
    }
}

/* ------------------------------------------------------------------------ */
/* O2: quantizer.                                                            */
/* ------------------------------------------------------------------------ */

/*
 * Compensator Tokens: r rank-one pairs (k~_h, u~_h) fitted to S one after the
 * other (sequential deflation).  Reading of the unspecified fit: for each pair
 *   x <- row l2 norms of the current residual M, normalised (zero -> pair 0)
 *   n_iter times: y <- M^T x; x <- M y; x <- x * (1/||x||) (zero -> pair 0)
 *   k~ <- fp16(x);  u~ <- fp16(M^T k~) evaluated with the rounded k~
 *   M <- M - k~ u~^T with the rounded pair,
 * so the quantized residual absorbs the FP16 rounding of the pair.  u~ = M^T k~
 * is the least-squares optimum for the unit vector k~; with enough sweeps the
 * pairs reach the leading singular pairs (Eckart-Young, Sec. 3.3).
 *
 * Residual smoothing (Sec. 3.4): c_k = sqrt(max(mean_v |R_kv|, 1e-12)) rounded
 * to fp32; the smoothed residual is R_kv * (1/c_k).
 *
 * Codes (App. B.3): per value channel v, a_v = max_k |R^C_kv|.  INT8:
 * delta_v = a_v/127, code = clamp(rint(R^C_kv * (127/a_v)), -127, 127), ties to
 * even.  E4M3: delta_v = a_v/448, code = e4m3(clamp(R^C_kv * (448/a_v), +-448)).
 * The 6- and 4-bit variants (Sec. 4.1, 4.2) read the same per-value-channel
 * symmetric rule with qmax = 2^(b-1) - 1: 31 and 7.
 * A zero column gets delta_v = 0 and zero codes.  The code decision is taken in
 * fp32 from the fp32-rounded residual, as the GPU takes it.
 */
static void quantize_impl(const lqo_cfg *cfg, const double *S_in, uint8_t *Z, float *delta,
                          float *c, double *Kt, double *Ut)
{
    const int dk = cfg->dk, dv = cfg->dv, r = cfg->n_comp;
    if (cfg->code == 4) {
        /* BF16 state (the per-window BF16 variant of Sec. 3.2): each entry rounded
         * to nearest even through fp32, unit scales, no tokens (r must be 0). */
        for (int i = 0; i < dk * dv; ++i) ((uint16_t *)Z)[i] = lqo_f32_to_bf16((float)S_in[i]);
        for (int k = 0; k < dk; ++k) c[k] = 1.0f;
        for (int v = 0; v < dv; ++v) delta[v] = 1.0f;
        return;
    }
    real *M = (real *)malloc(sizeof(real) * (size_t)dk * dv);
    real *x = (real *)malloc(sizeof(real) * (size_t)dk);
    real *y = (real *)malloc(sizeof(real) * (size_t)dv);
    for (int i = 0; i < dk * dv; ++i) M[i] = (real)S_in[i];

    for (int h = 0; h < r; ++h) {
        double *kh = Kt + (size_t)h * dk, *uh = Ut + (size_t)h * dv;
        for (int k = 0; k < dk; ++k) {
            real s = 0;
            for (int v = 0; v < dv; ++v) s += M[k * dv + v] * M[k * dv + v];
            x[k] = sqrt(s);
        }
        real n = 0;
        for (int k = 0; k < dk; ++k) n += x[k] * x[k];
        n = sqrt(n);
        int ok = n > 0;
        if (ok) {
            real inv = (real)1 / n;
            for (int k = 0; k < dk; ++k) x[k] *= inv;
        }
        for (int it = 0; ok && it < cfg->power_iters; ++it) {
            for (int v = 0; v < dv; ++v) {
                real s = 0;
                for (int k = 0; k < dk; ++k) s += M[k * dv + v] * x[k];
                y[v] = s;
            }
            for (int k = 0; k < dk; ++k) {
                real s = 0;
                for (int v = 0; v < dv; ++v) s += M[k * dv + v] * y[v];
                x[k] = s;
            }
            n = 0;
            for (int k = 0; k < dk; ++k) n += x[k] * x[k];
            n = sqrt(n);
            if (!(n > 0)) { ok = 0; break; }
            real inv = (real)1 / n;
            for (int k = 0; k < dk; ++k) x[k] *= inv;
        }
        if (!ok) {
            for (int k = 0; k < dk; ++k) kh[k] = 0;
            for (int v = 0; v < dv; ++v) uh[v] = 0;
            continue;
        }
        for (int k = 0; k < dk; ++k) kh[k] = (double)f16v(x[k]);
        for (int v = 0; v < dv; ++v) {
            real s = 0;
            for (int k = 0; k < dk; ++k) s += M[k * dv + v] * (real)kh[k];
            uh[v] = (double)f16v(s);
        }
        for (int k = 0; k < dk; ++k)
            for (int v = 0; v < dv; ++v) M[k * dv + v] -= (real)kh[k] * (real)uh[v];
    }

    /* residual smoothing over key rows */
    for (int k = 0; k < dk; ++k) {
        if (!cfg->smooth) { c[k] = 1.0f; continue; }
        real s = 0;
        for (int v = 0; v < dv; ++v) s += fabs(M[k * dv + v]);
        real m = s / dv;
        if (m < (real)1e-12f) m = (real)1e-12f;
        c[k] = (float)sqrt(m);
    }

    /* per-value-channel symmetric codes, decided in fp32 */
    const float qmax = code_qmax(cfg);
    for (int v = 0; v < dv; ++v) {
        float amax = 0.0f;
        for (int k = 0; k < dk; ++k) {
            float ic = 1.0f / c[k];
            float rc = (float)M[k * dv + v] * ic;
            if (fabsf(rc) > amax) amax = fabsf(rc);
        }
        if (amax == 0.0f) {
            delta[v] = 0.0f;
            for (int k = 0; k < dk; ++k) Z[k * dv + v] = 0;
            continue;
        }
        delta[v] = amax / qmax;
        float inv = qmax / amax;
        for (int k = 0; k < dk; ++k) {
            float ic = 1.0f / c[k];
            float rc = (float)M[k * dv + v] * ic;
            float t = rc * inv;
            if (cfg->code == 1) {
                if (t > 448.0f) t = 448.0f;
                if (t < -448.0f) t = -448.0f;
                Z[k * dv + v] = lqo_f32_to_e4m3(t);
            } else {
                float q = rintf(t);
                if (q > qmax) q = qmax;
                if (q < -qmax) q = -qmax;
                Z[k * dv + v] = (uint8_t)(int8_t)q;
            }
        }
    }
    free(M);
    free(x);
    free(y);
}

void OQ(quantize)(const lqo_cfg *cfg, const double *S, uint8_t *Z, float *delta, float *c,
                  double *Kt, double *Ut)
{
    quantize_impl(cfg, S, Z, delta, c, Kt, Ut);
}

/* Dequantized state: S~_kv = c_k * (code_kv * delta_v) + sum_h k~_h[k] u~_h[v]
 * (Sec. 3.3 Eq. (compensator-rank-r) with the smoothing of Sec. 3.4). */
void OQ(dequantize)(const lqo_cfg *cfg, const uint8_t *Z, const float *delta, const float *c,
                    const double *Kt, const double *Ut, double *S)
{
    const int dk = cfg->dk, dv = cfg->dv;
    for (int k = 0; k < dk; ++k)
        for (int v = 0; v < dv; ++v) {
            real s = (real)c[k] * (code_value(cfg, Z, (size_t)k * dv + v) * (real)delta[v]);
            for (int h = 0; h < cfg->n_comp; ++h)
                s += (real)Kt[(size_t)h * dk + k] * (real)Ut[(size_t)h * dv + v];
            S[k * dv + v] = (double)s;
        }
}

/* ------------------------------------------------------------------------ */
/* O1 / O5: one step of the recurrence on a dense state.                     */
/* ------------------------------------------------------------------------ */

static real state_round(int mode, real x)
{
    if (mode == LQO_STATE_F32) return (real)(float)x;
    if (mode == LQO_STATE_BF16) return (real)lqo_bf16_to_f32(lqo_f32_to_bf16((float)x));
    return x;
}

static void recurrent_step_impl(const lqo_cfg *cfg, real *S, const float *q, const float *k,
                                const float *b, const float *vv, const float *alpha, float beta,
                                double *o, int mode, real *w)
{
    const int dk = cfg->dk, dv = cfg->dv;
    if (cfg->rule == 2)
        for (int v = 0; v < dv; ++v) {
            real s = 0;
            for (int i = 0; i < dk; ++i) s += S[i * dv + v] * (real)b[i];  /* S_{t-1}^T b */
            w[v] = (real)vv[v] - s;                                         /* u */
        }
    for (int i = 0; i < dk; ++i) {
        real a = (real)alpha[cfg->gate ? i : 0];
        for (int v = 0; v < dv; ++v) S[i * dv + v] *= a;                   /* A = D S */
    }
    if (cfg->rule != 2)
        for (int v = 0; v < dv; ++v) {
            real s = 0;
            if (cfg->rule == 0)
                for (int i = 0; i < dk; ++i) s += S[i * dv + v] * (real)k[i];  /* A^T k */
            w[v] = (real)vv[v] - s;                                             /* u */
        }
    for (int i = 0; i < dk; ++i) {
        real wk = (real)beta * (real)k[i];                                  /* beta k */
        for (int v = 0; v < dv; ++v) S[i * dv + v] += wk * w[v];
    }
    for (int i = 0; i < dk * dv; ++i) S[i] = state_round(mode, S[i]);
    for (int v = 0; v < dv; ++v) {
        real s = 0;
        for (int i = 0; i < dk; ++i) s += S[i * dv + v] * (real)q[i];     /* S^T q */
        o[v] = (double)s;
    }
}

void OQ(recurrent_step)(const lqo_cfg *cfg, double *S, const float *q, const float *k,
                        const float *b, const float *v, const float *alpha, float beta, double *o,
                        int mode)
{
    const int n = cfg->dk * cfg->dv;
    real *Sr = (real *)malloc(sizeof(real) * (size_t)n);
    real *w = (real *)malloc(sizeof(real) * (size_t)cfg->dv);
    for (int i = 0; i < n; ++i) Sr[i] = (real)S[i];
    recurrent_step_impl(cfg, Sr, q, k, b, v, alpha, beta, o, mode, w);
    for (int i = 0; i < n; ++i) S[i] = (double)Sr[i];
    free(Sr);
    free(w);
}

/* ------------------------------------------------------------------------ */
/* O3: one token inside a window, dense form.                                */
/* The buffered record (alpha_i, beta_i k_i, u_i) is rounded to FP16 first   */
/* and the rounded values drive this token's output and every later use.     */
/* ------------------------------------------------------------------------ */

static void window_step_impl(const lqo_cfg *cfg, real *S, const float *q, const float *k,
                             const float *b, const float *vv, const float *alpha, float beta,
                             double *o, double *ra, double *rk, double *ru, real *u)
{
    const int dk = cfg->dk, dv = cfg->dv, g = cfg->gate ? dk : 1;
    for (int i = 0; i < g; ++i) ra[i] = (double)rec_round(cfg, (real)alpha[i]);
    if (cfg->rule == 2)
        for (int v = 0; v < dv; ++v) {
            real s = 0;
            for (int i = 0; i < dk; ++i) s += S[i * dv + v] * (real)b[i];
            u[v] = rec_round(cfg, (real)vv[v] - s);                         /* u_i = v_i - S_{i-1}^T b_i */
            ru[v] = (double)u[v];
        }
    for (int i = 0; i < dk; ++i) {
        real a = (real)ra[cfg->gate ? i : 0];
        for (int v = 0; v < dv; ++v) S[i * dv + v] *= a;                   /* A_i = D_i S_{i-1} */
    }
    if (cfg->rule != 2)
        for (int v = 0; v < dv; ++v) {
            real s = 0;
            if (cfg->rule == 0)
                for (int i = 0; i < dk; ++i) s += S[i * dv + v] * (real)k[i];
            u[v] = rec_round(cfg, (real)vv[v] - s);                         /* u_i = v_i - A_i^T k_i */
            ru[v] = (double)u[v];
        }
    for (int i = 0; i < dk; ++i) {
        /* beta*k as an fp32 product, the precision of the inputs */
        real tk = cfg->round_records ? f16v((real)(beta * k[i])) : (real)beta * (real)k[i];
        rk[i] = (double)tk;
        for (int v = 0; v < dv; ++v) S[i * dv + v] += tk * u[v];           /* S_i = A_i + k~_i u_i^T */
    }
    for (int v = 0; v < dv; ++v) {
        real s = 0;
        for (int i = 0; i < dk; ++i) s += S[i * dv + v] * (real)q[i];
        o[v] = (double)s;                                                   /* o_i = S_i^T q_i */
    }
}

void OQ(window_step)(const lqo_cfg *cfg, double *S, const float *q, const float *k,
                     const float *b, const float *v, const float *alpha, float beta, double *o,
                     double *ra, double *rk, double *ru)
{
    const int n = cfg->dk * cfg->dv;
    real *Sr = (real *)malloc(sizeof(real) * (size_t)n);
    real *u = (real *)malloc(sizeof(real) * (size_t)cfg->dv);
    for (int i = 0; i < n; ++i) Sr[i] = (real)S[i];
    window_step_impl(cfg, Sr, q, k, b, v, alpha, beta, o, ra, rk, ru, u);
    for (int i = 0; i < n; ++i) S[i] = (double)Sr[i];
    free(Sr);
    free(u);
}

/* ------------------------------------------------------------------------ */
/* O4: readout form.                                                         */
/* ------------------------------------------------------------------------ */

/* Gamma_{a:b}[ch] = prod_{m=a..b} alpha_m[ch] over 1-based token positions of
 * the window, I when a > b.  alpha_m for m <= n_rec comes from the records,
 * alpha_{n_rec+1} is `cur` (may be NULL when only n_rec records exist). */
static real gamma_range(const lqo_cfg *cfg, const double *rec_a, int n_rec, const double *cur,
                        int a, int b, int ch)
{
    const int g = cfg->gate ? cfg->dk : 1, idx = cfg->gate ? ch : 0;
    real p = 1;
    for (int m = a; m <= b; ++m) {
        const double *am = (m <= n_rec) ? rec_a + (size_t)(m - 1) * g : cur;
        p *= (real)am[idx];
    }
    return p;
}

/* S_ell^T x for the window state after `ell` tokens whose decays are known:
 * the base (quantized residual with smoothing, or a dense S0 when Z is NULL),
 * the Compensator Tokens, and records 1..n_use.  Eq. (smooth-readout). */
static void readout_impl(const lqo_cfg *cfg, const uint8_t *Z, const float *delta,
                         const float *c, const double *Kt, const double *Ut, const double *S0,
                         const double *rec_a, const double *rec_k, const double *rec_u,
                         int n_rec, const double *cur_a, int ell, int n_use, const float *x,
                         real *out, real *y, real *xg)
{
    const int dk = cfg->dk, dv = cfg->dv;
    for (int i = 0; i < dk; ++i) y[i] = gamma_range(cfg, rec_a, n_rec, cur_a, 1, ell, i) * (real)x[i];
    for (int v = 0; v < dv; ++v) {
        real s = 0;
        if (Z) {
            for (int i = 0; i < dk; ++i) s += code_value(cfg, Z, (size_t)i * dv + v) * (real)c[i] * y[i];
            s *= (real)delta[v];
        } else {
            for (int i = 0; i < dk; ++i) s += (real)S0[i * dv + v] * y[i];
        }
        out[v] = s;
    }
    for (int h = 0; h < cfg->n_comp; ++h) {
        real s = 0;
        for (int i = 0; i < dk; ++i) s += (real)Kt[(size_t)h * dk + i] * y[i];
        for (int v = 0; v < dv; ++v) out[v] += (real)Ut[(size_t)h * dv + v] * s;
    }
    for (int j = 1; j <= n_use; ++j) {
        for (int i = 0; i < dk; ++i)
            xg[i] = gamma_range(cfg, rec_a, n_rec, cur_a, j + 1, ell, i) * (real)x[i];
        real s = 0;
        for (int i = 0; i < dk; ++i) s += (real)rec_k[(size_t)(j - 1) * dk + i] * xg[i];
        for (int v = 0; v < dv; ++v) out[v] += (real)rec_u[(size_t)(j - 1) * dv + v] * s;
    }
}

void OQ(readout_step)(const lqo_cfg *cfg, const uint8_t *Z, const float *delta, const float *c,
                      const double *Kt, const double *Ut, const double *S0, const double *rec_a,
                      const double *rec_k, const double *rec_u, int n_rec, const float *q,
                      const float *k, const float *b, const float *vv, const float *alpha,
                      float beta, double *o, double *na, double *nk, double *nu)
{
    const int dk = cfg->dk, dv = cfg->dv, g = cfg->gate ? dk : 1;
    real *Ak = (real *)malloc(sizeof(real) * (size_t)dv);
    real *Aq = (real *)malloc(sizeof(real) * (size_t)dv);
    real *y = (real *)malloc(sizeof(real) * (size_t)dk);
    real *xg = (real *)malloc(sizeof(real) * (size_t)dk);
    for (int i = 0; i < g; ++i) na[i] = (double)rec_round(cfg, (real)alpha[i]);
    const int ell = n_rec + 1;
    /* A_i^T x = S_{i-1}^T (Gamma_{i:i} x): the base and all records decay
     * through token i, none of the records includes token i itself.  The
     * general rule reads S_{i-1}^T b instead: the same sum with the decays of
     * the records only (ell = n_rec). */
    if (cfg->rule == 2)
        readout_impl(cfg, Z, delta, c, Kt, Ut, S0, rec_a, rec_k, rec_u, n_rec, na, n_rec, n_rec, b, Ak, y, xg);
    else
        readout_impl(cfg, Z, delta, c, Kt, Ut, S0, rec_a, rec_k, rec_u, n_rec, na, ell, n_rec, k, Ak, y, xg);
    readout_impl(cfg, Z, delta, c, Kt, Ut, S0, rec_a, rec_k, rec_u, n_rec, na, ell, n_rec, q, Aq, y, xg);
    real kq = 0;
    for (int i = 0; i < dk; ++i) {
        real tk = cfg->round_records ? f16v((real)(beta * k[i])) : (real)beta * (real)k[i];
        nk[i] = (double)tk;
        kq += tk * (real)q[i];
    }
    for (int v = 0; v < dv; ++v) {
        real u = rec_round(cfg, (real)vv[v] - (cfg->rule == 1 ? (real)0 : Ak[v]));
        nu[v] = (double)u;
        o[v] = (double)(Aq[v] + u * kq);                                     /* S_i^T q */
    }
    free(Ak);
    free(Aq);
    free(y);
    free(xg);
}

/* Window-end reconstruction, Sec. 3.4 Eq. (smooth):
 * S_p = Gamma_{1:p} [C dequant(Z) + K~ U~^T] + sum_j Gamma_{j+1:p} k~_j u_j^T. */
void OQ(reconstruct)(const lqo_cfg *cfg, const uint8_t *Z, const float *delta, const float *c,
                     const double *Kt, const double *Ut, const double *S0, const double *rec_a,
                     const double *rec_k, const double *rec_u, int n_rec, double *S_out)
{
    const int dk = cfg->dk, dv = cfg->dv;
    for (int i = 0; i < dk; ++i) {
        real G = gamma_range(cfg, rec_a, n_rec, NULL, 1, n_rec, i);
        for (int v = 0; v < dv; ++v) {
            real base;
            if (Z) {
                base = (real)c[i] * (code_value(cfg, Z, (size_t)i * dv + v) * (real)delta[v]);
                for (int h = 0; h < cfg->n_comp; ++h)
                    base += (real)Kt[(size_t)h * dk + i] * (real)Ut[(size_t)h * dv + v];
            } else {
                base = (real)S0[i * dv + v];
            }
            real s = G * base;
            for (int j = 1; j <= n_rec; ++j)
                s += gamma_range(cfg, rec_a, n_rec, NULL, j + 1, n_rec, i) *
                     (real)rec_k[(size_t)(j - 1) * dk + i] * (real)rec_u[(size_t)(j - 1) * dv + v];
            S_out[i * dv + v] = (double)s;
        }
    }
}

/* ------------------------------------------------------------------------ */
/* Trajectory drivers over independent tiles.                                */
/* ------------------------------------------------------------------------ */

typedef struct {
    uint8_t *Z;        /* [tiles][n_snap][dk][dv] x code bytes (may be NULL) */
    float *delta;      /* [tiles][n_snap][dv] */
    float *c;          /* [tiles][n_snap][dk] */
    double *Kt;        /* [tiles][n_snap][r][dk] */
    double *Ut;        /* [tiles][n_snap][r][dv] */
    double *S_final;   /* [tiles][dk][dv] dense state after the last token (may be NULL) */
    double *rec_a;     /* [tiles][W][g] records of the open window (may be NULL) */
    double *rec_k;     /* [tiles][W][dk] */
    double *rec_u;     /* [tiles][W][dv] */
    int32_t *rec_len;  /* [tiles] */
    double *hist_a;    /* [tiles][T][g] every token's record (may be NULL) */
    double *hist_k;    /* [tiles][T][dk] */
    double *hist_u;    /* [tiles][T][dv] */
} lqo_outputs;

static void store_hist(const lqo_cfg *cfg, const lqo_outputs *out, size_t ts, const double *ra,
                       const double *rk, const double *ru)
{
    if (!out->hist_a) return;
    const int dk = cfg->dk, dv = cfg->dv, g = cfg->gate ? dk : 1;
    memcpy(out->hist_a + ts * g, ra, sizeof(double) * g);
    memcpy(out->hist_k + ts * dk, rk, sizeof(double) * dk);
    memcpy(out->hist_u + ts * dv, ru, sizeof(double) * dv);
}

typedef struct {
    const float *q;     /* [tiles][T][dk] */
    const float *k;     /* [tiles][T][dk] */
    const float *v;     /* [tiles][T][dv] */
    const float *alpha; /* [tiles][T][g] */
    const float *beta;  /* [tiles][T] */
    const float *b;     /* [tiles][T][dk] read vectors (rule 2 only; may be NULL otherwise) */
} lqo_inputs;

static const float *read_vec(const lqo_inputs *in, size_t ts, int dk)
{
    return in->b ? in->b + ts * dk : NULL;
}

static int n_snap_of(const lqo_cfg *cfg, int T) { return 1 + T / cfg->window; }

static void store_snap(const lqo_cfg *cfg, const lqo_outputs *out, int tile, int T, int s,
                       const uint8_t *Z, const float *delta, const float *c, const double *Kt,
                       const double *Ut)
{
    if (!out->Z) return;
    const int dk = cfg->dk, dv = cfg->dv, r = cfg->n_comp;
    const size_t idx = (size_t)tile * n_snap_of(cfg, T) + s;
    memcpy(out->Z + idx * dk * dv * code_bytes(cfg), Z, (size_t)dk * dv * code_bytes(cfg));
    memcpy(out->delta + idx * dv, delta, sizeof(float) * dv);
    memcpy(out->c + idx * dk, c, sizeof(float) * dk);
    if (r) {
        memcpy(out->Kt + idx * r * dk, Kt, sizeof(double) * r * dk);
        memcpy(out->Ut + idx * r * dv, Ut, sizeof(double) * r * dv);
    }
}

/*
 * Per-window method, dense form (O3), for `tiles` independent tiles and T
 * tokens.  Window start: the given fp32 state is quantized (O2).  After every
 * W tokens the dense state is re-quantized and dequantized.  With
 * cfg->quantize == 0 nothing is ever quantized (self-check mode).
 */
int OQ(run_dense)(const lqo_cfg *cfg, int tiles, int T, const double *S_init,
                  const lqo_inputs *in, double *o, const lqo_outputs *out, int n_threads)
{
    const int dk = cfg->dk, dv = cfg->dv, g = cfg->gate ? dk : 1, r = cfg->n_comp, W = cfg->window;
#pragma omp parallel for schedule(dynamic, 1) num_threads(n_threads > 0 ? n_threads : 1)
    for (int t = 0; t < tiles; ++t) {
        real *S = (real *)malloc(sizeof(real) * (size_t)dk * dv);
        double *Sd = (double *)malloc(sizeof(double) * (size_t)dk * dv);
        real *u = (real *)malloc(sizeof(real) * (size_t)dv);
        uint8_t *Z = (uint8_t *)calloc((size_t)dk * dv, code_bytes(cfg));
        float *delta = (float *)calloc((size_t)dv, sizeof(float));
        float *c = (float *)calloc((size_t)dk, sizeof(float));
        double *Kt = (double *)calloc((size_t)(r ? r : 1) * dk, sizeof(double));
        double *Ut = (double *)calloc((size_t)(r ? r : 1) * dv, sizeof(double));
        double *ra = (double *)calloc((size_t)W * g, sizeof(double));
        double *rk = (double *)calloc((size_t)W * dk, sizeof(double));
        double *ru = (double *)calloc((size_t)W * dv, sizeof(double));
        const double *S0 = S_init + (size_t)t * dk * dv;
        int snap = 0;
        if (cfg->quantize) {
            quantize_impl(cfg, S0, Z, delta, c, Kt, Ut);
            store_snap(cfg, out, t, T, snap++, Z, delta, c, Kt, Ut);
            OQ(dequantize)(cfg, Z, delta, c, Kt, Ut, Sd);
            for (int i = 0; i < dk * dv; ++i) S[i] = (real)Sd[i];
        } else {
            for (int i = 0; i < dk * dv; ++i) S[i] = (real)S0[i];
        }
        int n = 0;
        for (int s = 0; s < T; ++s) {
            const size_t ts = (size_t)t * T + s;
            window_step_impl(cfg, S, in->q + ts * dk, in->k + ts * dk, read_vec(in, ts, dk),
                             in->v + ts * dv, in->alpha + ts * g, in->beta[ts], o + ts * dv, ra + (size_t)n * g,
                             rk + (size_t)n * dk, ru + (size_t)n * dv, u);
            store_hist(cfg, out, ts, ra + (size_t)n * g, rk + (size_t)n * dk, ru + (size_t)n * dv);
            if (++n == W) {
                if (cfg->quantize) {
                    for (int i = 0; i < dk * dv; ++i) Sd[i] = (double)S[i];
                    quantize_impl(cfg, Sd, Z, delta, c, Kt, Ut);
                    store_snap(cfg, out, t, T, snap++, Z, delta, c, Kt, Ut);
                    OQ(dequantize)(cfg, Z, delta, c, Kt, Ut, Sd);
                    for (int i = 0; i < dk * dv; ++i) S[i] = (real)Sd[i];
                }
                n = 0;
            }
        }
        if (out->S_final)
            for (int i = 0; i < dk * dv; ++i) out->S_final[(size_t)t * dk * dv + i] = (double)S[i];
        if (out->rec_len) {
            out->rec_len[t] = n;
            memcpy(out->rec_a + (size_t)t * W * g, ra, sizeof(double) * (size_t)W * g);
            memcpy(out->rec_k + (size_t)t * W * dk, rk, sizeof(double) * (size_t)W * dk);
            memcpy(out->rec_u + (size_t)t * W * dv, ru, sizeof(double) * (size_t)W * dv);
        }
        free(S); free(Sd); free(u); free(Z); free(delta); free(c);
        free(Kt); free(Ut); free(ra); free(rk); free(ru);
    }
    return 0;
}

/*
 * Per-window method, readout form (O4): the window base is held fixed
 * (quantized, or dense when cfg->quantize == 0), every output is read through
 * Eq. (smooth-readout), and at each window end the state is reconstructed with
 * Eq. (smooth) before being quantized again.  Same interface as run_dense.
 */
int OQ(run_readout)(const lqo_cfg *cfg, int tiles, int T, const double *S_init,
                    const lqo_inputs *in, double *o, const lqo_outputs *out, int n_threads)
{
    const int dk = cfg->dk, dv = cfg->dv, g = cfg->gate ? dk : 1, r = cfg->n_comp, W = cfg->window;
#pragma omp parallel for schedule(dynamic, 1) num_threads(n_threads > 0 ? n_threads : 1)
    for (int t = 0; t < tiles; ++t) {
        double *Sd = (double *)malloc(sizeof(double) * (size_t)dk * dv);
        uint8_t *Z = (uint8_t *)calloc((size_t)dk * dv, code_bytes(cfg));
        float *delta = (float *)calloc((size_t)dv, sizeof(float));
        float *c = (float *)calloc((size_t)dk, sizeof(float));
        double *Kt = (double *)calloc((size_t)(r ? r : 1) * dk, sizeof(double));
        double *Ut = (double *)calloc((size_t)(r ? r : 1) * dv, sizeof(double));
        double *ra = (double *)calloc((size_t)W * g, sizeof(double));
        double *rk = (double *)calloc((size_t)W * dk, sizeof(double));
        double *ru = (double *)calloc((size_t)W * dv, sizeof(double));
        const double *S0 = S_init + (size_t)t * dk * dv;
        int snap = 0;
        if (cfg->quantize) {
            quantize_impl(cfg, S0, Z, delta, c, Kt, Ut);
            store_snap(cfg, out, t, T, snap++, Z, delta, c, Kt, Ut);
        } else {
            memcpy(Sd, S0, sizeof(double) * (size_t)dk * dv);
        }
        int n = 0;
        for (int s = 0; s < T; ++s) {
            const size_t ts = (size_t)t * T + s;
            OQ(readout_step)(cfg, cfg->quantize ? Z : NULL, delta, c, Kt, Ut, Sd, ra, rk, ru, n,
                             in->q + ts * dk, in->k + ts * dk, read_vec(in, ts, dk), in->v + ts * dv,
                             in->alpha + ts * g, in->beta[ts], o + ts * dv, ra + (size_t)n * g, rk + (size_t)n * dk,
                             ru + (size_t)n * dv);
            store_hist(cfg, out, ts, ra + (size_t)n * g, rk + (size_t)n * dk, ru + (size_t)n * dv);
            if (++n == W) {
                OQ(reconstruct)(cfg, cfg->quantize ? Z : NULL, delta, c, Kt, Ut, Sd, ra, rk, ru, n, Sd);
                if (cfg->quantize) {
                    quantize_impl(cfg, Sd, Z, delta, c, Kt, Ut);
                    store_snap(cfg, out, t, T, snap++, Z, delta, c, Kt, Ut);
                }
                n = 0;
            }
        }
        if (out->S_final) {
            double *Sf = out->S_final + (size_t)t * dk * dv;
            OQ(reconstruct)(cfg, cfg->quantize ? Z : NULL, delta, c, Kt, Ut, Sd, ra, rk, ru, n, Sf);
        }
        if (out->rec_len) {
            out->rec_len[t] = n;
            memcpy(out->rec_a + (size_t)t * W * g, ra, sizeof(double) * (size_t)W * g);
            memcpy(out->rec_k + (size_t)t * W * dk, rk, sizeof(double) * (size_t)W * dk);
            memcpy(out->rec_u + (size_t)t * W * dv, ru, sizeof(double) * (size_t)W * dv);
        }
        free(Sd); free(Z); free(delta); free(c); free(Kt); free(Ut);
        free(ra); free(rk); free(ru);
    }
    return 0;
}

/* Baselines (O5) and the unquantized reference trajectory (O1): the state is
 * rounded to fp32 / bf16 after each token, or kept exact (mode 0). */
int OQ(run_baseline)(const lqo_cfg *cfg, int tiles, int T, const double *S_init,
                     const lqo_inputs *in, double *o, double *S_final, int mode, int n_threads)
{
    const int dk = cfg->dk, dv = cfg->dv, g = cfg->gate ? dk : 1;
#pragma omp parallel for schedule(dynamic, 1) num_threads(n_threads > 0 ? n_threads : 1)
    for (int t = 0; t < tiles; ++t) {
        real *S = (real *)malloc(sizeof(real) * (size_t)dk * dv);
        real *w = (real *)malloc(sizeof(real) * (size_t)dv);
        double *od = (double *)malloc(sizeof(double) * (size_t)dv);
        for (int i = 0; i < dk * dv; ++i) S[i] = state_round(mode, (real)S_init[(size_t)t * dk * dv + i]);
        for (int s = 0; s < T; ++s) {
            const size_t ts = (size_t)t * T + s;
            recurrent_step_impl(cfg, S, in->q + ts * dk, in->k + ts * dk, read_vec(in, ts, dk),
                                in->v + ts * dv, in->alpha + ts * g, in->beta[ts], o ? o + ts * dv : od,
                                mode, w);
        }
        if (S_final)
            for (int i = 0; i < dk * dv; ++i) S_final[(size_t)t * dk * dv + i] = (double)S[i];
        free(S);
        free(w);
        free(od);
    }
    return 0;
}

/*
 * Drift of the per-window quantized trajectory (O3) from the unquantized fp32
 * trajectory (O5, fp32 state) driven by the same tokens (App. B.1): every
 * `every` tokens, ||S_window - S_fp32||_F / ||S_fp32||_F and the relative L2
 * error of that token's output.  drift and odrift are [tiles][T/every].  With
 * cfg->quantize == 0 the window path starts from the fp32 state and is never
 * quantized (then, in the fp32 build with exact records, both trajectories take
 * the same operations).
 */
int OQ(run_drift)(const lqo_cfg *cfg, int tiles, int T, int every, const double *S_init,
                  const lqo_inputs *in, double *drift, double *odrift, int n_threads)
{
    const int dk = cfg->dk, dv = cfg->dv, g = cfg->gate ? dk : 1, r = cfg->n_comp, W = cfg->window;
    const int nd = T / every;
#pragma omp parallel for schedule(dynamic, 1) num_threads(n_threads > 0 ? n_threads : 1)
    for (int t = 0; t < tiles; ++t) {
        real *S = (real *)malloc(sizeof(real) * (size_t)dk * dv);
        real *F = (real *)malloc(sizeof(real) * (size_t)dk * dv);
        double *Sd = (double *)malloc(sizeof(double) * (size_t)dk * dv);
        real *u = (real *)malloc(sizeof(real) * (size_t)dv);
        double *o1 = (double *)malloc(sizeof(double) * (size_t)dv);
        double *o2 = (double *)malloc(sizeof(double) * (size_t)dv);
        uint8_t *Z = (uint8_t *)calloc((size_t)dk * dv, code_bytes(cfg));
        float *delta = (float *)calloc((size_t)dv, sizeof(float));
        float *c = (float *)calloc((size_t)dk, sizeof(float));
        double *Kt = (double *)calloc((size_t)(r ? r : 1) * dk, sizeof(double));
        double *Ut = (double *)calloc((size_t)(r ? r : 1) * dv, sizeof(double));
        double *ra = (double *)calloc((size_t)g, sizeof(double));
        double *rk = (double *)calloc((size_t)dk, sizeof(double));
        double *ru = (double *)calloc((size_t)dv, sizeof(double));
        const double *S0 = S_init + (size_t)t * dk * dv;
        for (int i = 0; i < dk * dv; ++i) F[i] = (real)(float)S0[i];
        if (cfg->quantize) {
            quantize_impl(cfg, S0, Z, delta, c, Kt, Ut);
            OQ(dequantize)(cfg, Z, delta, c, Kt, Ut, Sd);
            for (int i = 0; i < dk * dv; ++i) S[i] = (real)Sd[i];
        } else {
            for (int i = 0; i < dk * dv; ++i) S[i] = (real)(float)S0[i];
        }
        int n = 0;
        for (int s = 0; s < T; ++s) {
            const size_t ts = (size_t)t * T + s;
            window_step_impl(cfg, S, in->q + ts * dk, in->k + ts * dk, read_vec(in, ts, dk),
                             in->v + ts * dv, in->alpha + ts * g, in->beta[ts], o1, ra, rk, ru, u);
            recurrent_step_impl(cfg, F, in->q + ts * dk, in->k + ts * dk, read_vec(in, ts, dk),
                                in->v + ts * dv, in->alpha + ts * g, in->beta[ts], o2, LQO_STATE_F32, u);
            if (++n == W) {
                if (cfg->quantize) {
                    for (int i = 0; i < dk * dv; ++i) Sd[i] = (double)S[i];
                    quantize_impl(cfg, Sd, Z, delta, c, Kt, Ut);
                    OQ(dequantize)(cfg, Z, delta, c, Kt, Ut, Sd);
                    for (int i = 0; i < dk * dv; ++i) S[i] = (real)Sd[i];
                }
                n = 0;
            }
            if ((s + 1) % every == 0 && (s + 1) / every <= nd) {
                double num = 0, den = 0, on = 0, od = 0;
                for (int i = 0; i < dk * dv; ++i) {
                    double d = (double)S[i] - (double)F[i];
                    num += d * d;
                    den += (double)F[i] * (double)F[i];
                }
                for (int v = 0; v < dv; ++v) {
                    double d = o1[v] - o2[v];
                    on += d * d;
                    od += o2[v] * o2[v];
                }
                drift[(size_t)t * nd + (s + 1) / every - 1] = den > 0 ? sqrt(num / den) : sqrt(num);
                odrift[(size_t)t * nd + (s + 1) / every - 1] = od > 0 ? sqrt(on / od) : sqrt(on);
            }
        }
        free(S); free(F); free(Sd); free(u); free(o1); free(o2); free(Z); free(delta); free(c);
        free(Kt); free(Ut); free(ra); free(rk); free(ru);
    }
    return 0;
}
