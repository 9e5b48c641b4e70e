/*
 * leapquant.h -- C ABI of the LeapQuant 8-bit recurrent-state decode path for
 * AMD Instinct MI355X (gfx950).
 *
 * LeapQuant (arXiv 2609.38166) keeps the recurrent state of a gated delta-rule
 * linear-attention head (GDN: scalar decay, KDA: per-key-channel decay) in 8
 * bits.  Within a window of W tokens the quantized state is held fixed and the
 * tokens' rank-one updates are buffered in FP16 (Sec. 3.2); outputs are read
 * from the fixed state plus the buffer (App. B.2-B.3).  At the window end the
 * state is reconstructed, its largest structure is refitted as r FP16
 * "Compensator Tokens" (Sec. 3.3), the rest is smoothed across key channels
 * (Sec. 3.4) and re-quantized per value channel (App. B.3).
 *
 * Conventions shared by every call
 * --------------------------------
 *  - One tile = one (request b, value head h) pair; tiles are numbered
 *    b * heads_v + h.  d_k = d_v = 128 in this version.
 *  - Every array argument is a caller-owned DEVICE pointer, dense, row-major,
 *    16-byte aligned, except the arrays read one element at a time: the
 *    per-tile scalars beta and (scalar gate) alpha, rec_len, err and the
 *    commit mask need 4-byte alignment, the scalar gate's rec_a 2-byte
 *    alignment.  So one step of a step-major token buffer, or a state whose
 *    arrays all start at the same tile of a larger one (a group of requests),
 *    can be passed for any tile count.
 *  - The library allocates no memory, keeps no device state and never
 *    synchronises (except leapquant_check_error).  Its only mutable state is
 *    a per-thread buffer with the text of the last HIP error it saw
 *    (leapquant_last_hip_error).  Work is enqueued on
 *    `stream` (a hipStream_t; NULL = the default stream) and returns at once.
 *    Calls on different streams with disjoint buffers may run concurrently
 *    (request groups of one state share only its error word, which the
 *    kernels update atomically).
 *  - The state of one tile is stored TRANSPOSED (value-major): row v holds the
 *    d_k key-channel entries of value channel v, S^T[v][k].
 *  - Status codes: LQ_OK (0) or a negative LQ_E* value.  Arguments are
 *    validated on the host before anything is enqueued; a failed validation
 *    enqueues nothing.  Data values are not checked: non-finite inputs give
 *    unspecified (but memory-safe) results.
 *  - Misuse only the device can see (a decode step on a tile whose window
 *    buffer is already full) sets a bit in the sticky word *err, writes NaN to
 *    that tile's output and leaves the tile's state untouched;
 *    leapquant_check_error() reports and clears it.
 */
#ifndef LEAPQUANT_H
#define LEAPQUANT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ---- */
#define LQ_OK            0
#define LQ_EINVAL       -1   /* NULL pointer, non-positive size, inconsistent heads   */
#define LQ_EALIGN       -2   /* a pointer is not aligned as its array requires     */
#define LQ_EUNSUPPORTED -3   /* d_k/d_v != 128, r > 16, W out of range, ...           */
#define LQ_EHIP         -4   /* a HIP call failed (kernel launch, synchronisation)    */
#define LQ_EDEVICE      -5   /* a sticky device error was found by check_error        */

/* ---- enumerations ---- */
#define LQ_GATE_SCALAR 0     /* GDN: D_t = alpha_t I                 (App. A table)   */
#define LQ_GATE_DIAG   1     /* KDA: D_t = Diag(alpha_t), alpha_t in R^{d_k}          */
#define LQ_CODE_INT8   0     /* symmetric INT8, dequant = code * delta_v, |code|<=127 */
#define LQ_CODE_E4M3   1     /* OCP FP8 E4M3FN codes, dequant = e4m3(code) * delta_v  */
#define LQ_CODE_INT4   2     /* symmetric 4-bit, |code| <= 7, two codes per byte      */
#define LQ_CODE_INT6   3     /* symmetric 6-bit, |code| <= 31, four codes per 3 bytes  */
#define LQ_CODE_BF16   4     /* the state itself in BF16 (per-window BF16, Sec. 3.2):
                              * rounded to nearest even at each window end; unit
                              * scales, no smoothing, n_comp must be 0            */
#define LQ_RULE_DELTA  0     /* delta rule: b_t = D_t k_t (DeltaNet, GDN, KDA)        */
#define LQ_RULE_ADD    1     /* b_t = 0: u_t = v_t (linear attention, RetNet, Mamba2,
                              * GLA / RWKV6 / HGRN2 with the matching gate)           */
#define LQ_RULE_GENERAL 2    /* b_t given with every token (App. A general form): the
                              * erase sub-step of RWKV7; only the *_general calls    */
#define LQ_STATE_F32   0     /* baseline state in fp32                               */
#define LQ_STATE_BF16  1     /* baseline state in bf16, rounded to nearest even      */

/* bits of the sticky device error word */
#define LQ_DEVERR_WINDOW_FULL 1   /* decode_step on a tile with rec_len == window      */
#define LQ_DEVERR_BAD_REC_LEN 2   /* a tile's rec_len is outside [0, window]; untouched */

/* Limits of this version. */
#define LQ_MAX_COMP        16
#define LQ_MAX_WINDOW_GDN 256
#define LQ_MAX_WINDOW_KDA 256
#define LQ_MAX_POWER_ITERS 64
/* Also: batch * heads_v <= 2^30 and batch * heads_v * (heads_v / heads_k) < 2^32
 * (LQ_EUNSUPPORTED otherwise). */

/* Shape and method parameters (host struct, read at each call). */
typedef struct {
    int32_t batch;       /* B, requests                                              */
    int32_t heads_v;     /* value heads per request; tiles = batch * heads_v         */
    int32_t heads_k;     /* key heads; value head h reads key head h / (heads_v/heads_k) */
    int32_t d_k, d_v;    /* head dimensions (128, 128)                               */
    int32_t window;      /* W >= 1: tokens buffered before the state is re-quantized */
    int32_t n_comp;      /* r in [0, 16]: Compensator Tokens per tile                */
    int32_t power_iters; /* power-iteration sweeps per token, >= 1 when r > 0        */
    int32_t gate;        /* LQ_GATE_SCALAR or LQ_GATE_DIAG                            */
    int32_t code;        /* LQ_CODE_INT8, LQ_CODE_E4M3, LQ_CODE_INT4, LQ_CODE_INT6 or
                          * LQ_CODE_BF16                                          */
    int32_t smooth;      /* 1: residual smoothing (Sec. 3.4); 0: c = 1               */
    int32_t rule;        /* LQ_RULE_DELTA, LQ_RULE_ADD or LQ_RULE_GENERAL: the read
                          * vector b_t of the general recurrence (App. A table).
                          * Only the decode and baseline steps read it; the state
                          * layout does not depend on it, so one state may be
                          * stepped under different rules (see the general step) */
} lq_dims;

/* The quantized state of all tiles (device pointers, caller-owned).
 * Sizes per tile; g = 1 for the scalar gate, g = d_k for the diagonal gate. */
typedef struct {
    void     *codes;   /* [d_v][d_k*b/8] bytes, b = 8, 8, 4, 6, 16 bits per code:
                        *   INT8: one two's-complement byte per key channel;
                        *   E4M3: one E4M3FN byte per key channel;
                        *   INT4: byte i holds channel 2i (low nibble) and 2i+1
                        *         (high nibble), two's complement;
                        *   INT6: bytes 3i..3i+2, read little-endian as 24 bits,
                        *         hold channels 4i..4i+3 at bits 6q..6q+5;
                        *   BF16: the state value of each key channel in BF16
                        *         (scale and smooth are then written as 1 by
                        *         quantize and commit and never read)       */
    float    *scale;   /* [d_v]  delta_v = max_k |R^C_kv| / 127 (INT8) or / 448    */
    float    *smooth;  /* [d_k]  c_k, the residual smoothing scale                 */
    uint16_t *comp_k;  /* [r][d_k] fp16 key vectors k~_h of the Compensator Tokens */
    uint16_t *comp_u;  /* [r][d_v] fp16 value vectors u~_h                          */
    uint16_t *rec_k;   /* [W][d_k] fp16 buffered write keys  k~_j = beta_j k_j      */
    uint16_t *rec_u;   /* [W][d_v] fp16 buffered corrections u_j                    */
    uint16_t *rec_a;   /* [W][g]   fp16 buffered decays alpha_j                     */
    int32_t  *rec_len; /* [1] per tile: records in the open window (0..W)           */
    int32_t  *err;     /* [1] sticky device error word (LQ_DEVERR_* bits); required */
} lq_state;

/*
 * leapquant_state_bytes -- host only, no device access.
 * Byte sizes of the ten lq_state buffers for all tiles, in field order
 * (codes, scale, smooth, comp_k, comp_u, rec_k, rec_u, rec_a, rec_len, err).
 * With r = 4, d = 128 the window-boundary representation (codes, scale,
 * smooth, comp_k, comp_u) is 1.1875 bytes per state element (Sec. 4.3,
 * "Memory reduction").
 */
int32_t leapquant_state_bytes(const lq_dims *dims, size_t bytes_out[10]);

/*
 * leapquant_quantize_state -- quantize given fp32 states (a prefill result or a
 * prefix-cache snapshot) into the window-start representation and open an
 * empty window.  Sec. 3.3 Eq. (compensator-rank-r), Sec. 3.4, App. B.3.
 *   S   [B][heads_v][d_v][d_k] fp32, S^T of every tile; read only.
 *   st  codes, scale, smooth, comp_k, comp_u written; rec_len set to 0.
 * The r tokens are fitted one after another by power iteration on the
 * deflated residual, starting each from the residual's key-row l2 norms; each
 * token is rounded to FP16 before it is subtracted, so the codes absorb that
 * rounding.  c_k = sqrt(max(mean_v |R_kv|, 1e-12)), R^C = R * (1/c_k),
 * delta_v = max_k |R^C_kv| / 127, code = clamp(rint(R^C * 127/max), +-127).
 * The 6- and 4-bit variants (the paper's lower-bit LeapQuant, Sec. 4.1-4.2)
 * use the same rule with qmax = 31 and 7 (2^(b-1) - 1) and packed storage.
 * LQ_CODE_BF16 (per-window BF16, Sec. 3.2) stores every entry rounded to
 * BF16 (nearest even) with unit scales and smoothing and no tokens.
 * The fit, the deflation and the smoothing statistic are carried in fp64;
 * the FP16 rounding of the tokens and the codes are decided in fp32.
 */
int32_t leapquant_quantize_state(const lq_dims *dims, const float *S, lq_state *st, void *stream);

/*
 * leapquant_decode_step -- one token for every tile.  Sec. 3.2 Eq. (record),
 * App. B.2 Eq. (readout), App. B.3 Eq. (smooth-readout).
 *   q, k   [B][heads_k][d_k] fp32      v [B][heads_v][d_v] fp32
 *   alpha  [B][heads_v] (scalar gate) or [B][heads_v][d_k] (diagonal gate) fp32
 *   beta   [B][heads_v] fp32           o [B][heads_v][d_v] fp32 (written)
 * With i = rec_len + 1 and the token's decay rounded to FP16:
 *   A^T x = delta . (Z^T (c . Gamma_{1:i} x)) + U~ (K~^T Gamma_{1:i} x)
 *           + sum_{j<i} u_j (k~_j^T Gamma_{j+1:i} x)          for x = k, q
 *   u_i = fp16(v - A^T k),  k~_i = fp16(beta k),  o = A^T q + u_i (k~_i . q)
 * and the record (alpha_i, k~_i, u_i) is appended; rec_len += 1.  Everything
 * that feeds u_i (A^T k) is evaluated at fp64 accuracy, the code product
 * exactly, so u_i is the correctly rounded FP16 value; the q side is fp32.
 * k~_i is beta k rounded to fp32 and then to FP16.  A tile whose
 * rec_len already equals W is not modified: its o is NaN and
 * LQ_DEVERR_WINDOW_FULL is raised in *err.  dims->rule LQ_RULE_GENERAL is
 * rejected (LQ_EINVAL): that rule takes its read vectors through
 * leapquant_decode_step_general.
 */
int32_t leapquant_decode_step(const lq_dims *dims, lq_state *st, const float *q, const float *k,
                              const float *v, const float *alpha, const float *beta, float *o,
                              void *stream);

/*
 * leapquant_decode_step_general -- one token for every tile under the general
 * recurrence with the read vector given (App. A, Eq. (general)):
 *   S_t = D_t S_{t-1} + (beta_t k_t) (v_t - S_{t-1}^T b_t)^T,  o_t = S_t^T q_t.
 *   b      [B][heads_v][d_k] fp32, the read vectors (one per tile);
 *          other arguments as leapquant_decode_step.
 * dims->rule must be LQ_RULE_GENERAL (LQ_EINVAL otherwise; leapquant_decode_step
 * rejects that rule).  With i = rec_len + 1 and d_i the token's FP16 decay,
 *   S_{i-1}^T b = delta . (Z^T (c . Gamma_{1:i-1} b)) + U~ (K~^T Gamma_{1:i-1} b)
 *                 + sum_{j<i} u_j (k~_j^T Gamma_{j+1:i-1} b),
 * and A^T q = S_{i-1}^T (d_i . q) by the same sum; then u_i = fp16(v - S_{i-1}^T b),
 * o = A^T q + u_i (k~_i . q) and the record is appended as in
 * leapquant_decode_step.  A model whose erase direction differs from its write
 * key runs as sub-steps (App. A): an RWKV7 token with transition
 * Diag(w) - kappa (a . kappa)^T and write k v^T is this call with alpha = w,
 * k = kappa, beta = 1, b = a . kappa, v = 0 (diagonal gate), then either this
 * call with alpha = 1, b = 0, or leapquant_decode_step on the same state with a
 * copy of dims whose rule is LQ_RULE_ADD, with k = k, beta = 1, v = v; each
 * sub-step is one record, so W counts sub-steps.
 */
int32_t leapquant_decode_step_general(const lq_dims *dims, lq_state *st, const float *q,
                                      const float *k, const float *b, const float *v,
                                      const float *alpha, const float *beta, float *o,
                                      void *stream);

/*
 * leapquant_decode_step_commit -- leapquant_decode_step, then, in the same
 * launch, the window commit of every tile whose window this token filled
 * (rec_len reached W).  Sec. 3.3 (the refit at the window end runs inside the
 * decode kernel, beside the other tiles' state reads), Sec. 4.1
 * "Implementation".  Arguments, layouts, validation and the device error rules
 * are those of leapquant_decode_step.  Every tile is decoded exactly as there;
 * a tile with rec_len == W - 1 before the call is then committed exactly as
 * leapquant_window_commit commits a full window (all W records, the new one
 * included) and leaves the call with rec_len = 0.  Requests at different window
 * positions may share one launch; only the tiles that reach W commit.  A tile
 * rejected by the decode (full or corrupt window) is not committed.
 * dims->rule must be LQ_RULE_DELTA or LQ_RULE_ADD (LQ_EINVAL otherwise).
 */
int32_t leapquant_decode_step_commit(const lq_dims *dims, lq_state *st, const float *q,
                                     const float *k, const float *v, const float *alpha,
                                     const float *beta, float *o, void *stream);

/*
 * leapquant_window_commit -- end the window of the selected tiles.  Sec. 3.3
 * (refit at the window end), Sec. 3.4 Eq. (smooth).
 *   mask  [B] int32 on the device, nonzero = commit every head of request b;
 *         NULL = commit all requests.
 * For a selected tile with p = rec_len > 0 records, reconstruct
 *   S_p = Gamma_{1:p} [C dequant(Z) + K~ U~^T] + sum_j Gamma_{j+1:p} k~_j u_j^T
 * in fp64, discard the old tokens, re-quantize S_p exactly as
 * leapquant_quantize_state does and set rec_len = 0.  A partial window
 * (p < W) is legal; tiles with rec_len == 0 or an unselected request are left
 * untouched.
 */
int32_t leapquant_window_commit(const lq_dims *dims, lq_state *st, const int32_t *mask,
                                void *stream);

/*
 * leapquant_baseline_step -- one token of the unquantized recurrence with a
 * dense state, the per-step baseline of Sec. 4.1.  Sec. 3.1 Eq. (general):
 *   A = D S,  u = v - A^T k,  S = A + (beta k) u^T,  o = S^T q,
 * state S [B][heads_v][d_v][d_k] updated in place, fp32 (LQ_STATE_F32) or
 * bf16 bits (LQ_STATE_BF16, rounded to nearest even after the step).
 * Arithmetic is fp32.  Other arguments as leapquant_decode_step (the decay is
 * not rounded); LQ_RULE_GENERAL is rejected as there.
 */
int32_t leapquant_baseline_step(const lq_dims *dims, void *S, int32_t state_dtype,
                                const float *q, const float *k, const float *v,
                                const float *alpha, const float *beta, float *o, void *stream);

/*
 * leapquant_baseline_step_general -- leapquant_baseline_step under the general
 * recurrence (App. A, Eq. (general)) with the read vectors b [B][heads_v][d_k]
 * fp32:  u = v - S^T b,  S = D S + (beta k) u^T,  o = S^T q.
 * dims->rule must be LQ_RULE_GENERAL (LQ_EINVAL otherwise).
 */
int32_t leapquant_baseline_step_general(const lq_dims *dims, void *S, int32_t state_dtype,
                                        const float *q, const float *k, const float *b,
                                        const float *v, const float *alpha, const float *beta,
                                        float *o, void *stream);

/*
 * leapquant_dequantize_state -- materialise the current fp32 state of every
 * tile, base plus the rec_len buffered records (Sec. 3.2 Eq. (window) with
 * Sec. 3.4 Eq. (smooth)), into S_out [B][heads_v][d_v][d_k] (S^T).  Read only
 * on st.  For inspection, checkpoint export and tests.
 */
int32_t leapquant_dequantize_state(const lq_dims *dims, const lq_state *st, float *S_out,
                                   void *stream);

/*
 * leapquant_check_error -- synchronise `stream`, copy the sticky word *err to
 * *bits_out (may be NULL), clear it, and return LQ_EDEVICE if any bit was set,
 * LQ_OK otherwise (LQ_EHIP if synchronisation failed).
 */
int32_t leapquant_check_error(const lq_state *st, void *stream, int32_t *bits_out);

/* Static description of a status code. */
const char *leapquant_strerror(int32_t status);

/* Text of the last HIP error seen by this thread in a failing call, or "". */
const char *leapquant_last_hip_error(void);

#ifdef __cplusplus
}
#endif

#endif /* LEAPQUANT_H */
