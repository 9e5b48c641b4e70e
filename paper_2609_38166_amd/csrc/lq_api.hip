// C ABI of the LeapQuant decode path: host-side validation and launches.
// Every entry point validates its arguments completely before it enqueues
// anything, allocates nothing and (except leapquant_check_error) never waits.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include "leapquant.h"
#include "lq_internal.hpp"

namespace {

thread_local char g_last_hip[256] = "";

int32_t hip_status(hipError_t e) {
    if (e == hipSuccess) return LQ_OK;
    strncpy(g_last_hip, hipGetErrorString(e), sizeof(g_last_hip) - 1);
    g_last_hip[sizeof(g_last_hip) - 1] = '\0';
    return LQ_EHIP;
}

bool aligned(const void *p) { return ((uintptr_t)p & 15u) == 0; }

int32_t check_ptr(const void *p) {
    if (!p) return LQ_EINVAL;
    if (!aligned(p)) return LQ_EALIGN;
    return LQ_OK;
}

int32_t check_dims(const lq_dims *d) {
    if (!d) return LQ_EINVAL;
    if (d->batch <= 0 || d->heads_v <= 0 || d->heads_k <= 0 || d->d_k <= 0 || d->d_v <= 0 ||
        d->window <= 0 || d->n_comp < 0 || d->power_iters < 0)
        return LQ_EINVAL;
    if (d->heads_v % d->heads_k != 0) return LQ_EINVAL;
    if (d->gate != LQ_GATE_SCALAR && d->gate != LQ_GATE_DIAG) return LQ_EINVAL;
    if (d->code != LQ_CODE_INT8 && d->code != LQ_CODE_E4M3 && d->code != LQ_CODE_INT4 &&
        d->code != LQ_CODE_INT6 && d->code != LQ_CODE_BF16)
        return LQ_EINVAL;
    if (d->smooth != 0 && d->smooth != 1) return LQ_EINVAL;
    if (d->rule != LQ_RULE_DELTA && d->rule != LQ_RULE_ADD && d->rule != LQ_RULE_GENERAL)
        return LQ_EINVAL;
    if (d->d_k != 128 || d->d_v != 128) return LQ_EUNSUPPORTED;
    if (d->n_comp > LQ_MAX_COMP) return LQ_EUNSUPPORTED;
    if (d->code == LQ_CODE_BF16 && d->n_comp != 0) return LQ_EUNSUPPORTED;   // no tokens on a BF16 state
    if (d->n_comp > 0 && (d->power_iters < 1 || d->power_iters > LQ_MAX_POWER_ITERS))
        return LQ_EUNSUPPORTED;
    const int wmax = d->gate == LQ_GATE_DIAG ? LQ_MAX_WINDOW_KDA : LQ_MAX_WINDOW_GDN;
    if (d->window > wmax) return LQ_EUNSUPPORTED;
    // tile index and per-buffer element counts must fit the kernels' integer types
    // (the decode maps a tile to its key head as tile * ceil(2^32 / group) >> 32,
    // exact while tiles * group < 2^32)
    const long long tiles = (long long)d->batch * d->heads_v;
    if (tiles > (1LL << 30)) return LQ_EUNSUPPORTED;
    if (tiles * (d->heads_v / d->heads_k) >= (1LL << 32)) return LQ_EUNSUPPORTED;
    return LQ_OK;
}

// Arrays that every kernel reads one element at a time need only the
// element's alignment: the per-tile scalars beta and (scalar gate) alpha,
// rec_len, err and the commit mask 4 bytes, the scalar gate's FP16 decays
// 2 bytes.  So step-major token buffers can be passed one step at a time, and
// a group of requests as views into a larger state, for any tile count.  Every
// other array is read in 16-byte vectors by some kernel.
int32_t check_ptr_n(const void *p, uintptr_t n) {
    if (!p) return LQ_EINVAL;
    if ((uintptr_t)p & (n - 1)) return LQ_EALIGN;
    return LQ_OK;
}
int32_t check_ptr4(const void *p) { return check_ptr_n(p, 4); }

int32_t check_state(const lq_dims *d, const lq_state *st) {
    if (!st) return LQ_EINVAL;
    int32_t e;
    const void *ptrs[] = {st->codes, st->scale, st->smooth, st->rec_k, st->rec_u};
    for (const void *p : ptrs)
        if ((e = check_ptr(p)) != LQ_OK) return e;
    if ((e = d->gate == LQ_GATE_DIAG ? check_ptr(st->rec_a) : check_ptr_n(st->rec_a, 2)) != LQ_OK) return e;
    if ((e = check_ptr4(st->rec_len)) != LQ_OK) return e;
    if (d->n_comp > 0) {
        if ((e = check_ptr(st->comp_k)) != LQ_OK) return e;
        if ((e = check_ptr(st->comp_u)) != LQ_OK) return e;
    }
    if ((e = check_ptr4(st->err)) != LQ_OK) return e;
    return LQ_OK;
}

int32_t check_tokens(const lq_dims *d, const float *q, const float *k, const float *v,
                     const float *alpha, const float *beta, const float *o) {
    int32_t e;
    if ((e = d->gate == LQ_GATE_DIAG ? check_ptr(alpha) : check_ptr4(alpha)) != LQ_OK) return e;
    if ((e = check_ptr4(beta)) != LQ_OK) return e;
    const void *ptrs[] = {q, k, v, o};
    for (const void *p : ptrs)
        if ((e = check_ptr(p)) != LQ_OK) return e;
    return LQ_OK;
}

lq::StatePtrs state_ptrs(const lq_state *st) {
    lq::StatePtrs s;
    s.codes = st->codes;
    s.scale = st->scale;
    s.smooth = st->smooth;
    s.comp_k = st->comp_k;
    s.comp_u = st->comp_u;
    s.rec_k = st->rec_k;
    s.rec_u = st->rec_u;
    s.rec_a = st->rec_a;
    s.rec_len = st->rec_len;
    s.err = st->err;
    return s;
}

}  // namespace

extern "C" {

int32_t leapquant_state_bytes(const lq_dims *d, size_t out[10]) {
    int32_t e = check_dims(d);
    if (e != LQ_OK) return e;
    if (!out) return LQ_EINVAL;
    const size_t t = (size_t)d->batch * d->heads_v, dk = d->d_k, dv = d->d_v;
    const size_t r = d->n_comp, W = d->window, g = d->gate == LQ_GATE_DIAG ? dk : 1;
    const size_t bits = d->code == LQ_CODE_INT4 ? 4 : d->code == LQ_CODE_INT6 ? 6 : d->code == LQ_CODE_BF16 ? 16 : 8;
    out[0] = t * dv * dk * bits / 8;   // codes
    out[1] = t * dv * 4;         // scale
    out[2] = t * dk * 4;         // smooth
    out[3] = t * r * dk * 2;     // comp_k
    out[4] = t * r * dv * 2;     // comp_u
    out[5] = t * W * dk * 2;     // rec_k
    out[6] = t * W * dv * 2;     // rec_u
    out[7] = t * W * g * 2;      // rec_a
    out[8] = t * 4;              // rec_len
    out[9] = 4;                  // err
    return LQ_OK;
}

int32_t leapquant_quantize_state(const lq_dims *d, const float *S, lq_state *st, void *stream) {
    int32_t e = check_dims(d);
    if (e != LQ_OK) return e;
    if ((e = check_state(d, st)) != LQ_OK) return e;
    if ((e = check_ptr(S)) != LQ_OK) return e;
    return hip_status(lq::launch_tile(*d, state_ptrs(st), lq::TILE_QUANTIZE, S, nullptr, nullptr,
                                      (hipStream_t)stream));
}

int32_t leapquant_decode_step(const lq_dims *d, lq_state *st, const float *q, const float *k,
                              const float *v, const float *alpha, const float *beta, float *o,
                              void *stream) {
    int32_t e = check_dims(d);
    if (e != LQ_OK) return e;
    if ((e = check_state(d, st)) != LQ_OK) return e;
    if (d->rule == LQ_RULE_GENERAL) return LQ_EINVAL;   // needs the read vectors
    if ((e = check_tokens(d, q, k, v, alpha, beta, o)) != LQ_OK) return e;
    lq::TokenPtrs t{q, k, v, alpha, beta, o, nullptr};
    return hip_status(lq::launch_decode(*d, state_ptrs(st), t, (hipStream_t)stream));
}

int32_t leapquant_decode_step_commit(const lq_dims *d, lq_state *st, const float *q, const float *k,
                                     const float *v, const float *alpha, const float *beta, float *o,
                                     void *stream) {
    int32_t e = check_dims(d);
    if (e != LQ_OK) return e;
    if ((e = check_state(d, st)) != LQ_OK) return e;
    if (d->rule == LQ_RULE_GENERAL) return LQ_EINVAL;   // needs the read vectors
    if ((e = check_tokens(d, q, k, v, alpha, beta, o)) != LQ_OK) return e;
    lq::TokenPtrs t{q, k, v, alpha, beta, o, nullptr};
    return hip_status(lq::launch_decode_commit(*d, state_ptrs(st), t, (hipStream_t)stream));
}

int32_t leapquant_decode_step_general(const lq_dims *d, lq_state *st, const float *q,
                                      const float *k, const float *b, const float *v,
                                      const float *alpha, const float *beta, float *o,
                                      void *stream) {
    int32_t e = check_dims(d);
    if (e != LQ_OK) return e;
    if ((e = check_state(d, st)) != LQ_OK) return e;
    if (d->rule != LQ_RULE_GENERAL) return LQ_EINVAL;
    if ((e = check_tokens(d, q, k, v, alpha, beta, o)) != LQ_OK) return e;
    if ((e = check_ptr(b)) != LQ_OK) return e;
    lq::TokenPtrs t{q, k, v, alpha, beta, o, b};
    return hip_status(lq::launch_decode(*d, state_ptrs(st), t, (hipStream_t)stream));
}

int32_t leapquant_window_commit(const lq_dims *d, lq_state *st, const int32_t *mask, void *stream) {
    int32_t e = check_dims(d);
    if (e != LQ_OK) return e;
    if ((e = check_state(d, st)) != LQ_OK) return e;
    if (mask && ((uintptr_t)mask & 3u)) return LQ_EALIGN;
    return hip_status(lq::launch_tile(*d, state_ptrs(st), lq::TILE_COMMIT, nullptr, nullptr, mask,
                                      (hipStream_t)stream));
}

int32_t leapquant_baseline_step(const lq_dims *d, void *S, int32_t state_dtype, const float *q,
                                const float *k, const float *v, const float *alpha,
                                const float *beta, float *o, void *stream) {
    int32_t e = check_dims(d);
    if (e != LQ_OK) return e;
    if (state_dtype != LQ_STATE_F32 && state_dtype != LQ_STATE_BF16) return LQ_EINVAL;
    if ((e = check_ptr(S)) != LQ_OK) return e;
    if (d->rule == LQ_RULE_GENERAL) return LQ_EINVAL;   // needs the read vectors
    if ((e = check_tokens(d, q, k, v, alpha, beta, o)) != LQ_OK) return e;
    lq::TokenPtrs t{q, k, v, alpha, beta, o, nullptr};
    return hip_status(lq::launch_baseline(*d, S, state_dtype, t, (hipStream_t)stream));
}

int32_t leapquant_baseline_step_general(const lq_dims *d, void *S, int32_t state_dtype,
                                        const float *q, const float *k, const float *b,
                                        const float *v, const float *alpha, const float *beta,
                                        float *o, void *stream) {
    int32_t e = check_dims(d);
    if (e != LQ_OK) return e;
    if (state_dtype != LQ_STATE_F32 && state_dtype != LQ_STATE_BF16) return LQ_EINVAL;
    if (d->rule != LQ_RULE_GENERAL) return LQ_EINVAL;
    if ((e = check_ptr(S)) != LQ_OK) return e;
    if ((e = check_tokens(d, q, k, v, alpha, beta, o)) != LQ_OK) return e;
    if ((e = check_ptr(b)) != LQ_OK) return e;
    lq::TokenPtrs t{q, k, v, alpha, beta, o, b};
    return hip_status(lq::launch_baseline(*d, S, state_dtype, t, (hipStream_t)stream));
}

int32_t leapquant_dequantize_state(const lq_dims *d, const lq_state *st, float *S_out,
                                   void *stream) {
    int32_t e = check_dims(d);
    if (e != LQ_OK) return e;
    if ((e = check_state(d, st)) != LQ_OK) return e;
    if ((e = check_ptr(S_out)) != LQ_OK) return e;
    return hip_status(lq::launch_tile(*d, state_ptrs(st), lq::TILE_DEQUANT, nullptr, S_out,
                                      nullptr, (hipStream_t)stream));
}

int32_t leapquant_check_error(const lq_state *st, void *stream, int32_t *bits_out) {
    if (!st || !st->err) return LQ_EINVAL;
    hipStream_t s = (hipStream_t)stream;
    int32_t bits = 0;
    hipError_t h = hipMemcpyAsync(&bits, st->err, sizeof(bits), hipMemcpyDeviceToHost, s);
    if (h == hipSuccess) h = hipStreamSynchronize(s);
    if (h != hipSuccess) return hip_status(h);
    if (bits_out) *bits_out = bits;
    if (bits) {
        const int32_t zero = 0;
        h = hipMemcpyAsync(st->err, &zero, sizeof(zero), hipMemcpyHostToDevice, s);
        if (h == hipSuccess) h = hipStreamSynchronize(s);
        if (h != hipSuccess) return hip_status(h);
        return LQ_EDEVICE;
    }
    return LQ_OK;
}

const char *leapquant_strerror(int32_t status) {
    switch (status) {
        case LQ_OK: return "success";
        case LQ_EINVAL: return "invalid argument (NULL pointer, non-positive size or bad enum)";
        case LQ_EALIGN: return "pointer not aligned (16 bytes; 4 for beta, scalar-gate alpha, rec_len, err "
                               "and mask; 2 for scalar-gate rec_a)";
        case LQ_EUNSUPPORTED: return "unsupported shape or parameter (d_k/d_v must be 128, r <= 16, "
                                     "W within the gate's limit)";
        case LQ_EHIP: return "HIP runtime error (see leapquant_last_hip_error)";
        case LQ_EDEVICE: return "device-side error flag was set (e.g. decode on a full window)";
        default: return "unknown status";
    }
}

const char *leapquant_last_hip_error(void) { return g_last_hip; }

}  // extern "C"
