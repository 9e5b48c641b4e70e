// Decode step: one token for every (request, head) tile.
//
// One 256-thread workgroup owns one tile.  With i = rec_len + 1 it reads
//   A_i^T x = delta . (Z^T (c . Gamma_{1:i} x))            quantized residual
//           + U~ (K~^T (Gamma_{1:i} x))                     Compensator Tokens
//           + sum_{j<i} u_j (k~_j^T (Gamma_{j+1:i} x))      buffered records
// for x = k_t and x = q_t in one pass over the codes (App. B.2 Eq. (readout),
// App. B.3 Eq. (smooth-readout)), then forms u_t = fp16(v_t - A^T k_t), the
// output o_t = A^T q_t + u_t (k~_t . q_t) (post-update state, Sec. 3.1) and
// appends the record (alpha_t, k~_t, u_t) (Sec. 3.2 Eq. (record)).
//
// Every global load of the tile is issued before the first barrier, those that
// do not depend on rec_len first: the token inputs, the d_v x d_k codes (16
// codes per lane: 16, 12 or 8 bytes for 8-, 6- or 4-bit codes, 8 lanes per
// row), the compensators, then rec_len and
// one pass of records (16 slots of 16 lanes, each slot a contiguous block of
// records, 16 bytes of key, correction and decay per lane).  The decays
// Gamma_{j+1:i} are products of the FP16 record decays: each slot forms the
// product of its block, one scan over the 16 slots gives every block the decay
// of all newer records, and the slot walks its block from the newest record
// back.  No d_k x d_v intermediate exists.
#include "lq_device.hpp"
#include "lq_internal.hpp"

namespace lq {

namespace {

constexpr int SLOTS = 16;            // 16-lane groups per workgroup
// Records per slot and pass: the diagonal gate carries a 16-byte decay per lane
// and record, so it holds two per slot (32 per pass) to stay at 4 resident
// workgroups per CU; the scalar gate holds four (64 per pass).
template <int GATE> struct Pass {
    static constexpr int PER_SLOT = GATE ? 2 : 4;
    static constexpr int N = SLOTS * PER_SLOT;
};

struct DecodeArgs {
    const uint8_t *codes;
    const float *scale;
    const float *smooth;
    const uint16_t *comp_k;
    const uint16_t *comp_u;
    uint16_t *rec_k;
    uint16_t *rec_u;
    uint16_t *rec_a;
    int32_t *rec_len;
    int32_t *err;
    const float *q;
    const float *k;
    const float *v;
    const float *alpha;
    const float *beta;
    float *o;
    int heads_v;
    int group;      // heads_v / heads_k
    int window;
    int n_comp;
    int tiles;
};

template <int GATE>
struct RecRegs {
    static constexpr int PER_SLOT = Pass<GATE>::PER_SLOT;
    uint4 k[PER_SLOT];               // FP16 keys, 8 channels
    uint4 u[PER_SLOT];               // FP16 corrections, 8 values
    uint4 a[GATE ? PER_SLOT : 1];    // FP16 decays, 8 channels (diagonal gate)
    float as[PER_SLOT];              // decay (scalar gate)
};

// Issue the loads of the records in [lo, hi) that belong to slot ts: record
// hi-1-(PER_SLOT*ts+q) goes to register set q (newest first).
// y = Gamma_{1:i} x and w = c . y for x = k_t, q_t (thread t < D: channel t).
__device__ __forceinline__ void write_base_vectors(float G, float kx, float qx, float cs, float (*s_y)[D],
                                                   float (*s_w)[D], int t) {
    const float yk = G * kx, yq = G * qx;
    s_y[0][t] = yk;
    s_y[1][t] = yq;
    s_w[0][t] = cs * yk;
    s_w[1][t] = cs * yq;
}

// 16 consecutive codes of a row: 16 bytes (byte formats), 8 (INT4) or 12 (INT6).
template <int CODE>
__device__ __forceinline__ uint4 load_codes16(const uint8_t *p) {
    if (CODE <= 1) return *(const uint4 *)p;
    if (CODE == 2) {
        const uint2 w = *(const uint2 *)p;
        return make_uint4(w.x, w.y, 0u, 0u);
    }
    const uint32_t *w = (const uint32_t *)p;
    return make_uint4(w[0], w[1], w[2], 0u);
}

template <int GATE>
__device__ __forceinline__ void load_records(const DecodeArgs &a, size_t rbase, int lo, int hi,
                                             int ts, int l16, RecRegs<GATE> &R) {
    constexpr int PER_SLOT = Pass<GATE>::PER_SLOT;
#pragma unroll
    for (int q = 0; q < PER_SLOT; ++q) {
        const int r = hi - 1 - (PER_SLOT * ts + q);
        if (r >= lo) {
            R.k[q] = *(const uint4 *)(a.rec_k + (rbase + r) * D + 8 * l16);
            R.u[q] = *(const uint4 *)(a.rec_u + (rbase + r) * D + 8 * l16);
            if (GATE) R.a[q] = *(const uint4 *)(a.rec_a + (rbase + r) * D + 8 * l16);
            else R.as[q] = h2f(a.rec_a[rbase + r]);
        }
    }
}

template <int GATE, int CODE, int RULE>
__global__ __launch_bounds__(NT) void decode_kernel(DecodeArgs a) {
    constexpr int G = GATE ? D : 1;     // decay values per record
    __shared__ float s_x[2][D];          // x = k_t, q_t
    __shared__ float s_w[2][D];          // c . Gamma_{1:i} . x
    __shared__ float s_y[2][D];          // Gamma_{1:i} . x
    __shared__ float s_z[2][D];          // quantized-residual readout
    __shared__ float s_kq[2];            // k~_t . q_t (per wave pair)
    __shared__ union {
        struct {
            float bp[SLOTS][G];          // decay product of each slot's block
            float pre[SLOTS][G];         // decay of everything newer than the block
        } scan;
        float red[SLOTS][2][D];          // per-slot partial readouts
    } u_;

    const int tile = blockIdx.x;
    const int tid = threadIdx.x;
    const int b = tile / a.heads_v, hv = tile - b * a.heads_v;
    const size_t kvec = ((size_t)b * (a.heads_v / a.group) + hv / a.group) * D;
    const size_t tvec = (size_t)tile * D;

    const int l16 = tid & 15;            // 8-channel key segment / 8-value segment
    const int ts = tid >> 4;             // slot 0..15
    const int g8 = tid & 7;              // 16-channel key segment of the code rows
    const int rg = tid >> 3;             // code rows rg, rg+32, rg+64, rg+96
    const size_t rbase = (size_t)tile * a.window;

    // ---- issue every load of the tile: first what does not depend on rec_len ----
    float kx = 0.0f, qx = 0.0f, cs = 0.0f, al = 0.0f, vx = 0.0f, bt = 0.0f;
    if (tid < D) {
        kx = a.k[kvec + tid];
        qx = a.q[kvec + tid];
        cs = a.smooth[tvec + tid];
        al = GATE ? a.alpha[tvec + tid] : a.alpha[tile];
        vx = a.v[tvec + tid];
        bt = a.beta[tile];
    }
    constexpr int ROWB = D * CodeFmt<CODE>::BITS / 8;   // code bytes per value row
    const uint8_t *zt = a.codes + (size_t)tile * D * ROWB;
    uint4 zr[4];
#pragma unroll
    for (int m = 0; m < 4; ++m) zr[m] = load_codes16<CODE>(zt + (size_t)(rg + 32 * m) * ROWB + 2 * CodeFmt<CODE>::BITS * g8);
    float dlt[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    if (g8 == 0) {
#pragma unroll
        for (int m = 0; m < 4; ++m) dlt[m] = a.scale[tvec + rg + 32 * m];
    }
    uint4 ck = make_uint4(0, 0, 0, 0), cu = make_uint4(0, 0, 0, 0);
    if (ts < a.n_comp) {
        const size_t cb = ((size_t)tile * a.n_comp + ts) * D + 8 * l16;
        ck = *(const uint4 *)(a.comp_k + cb);
        cu = *(const uint4 *)(a.comp_u + cb);
    }
    const int n = a.rec_len[tile];
    if (n >= a.window || n < 0) {        // window buffer full (or corrupt): tile untouched
        if (tid == 0) atomicOr(a.err, n < 0 ? (int)LQ_DEVERR_BAD_REC_LEN : (int)LQ_DEVERR_WINDOW_FULL);
        if (tid < D) a.o[tvec + tid] = __builtin_nanf("");
        return;
    }
    RecRegs<GATE> R;
    constexpr int PER_SLOT = Pass<GATE>::PER_SLOT, PASS = Pass<GATE>::N;
    int hi = n, lo = n > PASS ? n - PASS : 0;
    load_records<GATE>(a, rbase, lo, hi, ts, l16, R);

    // ---- token inputs, this token's record -------------------------------------
    // carry: decay of every record newer than the current pass, channel tid
    // (the scalar gate keeps the same product in every thread below D)
    float carry = 1.0f;
    if (tid < D) {
        s_x[0][tid] = kx;
        s_x[1][tid] = qx;
        const uint16_t ah = f2h(al);
        carry = h2f(ah);
        const size_t slot = rbase + n;
        if (GATE) a.rec_a[slot * D + tid] = ah;
        else if (tid == 0) a.rec_a[slot] = ah;
        const uint16_t tkh = f2h(bt * kx);                   // k~_t = fp16(beta_t k_t)
        a.rec_k[slot * D + tid] = tkh;
        const float kq = wave_sum(h2f(tkh) * qx);
        if ((tid & 63) == 0) s_kq[tid >> 6] = kq;
    }

    float acc_k[8], acc_q[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) acc_k[j] = acc_q[j] = 0.0f;

    // ---- buffered records, newest first, up to PASS per pass ----------------------
    if (n > 0) {
        bool first = true;
        float xk[8], xq[8];
        while (true) {
            // decay product of this slot's block, per channel of its segment
            float bp[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) bp[j] = 1.0f;
#pragma unroll
            for (int q = 0; q < PER_SLOT; ++q) {
                if (hi - 1 - (PER_SLOT * ts + q) >= lo) {
                    if (GATE) {
                        float av[8];
                        unpack_h8(R.a[q], av);
#pragma unroll
                        for (int j = 0; j < 8; ++j) bp[j] *= av[j];
                    } else {
                        bp[0] *= R.as[q];
                    }
                }
            }
            if (GATE) {
#pragma unroll
                for (int j = 0; j < 8; ++j) u_.scan.bp[ts][8 * l16 + j] = bp[j];
            } else if (l16 == 0) {
                u_.scan.bp[ts][0] = bp[0];
            }
            __syncthreads();
            if (first) {
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    xk[j] = s_x[0][8 * l16 + j];
                    xq[j] = s_x[1][8 * l16 + j];
                }
                first = false;
            }
            // exclusive scan over the slots; slot 0 holds the newest block
            if (tid < D) {
                const int ch = GATE ? tid : 0;
                float c = carry;
                if (GATE) {                  // slot products read ahead of the chain
                    float bv[SLOTS];
#pragma unroll
                    for (int s = 0; s < SLOTS; ++s) bv[s] = u_.scan.bp[s][ch];
#pragma unroll
                    for (int s = 0; s < SLOTS; ++s) {
                        u_.scan.pre[s][ch] = c;
                        c *= bv[s];
                    }
                } else {
#pragma unroll
                    for (int s = 0; s < SLOTS; ++s) {
                        if (tid == 0) u_.scan.pre[s][0] = c;
                        c *= u_.scan.bp[s][0];
                    }
                }
                carry = c;
                if (lo == 0) write_base_vectors(carry, kx, qx, cs, s_y, s_w, tid);   // carry = Gamma_{1:i}
            }
            __syncthreads();
            if (GATE) {
                float P[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) P[j] = u_.scan.pre[ts][8 * l16 + j];
#pragma unroll
                for (int q = 0; q < PER_SLOT; ++q) {
                    if (hi - 1 - (PER_SLOT * ts + q) < lo) break;    // uniform within the slot
                    // products with an FP16 operand are written as fma(h, x, 0), which
                    // takes the half directly (same value as the product)
                    float kv[8], uv[8];
                    unpack_h8(R.k[q], kv);
                    unpack_h8(R.u[q], uv);
                    float pk = 0.0f, pq = 0.0f;
#pragma unroll
                    for (int j = 0; j < 8; ++j) {
                        const float t = fmaf(kv[j], P[j], 0.0f);
                        pk = fmaf(t, xk[j], pk);
                        pq = fmaf(t, xq[j], pq);
                    }
                    pk = row16_sum(pk);
                    pq = row16_sum(pq);
#pragma unroll
                    for (int j = 0; j < 8; ++j) {
                        acc_k[j] = fmaf(pk, uv[j], acc_k[j]);
                        acc_q[j] = fmaf(pq, uv[j], acc_q[j]);
                    }
                    float av[8];
                    unpack_h8(R.a[q], av);
#pragma unroll
                    for (int j = 0; j < 8; ++j) P[j] = fmaf(av[j], P[j], 0.0f);
                }
            } else {
                // scalar decay: one product per slot, applied to the two dot products
                float P = u_.scan.pre[ts][0];
#pragma unroll
                for (int q = 0; q < PER_SLOT; ++q) {
                    if (hi - 1 - (PER_SLOT * ts + q) < lo) break;    // uniform within the slot
                    float kv[8], uv[8];
                    unpack_h8(R.k[q], kv);
                    unpack_h8(R.u[q], uv);
                    float pk = 0.0f, pq = 0.0f;
#pragma unroll
                    for (int j = 0; j < 8; ++j) {
                        pk = fmaf(kv[j], xk[j], pk);
                        pq = fmaf(kv[j], xq[j], pq);
                    }
                    pk = row16_sum(pk) * P;
                    pq = row16_sum(pq) * P;
#pragma unroll
                    for (int j = 0; j < 8; ++j) {
                        acc_k[j] = fmaf(pk, uv[j], acc_k[j]);
                        acc_q[j] = fmaf(pq, uv[j], acc_q[j]);
                    }
                    P *= R.as[q];
                }
            }
            if (lo == 0) break;
            // older records: another pass (scalar gate with W > 64 only).  The
            // next pass's first barrier orders these scan reads before its writes.
            hi = lo;
            lo = hi > PASS ? hi - PASS : 0;
            load_records<GATE>(a, rbase, lo, hi, ts, l16, R);
        }
    }

    // ---- base and token read vectors (written with the last scan when n > 0) -----
    if (n == 0) {
        if (tid < D) write_base_vectors(carry, kx, qx, cs, s_y, s_w, tid);
        __syncthreads();
    }

    // ---- quantized residual: rows rg + 32m, channels 16*g8 .. +15 ---------------
    {
        float wk[16], wq[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            wk[j] = s_w[0][16 * g8 + j];
            wq[j] = s_w[1][16 * g8 + j];
        }
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            float f[16];
            decode16<CODE>(zr[m], f);
            float pk = 0.0f, pq = 0.0f;
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                pk = fmaf(f[j], wk[j], pk);
                pq = fmaf(f[j], wq[j], pq);
            }
            pk = row8_sum(pk);
            pq = row8_sum(pq);
            if (g8 == 0) {
                const int vrow = rg + 32 * m;
                s_z[0][vrow] = dlt[m] * pk;
                s_z[1][vrow] = dlt[m] * pq;
            }
        }
    }

    // ---- Compensator Tokens: token ts, same decay as the base -------------------
    if (ts < a.n_comp) {
        float kv[8], uv[8];
        unpack_h8(ck, kv);
        unpack_h8(cu, uv);
        float pk = 0.0f, pq = 0.0f;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            pk = fmaf(kv[j], s_y[0][8 * l16 + j], pk);
            pq = fmaf(kv[j], s_y[1][8 * l16 + j], pq);
        }
        pk = row16_sum(pk);
        pq = row16_sum(pq);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            acc_k[j] = fmaf(pk, uv[j], acc_k[j]);
            acc_q[j] = fmaf(pq, uv[j], acc_q[j]);
        }
    }
    // the scan buffers are dead since the barrier above; reuse them
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        u_.red[ts][0][8 * l16 + j] = acc_k[j];
        u_.red[ts][1][8 * l16 + j] = acc_q[j];
    }
    __syncthreads();

    // ---- combine, correction, output, record ------------------------------------
    if (tid < D) {
        float ak = s_z[0][tid], aq = s_z[1][tid];
#pragma unroll
        for (int s = 0; s < SLOTS; ++s) {
            ak += u_.red[s][0][tid];
            aq += u_.red[s][1][tid];
        }
        // u_t = fp16(v_t - A^T k_t); the b_t = 0 rule reads nothing (the k-side
        // readouts above are then dead code and compiled out)
        const uint16_t uh = f2h(RULE == LQ_RULE_ADD ? vx : vx - ak);
        a.rec_u[(rbase + n) * D + tid] = uh;
        a.o[tvec + tid] = fmaf(h2f(uh), s_kq[0] + s_kq[1], aq);
        if (tid == 0) a.rec_len[tile] = n + 1;
    }
}

template <int GATE, int CODE>
hipError_t launch(const DecodeArgs &args, int rule, hipStream_t st) {
    if (rule == LQ_RULE_ADD)
        hipLaunchKernelGGL((decode_kernel<GATE, CODE, LQ_RULE_ADD>), dim3(args.tiles), dim3(NT), 0, st, args);
    else
        hipLaunchKernelGGL((decode_kernel<GATE, CODE, LQ_RULE_DELTA>), dim3(args.tiles), dim3(NT), 0, st, args);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_decode(const lq_dims &d, const StatePtrs &s, const TokenPtrs &t, hipStream_t st) {
    DecodeArgs a;
    a.codes = (const uint8_t *)s.codes;
    a.scale = s.scale;
    a.smooth = s.smooth;
    a.comp_k = s.comp_k;
    a.comp_u = s.comp_u;
    a.rec_k = s.rec_k;
    a.rec_u = s.rec_u;
    a.rec_a = s.rec_a;
    a.rec_len = s.rec_len;
    a.err = s.err;
    a.q = t.q;
    a.k = t.k;
    a.v = t.v;
    a.alpha = t.alpha;
    a.beta = t.beta;
    a.o = t.o;
    a.heads_v = d.heads_v;
    a.group = d.heads_v / d.heads_k;
    a.window = d.window;
    a.n_comp = d.n_comp;
    a.tiles = d.batch * d.heads_v;
    if (d.gate == LQ_GATE_DIAG) {
        switch (d.code) {
            case LQ_CODE_E4M3: return launch<1, 1>(a, d.rule, st);
            case LQ_CODE_INT4: return launch<1, 2>(a, d.rule, st);
            case LQ_CODE_INT6: return launch<1, 3>(a, d.rule, st);
            default: return launch<1, 0>(a, d.rule, st);
        }
    }
    switch (d.code) {
        case LQ_CODE_E4M3: return launch<0, 1>(a, d.rule, st);
        case LQ_CODE_INT4: return launch<0, 2>(a, d.rule, st);
        case LQ_CODE_INT6: return launch<0, 3>(a, d.rule, st);
        default: return launch<0, 0>(a, d.rule, st);
    }
}

}  // namespace lq
