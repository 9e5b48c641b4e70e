// Decode step: one token for every (request, head) tile.
//
// One 256-thread workgroup owns one tile.  With i = rec_len + 1 it reads
//   A_i^T x = delta . (Z^T (c . Gamma_{1:i} x))            quantized residual
//           + U~ (K~^T (Gamma_{1:i} x))                     Compensator Tokens
//           + sum_{j<i} u_j (k~_j^T (Gamma_{j+1:i} x))      buffered records
// for x = k_t and x = q_t in one pass over the codes (App. B.2 Eq. (readout),
// App. B.3 Eq. (smooth-readout)), then forms the correction
// u_t = fp16(v_t - A^T k_t), the output o_t = A^T q_t + u_t (k~_t . q_t)
// (post-update state, Sec. 3.1) and appends the record (alpha_t, k~_t, u_t)
// (Sec. 3.2 Eq. (record)).  Under the general rule (read vector b_t given,
// App. A) the same pass reads S_{i-1}^T x, i.e. the decays Gamma_{.:i-1}
// without this token's, for x = b_t and x = d_t . q_t (d_t the FP16 decay),
// and u_t = fp16(v_t - S_{i-1}^T b_t).
//
// Precision.  The correction is rounded to FP16 and stored; every later step
// and the window-end refit read the rounded value, so a rounding decision
// taken differently here changes the state.  The k side (the readout that
// feeds u_t) is therefore carried at fp64 accuracy, which makes u_t the
// correctly rounded FP16 value of the exact expression except in cases of
// probability ~1e-10: decay products, record and compensator readouts in
// fp64, and the code product exact in integer arithmetic.  The read vector
// w = c . Gamma x is written as a fixed-point number, an exponent per 64
// channels and five base-128 digits (34 bits, each digit an int8), and
// Z^T w is a sum of int8 x int8 products per digit, taken on the int8 matrix
// cores (v_mfma_i32_16x16x64_i8, exact int32 sums) and combined in fp64
// exactly.  The q side, which only feeds the output, uses three digits and
// fp32.  E4M3 codes are not integers, and the BF16 state is not either; their
// products are taken in fp64 (k side) and fp32 (q side) on the vector ALU.
//
// Every global load of the tile is issued before the first barrier: rec_len (a
// scalar load, which the record loads wait for), the token inputs, the
// d_v x d_k codes and row scales (copied straight into LDS, 16 bytes per lane
// and instruction, so they hold no registers), the compensators, then one pass
// of records, loaded non-temporally (16 slots of 16 lanes, each slot a
// contiguous block of ceil(count / 16) records, 16 bytes of key, correction
// and decay per lane).  The decays Gamma_{j+1:i} are products of the FP16 record decays:
// each slot forms the product of its block, one scan over the 16 slots gives
// every block the decay of all newer records, and the slot walks its block
// from the newest record back.  No d_k x d_v intermediate exists.
#pragma once

#include "lq_device.hpp"
#include "lq_internal.hpp"

namespace lq {

namespace {

constexpr int SLOTS = 16;            // 16-lane groups per workgroup
// Records per slot and pass: the diagonal gate carries a 16-byte decay per lane
// and record, so it holds three per slot (48 per pass); the scalar gate holds
// four (64 per pass).
template <int GATE> struct Pass {
    static constexpr int PER_SLOT = GATE ? 3 : 4;
    static constexpr int N = SLOTS * PER_SLOT;
};

// Base-128 digits of the read vectors of the code product.
constexpr int KDIG = 5;              // k side: 6 + 4 x 7 = 34 bits
constexpr int QDIG = 3;              // q side: 20 bits
constexpr int NDIG = KDIG + QDIG;

// Per-channel vectors that the slots read 8 channels at a time are kept in LDS
// in a swizzled order: channel 8*l16 + j sits at position 16*j + l16, so for
// each j the 16 lanes of a slot touch 16 consecutive words.  A thread t < D
// that works on a whole vector (the scan, the base vectors, the final combine)
// owns position t, i.e. channel CH(t); POS is the inverse map.  Threads
// 0..63 own the channels c with (c & 7) < 4, threads 64..127 the others.
__device__ __forceinline__ constexpr int SW(int l16, int j) { return 16 * j + l16; }
__device__ __forceinline__ constexpr int CH(int t) { return 8 * (t & 15) + (t >> 4); }
__device__ __forceinline__ constexpr int POS(int c) { return 16 * (c & 7) + (c >> 3); }
static_assert(CH(POS(77)) == 77 && POS(CH(77)) == 77, "CH and POS are inverse");

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
    const float *b;  // read vectors [tiles][D] (general rule)
    uint64_t kv_mul; // ceil(2^32 / group), group = heads_v / heads_k
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
    uint32_t as[PER_SLOT];           // FP16 decay (scalar gate), converted where used
};

// Non-temporal 16-byte load, for the records: a step streams every tile's
// buffered records once, and as plain loads they would evict the codes from
// the last-level (Infinity) cache, where a batch's codes can stay resident
// from one step to the next.
__device__ __forceinline__ uint4 ld_stream16(const uint16_t *p) {
    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
    const u32x4 v = __builtin_nontemporal_load((const u32x4 *)p);
    return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ double h2d(uint32_t w, int hi) {
    return (double)h2f((uint16_t)(w >> (16 * hi)));
}

// Cross-row swaps of a double (two 32-bit halves).
__device__ __forceinline__ void swap32_d(double a, double b, double &ra, double &rb) {
    const auto lo = __builtin_amdgcn_permlane32_swap(__double2loint(a), __double2loint(b), false, false);
    const auto hi = __builtin_amdgcn_permlane32_swap(__double2hiint(a), __double2hiint(b), false, false);
    ra = __hiloint2double(hi[0], lo[0]);
    rb = __hiloint2double(hi[1], lo[1]);
}
__device__ __forceinline__ void swap16_d(double a, double b, double &ra, double &rb) {
    const auto lo = __builtin_amdgcn_permlane16_swap(__double2loint(a), __double2loint(b), false, false);
    const auto hi = __builtin_amdgcn_permlane16_swap(__double2hiint(a), __double2hiint(b), false, false);
    ra = __hiloint2double(hi[0], lo[0]);
    rb = __hiloint2double(hi[1], lo[1]);
}

// Sum of x over the 4 slots (16-lane rows) of a wave, for 8 values per lane,
// as a reduce-scatter: lane (row rho, l16) returns the sums of values 2 rho
// and 2 rho + 1.  A cross-row swap of registers (a, b) hands the lower rows
// the upper rows' a and the upper rows the lower rows' b, so own + received is
// the sum wanted in every lane without a select.
__device__ __forceinline__ void rows4_reduce_scatter(const float *x, float &s0, float &s1) {
    float h[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {           // rows rho, rho ^ 2: keep values 4 (rho >> 1) + 0..3
        const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x[i]), __float_as_uint(x[4 + i]), false, false);
        h[i] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
    }
    // rows rho, rho ^ 1: keep 2 of those 4
    const auto r0 = __builtin_amdgcn_permlane16_swap(__float_as_uint(h[0]), __float_as_uint(h[2]), false, false);
    const auto r1 = __builtin_amdgcn_permlane16_swap(__float_as_uint(h[1]), __float_as_uint(h[3]), false, false);
    s0 = __uint_as_float(r0[0]) + __uint_as_float(r0[1]);
    s1 = __uint_as_float(r1[0]) + __uint_as_float(r1[1]);
}
__device__ __forceinline__ void rows4_reduce_scatter(const double *x, double &s0, double &s1) {
    double h[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        double a, b;
        swap32_d(x[i], x[4 + i], a, b);
        h[i] = a + b;
    }
    double a, b;
    swap16_d(h[0], h[2], a, b);
    s0 = a + b;
    swap16_d(h[1], h[3], a, b);
    s1 = a + b;
}

// Largest value of x over the 64 lanes of the wave (every lane gets it).
__device__ __forceinline__ int wave_max_i32(int x) {
    x = max(x, __builtin_amdgcn_update_dpp(0, x, DPP_XOR1, 0xF, 0xF, false));
    x = max(x, __builtin_amdgcn_update_dpp(0, x, DPP_XOR2, 0xF, 0xF, false));
    x = max(x, __builtin_amdgcn_update_dpp(0, x, DPP_ROR4, 0xF, 0xF, false));
    x = max(x, __builtin_amdgcn_update_dpp(0, x, DPP_ROR8, 0xF, 0xF, false));
    const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);     // rows rho, rho ^ 2
    x = max((int)r[0], (int)r[1]);
    const auto r2 = __builtin_amdgcn_permlane16_swap(x, x, false, false);    // rows rho, rho ^ 1
    return max((int)r2[0], (int)r2[1]);
}

// Code rows in LDS are stored in 16-byte chunks, each row rotated by zrot(v)
// chunks, so that the lanes of one matrix-core operand read (16 consecutive
// rows at one chunk position) fall in distinct banks.  The rotation is applied
// when the copy is issued (lane L's destination is fixed; its source chunk is
// chosen).  The 6-bit rows (96 bytes) are not rotated.
template <int CODE> struct Rows {
    static constexpr int BYTES = D * CodeFmt<CODE>::BITS / 8;
    static constexpr int SEGS = BYTES / 16;                 // 16-byte chunks per row
};
template <int CODE> __device__ __forceinline__ int zrot(int v) {
    return CODE == 3 ? 0 : (v & (Rows<CODE>::SEGS - 1));
}
// Chunk c (global numbering) of row v from the rotated LDS copy.
template <int CODE>
__device__ __forceinline__ uint4 lds_chunk(const uint4 *z, int v, int c) {
    constexpr int SEGS = Rows<CODE>::SEGS;
    if (CODE == 3) return z[v * SEGS + c];
    return z[v * SEGS + ((c + zrot<CODE>(v)) & (SEGS - 1))];
}

// Four signed 4-bit codes (a 16-bit field of nibbles) as four int8 bytes:
// bytes b0 b1 of h16 = (n1 n0), (n3 n2) become n0, n1, n2, n3, each sign
// extended through (n ^ 8) + 0x78 ^ 0x80 per byte (no carry between bytes).
__device__ __forceinline__ uint32_t int4x4_to_bytes(uint32_t w, int half) {
    const uint32_t p = __builtin_amdgcn_perm(w, w, half ? 0x03030202u : 0x01010000u);
    const uint32_t t = (p & 0x000F000Fu) | ((p >> 4) & 0x0F000F00u);
    return ((t ^ 0x08080808u) + 0x78787878u) ^ 0x80808080u;
}
// Four signed 6-bit codes (a 24-bit field) as four int8 bytes.
__device__ __forceinline__ uint32_t int6x4_to_bytes(uint32_t g) {
    const uint32_t t = (g & 0x3Fu) | ((g << 2) & 0x3F00u) | ((g << 4) & 0x3F0000u) | ((g << 6) & 0x3F000000u);
    return ((t ^ 0x20202020u) + 0x60606060u) ^ 0x80808080u;
}

// A pass [lo, hi) of records, newest first, is dealt to the slots in
// contiguous blocks of d = ceil((hi - lo) / SLOTS) <= PER_SLOT: slot ts takes
// offsets d ts .. d ts + d - 1, so a short pass spreads over every slot and
// its walk is d records deep.  Record q of slot ts, or -1.
__device__ __forceinline__ int slot_record(int lo, int hi, int d, int ts, int q) {
    const int j = d * ts + q;
    return q < d && j < hi - lo ? hi - 1 - j : -1;
}

template <int GATE>
__device__ __forceinline__ void load_records(const DecodeArgs &a, size_t rbase, int lo, int hi, int d,
                                             int ts, int l16, RecRegs<GATE> &R) {
    constexpr int PER_SLOT = Pass<GATE>::PER_SLOT;
#pragma unroll
    for (int q = 0; q < PER_SLOT; ++q) {
        const int r = slot_record(lo, hi, d, ts, q);
        if (r >= 0) {
            R.k[q] = ld_stream16(a.rec_k + (rbase + r) * D + 8 * l16);
            R.u[q] = ld_stream16(a.rec_u + (rbase + r) * D + 8 * l16);
            if (GATE) R.a[q] = ld_stream16(a.rec_a + (rbase + r) * D + 8 * l16);
            else R.as[q] = __builtin_nontemporal_load(a.rec_a + rbase + r);
        }
    }
}

// LDS of one tile.  The decay array s_bp is reused at the end: wave w writes
// its partial readouts into rows 4w .. 4w+3, which only its own slots read.
template <int CODE>
struct DecodeShared {
    static constexpr int ZCH = D * Rows<CODE>::BYTES / 16;   // 16-byte chunks of a tile's codes
    float x[2][D];                 // x = k_t, q_t (swizzled)
    double yk[D];                  // Gamma_{1:i} . x_k (swizzled), for the compensators
    float yq[D];                   // Gamma_{1:i} . x_q (swizzled)
    double zk[D];                  // code readout delta . Z^T w, k side (by position)
    float zq[D];                   // q side
    float kq[2];                   // k~_t . q_t (per wave)
    int ex[2][2];                  // digit exponents [k, q][scan wave]
    double pre0[SLOTS];            // scalar gate: decay of everything newer than a slot's block
    // read vectors of the code product: NDIG digit rows of D int8 (integer
    // codes), or w_k (fp64) and w_q (fp32) (E4M3), channel order
    __align__(16) uint8_t rv[D * 8 + D * 4];
    __align__(16) double bp[SLOTS][D];   // decay products (swizzled); later the wave partials
    __align__(16) uint4 codes[ZCH];      // the tile's codes, rows rotated by zrot
    __align__(16) float dlt[D];          // the tile's per-row scales
};

// The read vectors of the code product for channel ch (thread t < D):
// w_k = c . y_k and w_q = c . y_q, with y = Gamma_{1:i} x.
template <int CODE, bool KS>
__device__ __forceinline__ void base_vectors(DecodeShared<CODE> &sh, double G, float kx, float qx, float cs,
                                             int t) {
    const int ch = CH(t);
    const double yk = G * (double)kx, yq = G * (double)qx;
    sh.yk[t] = yk;
    sh.yq[t] = (float)yq;
    const double wk = (double)cs * yk, wq = (double)cs * yq;
    if (CODE == 1 || CODE == 4) {
        double *wkv = (double *)sh.rv;
        float *wqv = (float *)(sh.rv + D * 8);
        if (KS) wkv[ch] = wk;
        wqv[ch] = (float)wq;
        return;
    }
    // w = 2^(E - 6) * sum_d digit_d 128^-d with |w| < 2^E over the wave's 64
    // channels, every digit in [-64, 64]: x - rint(x) is exact and in
    // [-1/2, 1/2], and scaling by 128 is exact.
    int8_t *dig = (int8_t *)sh.rv;
    if (KS) {
        const int e = wave_max_i32(__builtin_amdgcn_frexp_exp(wk));
        double x = __builtin_ldexp(wk, 6 - e);
#pragma unroll
        for (int d = 0; d < KDIG; ++d) {
            const double r = __builtin_rint(x);
            dig[d * D + ch] = (int8_t)(int)r;
            x = (x - r) * 128.0;
        }
        if ((t & 63) == 0) sh.ex[0][t >> 6] = e;
    }
    {
        const int e = wave_max_i32(__builtin_amdgcn_frexp_exp(wq));
        double x = __builtin_ldexp(wq, 6 - e);
#pragma unroll
        for (int d = 0; d < QDIG; ++d) {
            const double r = __builtin_rint(x);
            dig[(KDIG + d) * D + ch] = (int8_t)(int)r;
            x = (x - r) * 128.0;
        }
        if ((t & 63) == 0) sh.ex[1][t >> 6] = e;
    }
}

// E4M3 code product of one half row: thread (v, h) sums over channels
// 64h .. 64h+63 of row v, k side in fp64, q side in fp32 (E4M3 codes are not
// integers, so the digit product below does not apply).
template <int CODE, bool KS>
__device__ __forceinline__ void code_product_e4m3(const DecodeShared<CODE> &sh, int v, int h, double &zk,
                                                  float &zq) {
    const double *wkv = (const double *)sh.rv;
    const float *wqv = (const float *)(sh.rv + D * 8);
    double sk = 0.0;
    float sq = 0.0f;
#pragma unroll 1
    for (int m = 0; m < 4; ++m) {
        const int c = 4 * h + m;
        const uint4 z = lds_chunk<CODE>(sh.codes, v, c);
        const uint32_t zw[4] = {z.x, z.y, z.z, z.w};
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            const int c0 = 16 * c + 4 * p;         // channels c0 .. c0 + 3
            const float4 wq = *(const float4 *)&wqv[c0];
            const float f0 = e4m3_to_f<0>(zw[p]), f1 = e4m3_to_f<1>(zw[p]);
            const float f2 = e4m3_to_f<2>(zw[p]), f3 = e4m3_to_f<3>(zw[p]);
            sq = fmaf(f0, wq.x, sq);
            sq = fmaf(f1, wq.y, sq);
            sq = fmaf(f2, wq.z, sq);
            sq = fmaf(f3, wq.w, sq);
            if (KS) {
                const double2 wa = *(const double2 *)&wkv[c0], wb = *(const double2 *)&wkv[c0 + 2];
                sk = fma((double)f0, wa.x, sk);
                sk = fma((double)f1, wa.y, sk);
                sk = fma((double)f2, wb.x, sk);
                sk = fma((double)f3, wb.y, sk);
            }
        }
    }
    zk = sk;
    zq = sq;
}

// BF16-state code product of one half row: thread (v, h) sums over channels
// 64h .. 64h+63 of row v (eight 16-byte chunks of eight values), k side in
// fp64, q side in fp32.
template <int CODE, bool KS>
__device__ __forceinline__ void code_product_bf16(const DecodeShared<CODE> &sh, int v, int h, double &zk,
                                                  float &zq) {
    const double *wkv = (const double *)sh.rv;
    const float *wqv = (const float *)(sh.rv + D * 8);
    double sk = 0.0;
    float sq = 0.0f;
#pragma unroll 2
    for (int m = 0; m < 8; ++m) {
        const int c = 8 * h + m;
        const uint4 z = lds_chunk<CODE>(sh.codes, v, c);
        const uint32_t zw[4] = {z.x, z.y, z.z, z.w};
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            const int c0 = 8 * c + 2 * p;          // channels c0, c0 + 1
            const float f0 = __uint_as_float(zw[p] << 16), f1 = __uint_as_float(zw[p] & 0xFFFF0000u);
            const float2 wq = *(const float2 *)&wqv[c0];
            sq = fmaf(f0, wq.x, sq);
            sq = fmaf(f1, wq.y, sq);
            if (KS) {
                const double2 wk = *(const double2 *)&wkv[c0];
                sk = fma((double)f0, wk.x, sk);
                sk = fma((double)f1, wk.y, sk);
            }
        }
    }
    zk = sk;
    zq = sq;
}

typedef int v4i __attribute__((ext_vector_type(4)));

// Codes of channels c0 .. c0 + 15 of row v as sixteen int8 bytes, in channel
// order (c0 a multiple of 16).
template <int CODE>
__device__ __forceinline__ v4i codes_i8(const DecodeShared<CODE> &sh, int v, int c0) {
    if (CODE == 0) {
        const uint4 z = lds_chunk<CODE>(sh.codes, v, c0 >> 4);
        return v4i{(int)z.x, (int)z.y, (int)z.z, (int)z.w};
    }
    if (CODE == 2) {                                     // 32 codes per chunk
        const uint4 z = lds_chunk<CODE>(sh.codes, v, c0 >> 5);
        const uint32_t w0 = (c0 & 16) ? z.z : z.x, w1 = (c0 & 16) ? z.w : z.y;
        return v4i{(int)int4x4_to_bytes(w0, 0), (int)int4x4_to_bytes(w0, 1), (int)int4x4_to_bytes(w1, 0),
                   (int)int4x4_to_bytes(w1, 1)};
    }
    // 6-bit rows are not rotated; channels c0 .. c0 + 15 are 12 bytes at 3 c0 / 4
    const uint32_t *zr = (const uint32_t *)sh.codes + v * (Rows<CODE>::BYTES / 4) + 3 * (c0 >> 4);
    const uint32_t w0 = zr[0], w1 = zr[1], w2 = zr[2];
    return v4i{(int)int6x4_to_bytes(w0 & 0xFFFFFFu),
               (int)int6x4_to_bytes(__builtin_amdgcn_alignbit(w1, w0, 24) & 0xFFFFFFu),
               (int)int6x4_to_bytes(__builtin_amdgcn_alignbit(w2, w1, 16) & 0xFFFFFFu),
               (int)int6x4_to_bytes(w2 >> 8)};
}

// The same product on the vector ALU (a build-time alternative, selected by
// LQ_CODE_PRODUCT_VALU, kept to measure the matrix-core form against):
// thread (v, h) takes half h of code row v, one v_dot4_i32_i8 per 4 channels
// and digit, per exponent group g = (c >> 2) & 1; the digit sums are
// combined like the matrix-core ones.
#ifdef LQ_CODE_PRODUCT_VALU
template <int CODE, bool KS>
__device__ __forceinline__ void code_product_valu(const DecodeShared<CODE> &sh, int v, int h, double &zk,
                                                  float &zq) {
    constexpr int D0 = KS ? 0 : KDIG;            // first digit row used
    const uint32_t *dig = (const uint32_t *)sh.rv;   // [NDIG][D / 4] words
    int acc[NDIG][2];
#pragma unroll
    for (int d = 0; d < NDIG; ++d) acc[d][0] = acc[d][1] = 0;
    // the 4-channel words of this half row as int8 bytes: word i holds
    // channels 64h + 4i .. 64h + 4i + 3, exponent group i & 1
    auto dot_word = [&](uint32_t zb, int i) {
        const int g = i & 1;
#pragma unroll
        for (int d = D0; d < NDIG; ++d)
            acc[d][g] = __builtin_amdgcn_sdot4((int)zb, (int)dig[d * (D / 4) + 16 * h + i], acc[d][g], false);
    };
    if (CODE == 0) {
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            const uint4 z = lds_chunk<CODE>(sh.codes, v, 4 * h + m);
            dot_word(z.x, 4 * m + 0);
            dot_word(z.y, 4 * m + 1);
            dot_word(z.z, 4 * m + 2);
            dot_word(z.w, 4 * m + 3);
        }
    } else if (CODE == 2) {
        // 32 codes per chunk, two chunks per half row; each word holds 8 channels
#pragma unroll
        for (int m = 0; m < 2; ++m) {
            const uint4 z = lds_chunk<CODE>(sh.codes, v, 2 * h + m);
            const uint32_t zw[4] = {z.x, z.y, z.z, z.w};
#pragma unroll
            for (int p = 0; p < 4; ++p) {
                dot_word(int4x4_to_bytes(zw[p], 0), 8 * m + 2 * p);
                dot_word(int4x4_to_bytes(zw[p], 1), 8 * m + 2 * p + 1);
            }
        }
    } else {
        // 48 bytes per half row, four units of 12 bytes = 4 groups of 3 bytes
        const uint32_t *zr = (const uint32_t *)sh.codes + v * (Rows<CODE>::BYTES / 4) + 12 * h;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const uint32_t w0 = zr[3 * u], w1 = zr[3 * u + 1], w2 = zr[3 * u + 2];
            dot_word(int6x4_to_bytes(w0 & 0xFFFFFFu), 4 * u);
            dot_word(int6x4_to_bytes(__builtin_amdgcn_alignbit(w1, w0, 24) & 0xFFFFFFu), 4 * u + 1);
            dot_word(int6x4_to_bytes(__builtin_amdgcn_alignbit(w2, w1, 16) & 0xFFFFFFu), 4 * u + 2);
            dot_word(int6x4_to_bytes(w2 >> 8), 4 * u + 3);
        }
    }
    // sum_d acc_d 128^-d is exact in fp64 (|acc_d| < 2^19, 34 bits below)
    double sk = 0.0;
    if (KS) {
#pragma unroll
        for (int g = 0; g < 2; ++g) {
            double s = (double)acc[KDIG - 1][g];
#pragma unroll
            for (int d = KDIG - 2; d >= 0; --d) s = fma(s, 0x1p-7, (double)acc[d][g]);
            sk += __builtin_ldexp(s, sh.ex[0][g] - 6);
        }
    }
    float sq = 0.0f;
#pragma unroll
    for (int g = 0; g < 2; ++g) {
        float s = (float)acc[NDIG - 1][g];
#pragma unroll
        for (int d = NDIG - 2; d >= KDIG; --d) s = fmaf(s, 0x1p-7f, (float)acc[d][g]);
        sq += __builtin_ldexpf(s, sh.ex[1][g] - 6);
    }
    zk = sk;
    zq = sq;
}
#endif

// Integer code product of wave w's 32 rows on the integer matrix cores.  The
// products are exact: every code and every digit is an int8, and the int32
// sums are exact.  Column n of the 16 x 16 x 64 product is digit d = n & 7 of
// exponent group g = n >> 3 (the channels of the other group contribute 0),
// so one v_mfma_i32_16x16x64_i8 per 16 rows and 64 channels gives every
// digit sum at once.  The digit sums pass through the wave's own rows
// 4w+2 .. 4w+3 of the decay array (a 16 x 32 int32 transpose), and lane
// (side, r) combines row 32w + r: side 0 the k digits in fp64 (exactly, the
// sums being below 2^19 and 34 bits deep), side 1 the q digits in fp32.
template <int CODE, bool KS>
__device__ __forceinline__ void code_product_mfma(DecodeShared<CODE> &sh, int tid) {
    const int lane = tid & 63, w = tid >> 6, i16 = lane & 15, kb = lane >> 4;
    const int d = i16 & 7, g = i16 >> 3;
    v4i acc[2] = {v4i{0, 0, 0, 0}, v4i{0, 0, 0, 0}};
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        const int c0 = 64 * s + 16 * kb;                 // this lane's 16 channels
        const uint4 bq = *(const uint4 *)(sh.rv + d * D + c0);
        // words 0 and 2 hold exponent group 0 (channels c with (c >> 2) & 1 = 0)
        const v4i b = {g ? 0 : (int)bq.x, g ? (int)bq.y : 0, g ? 0 : (int)bq.z, g ? (int)bq.w : 0};
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
            acc[rb] = __builtin_amdgcn_mfma_i32_16x16x64_i8(codes_i8<CODE>(sh, 32 * w + 16 * rb + i16, c0), b,
                                                           acc[rb], 0, 0, 0);
    }
    // lane (kb, i16) holds rows 16 rb + 4 kb + 0..3 of column i16
    int *T = (int *)&sh.bp[4 * w + 2][0];                // [16 columns][32 rows]
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) *(v4i *)&T[i16 * 32 + 16 * rb + 4 * kb] = acc[rb];
    const int r = lane & 31, v = 32 * w + r;
    const float dl = sh.dlt[v];
    if (lane < 32) {
        if (KS) {
            double zk = 0.0;
#pragma unroll
            for (int gg = 0; gg < 2; ++gg) {
                double t = (double)T[(8 * gg + KDIG - 1) * 32 + r];
#pragma unroll
                for (int dd = KDIG - 2; dd >= 0; --dd) t = fma(t, 0x1p-7, (double)T[(8 * gg + dd) * 32 + r]);
                zk += __builtin_ldexp(t, sh.ex[0][gg] - 6);
            }
            sh.zk[POS(v)] = (double)dl * zk;
        }
    } else {
        float zq = 0.0f;
#pragma unroll
        for (int gg = 0; gg < 2; ++gg) {
            float t = (float)T[(8 * gg + NDIG - 1) * 32 + r];
#pragma unroll
            for (int dd = NDIG - 2; dd >= KDIG; --dd) t = fmaf(t, 0x1p-7f, (float)T[(8 * gg + dd) * 32 + r]);
            zq += __builtin_ldexpf(t, sh.ex[1][gg] - 6);
        }
        sh.zq[POS(v)] = dl * zq;
    }
}

// One token of one tile (the whole workgroup).  Returns the number of records
// the window held before this token, or -1 when the tile was left untouched
// (full or corrupt window).
template <int GATE, int CODE, int RULE>
__device__ __forceinline__ int decode_body(const DecodeArgs &a, DecodeShared<CODE> &sh, int tile) {
    constexpr bool KS = RULE != LQ_RULE_ADD;     // the k side is read (not for b_t = 0)
    constexpr int ZCH = DecodeShared<CODE>::ZCH;
    static_assert(ZCH % NT == 0, "whole chunks per thread");

    const int tid = threadIdx.x;
    // tile = b H_v + h_v and H_v = H_k group, so the key/query head row is
    // b H_k + h_v / group = tile / group, taken as a multiply by ceil(2^32 /
    // group) and a shift (exact while tiles * group < 2^32, which the launch
    // checks)
    const size_t tvec = (size_t)tile * D;

    const int l16 = tid & 15;            // 8-channel key segment / 8-value segment
    const int ts = tid >> 4;             // slot 0..15
    const size_t rbase = (size_t)tile * a.window;

    // ---- issue every load of the tile: rec_len (a scalar load, which the record
    // loads wait for), then what does not depend on it ---------------------------
    // (thread t < D: channel ch = CH(t))
    const int n = a.rec_len[tile];
    const int ch = CH(tid & (D - 1));
    // (beta, and alpha of the scalar gate, are per-tile scalars)
    float bt = a.beta[tile];
    float al = GATE ? 0.0f : a.alpha[tile];
    // The token pointers are pinned here so that their kernel-argument loads
    // join the others at the top instead of being sunk into the branch below
    // behind a second wait.
    // (cast back to the global address space: out of the asm they are generic
    // pointers, which would be read with flat loads)
    const float *pk = a.k, *pq = a.q, *pc = a.smooth, *pa = a.alpha, *pv = a.v;
    uint64_t kvm = a.kv_mul;
    asm volatile("" : "+s"(pk), "+s"(pq), "+s"(pc), "+s"(pa), "+s"(pv), "+s"(kvm));
    using gf = const __attribute__((address_space(1))) float;
    const size_t kvec = (size_t)(((uint64_t)(uint32_t)tile * kvm) >> 32) * D;
    const float *pb = a.b;
    if (RULE == LQ_RULE_GENERAL) asm volatile("" : "+s"(pb));
    float kx = 0.0f, qx = 0.0f, cs = 0.0f, vx = 0.0f, bx = 0.0f;
    if (tid < D) {
        kx = ((gf *)pk)[kvec + ch];
        qx = ((gf *)pq)[kvec + ch];
        cs = IsBF16<CODE>::value ? 1.0f : ((gf *)pc)[tvec + ch];
        if (GATE) al = ((gf *)pa)[tvec + ch];
        vx = ((gf *)pv)[tvec + ch];
        if (RULE == LQ_RULE_GENERAL) bx = ((gf *)pb)[tvec + ch];
    }
    {
        // LDS chunk P = NT m + 64 w + L (wave w's lanes fill 1 KiB) holds chunk
        // (P - zrot(v)) mod SEGS of row v = P / SEGS
        constexpr int SEGS = Rows<CODE>::SEGS;
        const uint4 *zt = (const uint4 *)(a.codes + (size_t)tile * D * Rows<CODE>::BYTES);
        const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
#pragma unroll
        for (int m = 0; m < ZCH / NT; ++m) {
            const int P = NT * m + tid, v = P / SEGS, c = P - v * SEGS;
            dma16(zt + v * SEGS + ((c - zrot<CODE>(v) + SEGS) % SEGS), lds_addr(&sh.codes[NT * m + 64 * w]));
        }
    }
    // per-row scales, wave 0 (the BF16 state has unit scales and does not read them)
    if (!IsBF16<CODE>::value && tid < D / 4) dma16(a.scale + tvec + 4 * tid, lds_addr(sh.dlt));
    uint4 ck = make_uint4(0, 0, 0, 0), cu = make_uint4(0, 0, 0, 0);
    // Compensator Token j is read by slot 15 - j: a pass's records are dealt
    // to the first slots, so at the early window positions the token readouts
    // run on waves that walk no records, beside the walk instead of after it
    const int cj = SLOTS - 1 - ts;
    if (cj < a.n_comp) {
        const size_t cb = ((size_t)tile * a.n_comp + cj) * D + 8 * l16;
        ck = *(const uint4 *)(a.comp_k + cb);
        cu = *(const uint4 *)(a.comp_u + cb);
    }
    if (n >= a.window || n < 0) {        // window buffer full (or corrupt): tile untouched
        if (tid == 0) atomicOr(a.err, n < 0 ? (int)LQ_DEVERR_BAD_REC_LEN : (int)LQ_DEVERR_WINDOW_FULL);
        if (tid < D) a.o[tvec + tid] = __builtin_nanf("");
        wait_vm_all();                   // no copy into LDS outlives the workgroup
        return -1;
    }
    RecRegs<GATE> R;
    constexpr int PER_SLOT = Pass<GATE>::PER_SLOT, PASS = Pass<GATE>::N;
    int hi = n, lo = n > PASS ? n - PASS : 0;
    int d = (hi - lo + SLOTS - 1) / SLOTS;
    load_records<GATE>(a, rbase, lo, hi, d, ts, l16, R);
    // Nothing that consumes the token inputs may be scheduled above this point:
    // a wait for one of them ahead of the code and record loads would delay
    // every load of the tile by a memory round trip.
    asm volatile("" : "+v"(kx), "+v"(qx), "+v"(cs), "+v"(al), "+v"(vx), "+v"(bt));
    if (RULE == LQ_RULE_GENERAL) asm volatile("" : "+v"(bx));

    // ---- token inputs, this token's record -------------------------------------
    // carry0: this token's FP16 decay (1 under the general rule), exact in fp32
    float carry0 = 1.0f;
    if (tid < D) {
        const uint16_t ah = f2h(al);
        // read vectors: k_t and q_t under the decay of this token (carry), or
        // b_t and d_t . q_t read against S_{i-1} (carry starts at 1)
        const bool gen = RULE == LQ_RULE_GENERAL;
        const float xk = gen ? bx : kx, xq = gen ? h2f(ah) * qx : qx;
        sh.x[0][tid] = xk;
        sh.x[1][tid] = xq;
        if (!gen) carry0 = h2f(ah);
        const size_t slot = rbase + n;
        if (GATE) a.rec_a[slot * D + ch] = ah;
        else if (tid == 0) a.rec_a[slot] = ah;
        const uint16_t tkh = f2h_mul(bt, kx);                // k~_t = fp16(fp32(beta_t k_t))
        a.rec_k[slot * D + ch] = tkh;
        const float kq = wave_sum(h2f(tkh) * qx);
        if ((tid & 63) == 0) sh.kq[tid >> 6] = kq;
        kx = xk;                                             // the base vectors read these
        qx = xq;
        // parked in LDS until the first scan (or the base vectors) reads it back,
        // so that no register holds it across the record loads
        sh.yk[tid] = (double)carry0;
    }

    // partial readouts of this thread's slot, k side and q side (defined after
    // the first scan, so that they hold no registers before it)
    double acc_k[8];
    float acc_q[8];

    // decay product of this slot's block, per channel of its segment (up to
    // three FP16 factors: exact in fp64)
    auto block_products = [&]() {
        if (GATE) {
            double bp[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) bp[j] = 1.0;
#pragma unroll
            for (int q = 0; q < PER_SLOT; ++q) {
                if (slot_record(lo, hi, d, ts, q) >= 0) {
                    const uint32_t w4[4] = {R.a[q].x, R.a[q].y, R.a[q].z, R.a[q].w};
#pragma unroll
                    for (int j = 0; j < 8; ++j) bp[j] *= h2d(w4[j >> 1], j & 1);
                }
            }
#pragma unroll
            for (int j = 0; j < 8; ++j) sh.bp[ts][SW(l16, j)] = bp[j];
        } else {
            double bp = 1.0;
#pragma unroll
            for (int q = 0; q < PER_SLOT; ++q)
                if (slot_record(lo, hi, d, ts, q) >= 0) bp *= (double)h2f((uint16_t)R.as[q]);
            if (l16 == 0) sh.bp[ts][0] = bp;
        }
    };
    // exclusive scan over the slots (threads t < D); after the last pass the
    // carry is Gamma_{1:i} and the base read vectors are written
    // carry: decay of every record newer than the current pass, channel ch
    // (the scalar gate keeps the same product in every thread below D)
    double carry = 1.0;
    auto scan = [&](bool first) {
        // slot 0 holds the newest block
        if (tid < D) {
            double c = first ? sh.yk[tid] : carry;
            // slot products read ahead of the chain (eight at a time), then
            // overwritten
#pragma unroll
            for (int s0 = 0; s0 < SLOTS; s0 += 8) {
                double bv[8];
#pragma unroll
                for (int s = 0; s < 8; ++s) bv[s] = sh.bp[s0 + s][GATE ? tid : 0];
#pragma unroll
                for (int s = 0; s < 8; ++s) {
                    if (GATE) sh.bp[s0 + s][tid] = c;
                    else if (tid == 0) sh.pre0[s0 + s] = c;
                    c *= bv[s];
                }
            }
            carry = c;
            if (lo == 0) {
                // (opaque copies: nothing derived from them is hoisted out of
                // the pass loop to be held across it)
                float k2 = kx, q2 = qx, c2 = cs;
                asm volatile("" : "+v"(k2), "+v"(q2), "+v"(c2));
                base_vectors<CODE, KS>(sh, carry, k2, q2, c2, tid);   // carry = Gamma_{1:i}
            }
        }
    };
    // the slot's records, newest first
    auto walk = [&]() {
        if (GATE) {
            // Y = Gamma_{j+1:i} . x for the slot's newest record, then older
            double Yk[8];
            float Yq[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const double P = sh.bp[ts][SW(l16, j)];
                Yk[j] = P * (double)sh.x[0][SW(l16, j)];
                Yq[j] = (float)P * sh.x[1][SW(l16, j)];
            }
#pragma unroll
            for (int q = 0; q < PER_SLOT; ++q) {
                if (slot_record(lo, hi, d, ts, q) < 0) break;    // uniform within the slot
                float kv[8], uv[8], av[8];
                unpack_h8(R.k[q], kv);
                unpack_h8(R.u[q], uv);
                unpack_h8(R.a[q], av);
                double sk = 0.0;
                float sq = 0.0f;
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    if (KS) sk = fma((double)kv[j], Yk[j], sk);
                    sq = fmaf(kv[j], Yq[j], sq);
                }
                if (KS) sk = row16_sum(sk);
                sq = row16_sum(sq);
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    if (KS) acc_k[j] = fma(sk, (double)uv[j], acc_k[j]);
                    acc_q[j] = fmaf(sq, uv[j], acc_q[j]);
                }
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    if (KS) Yk[j] *= (double)av[j];
                    Yq[j] *= av[j];
                }
            }
        } else {
            // scalar decay: one product per slot, applied to the two dot products
            double P = sh.pre0[ts];
            float xk[8], xq[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                xk[j] = sh.x[0][SW(l16, j)];
                xq[j] = sh.x[1][SW(l16, j)];
            }
#pragma unroll
            for (int q = 0; q < PER_SLOT; ++q) {
                if (slot_record(lo, hi, d, ts, q) < 0) break;    // uniform within the slot
                float kv[8], uv[8];
                unpack_h8(R.k[q], kv);
                unpack_h8(R.u[q], uv);
                double sk = 0.0;
                float sq = 0.0f;
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    if (KS) sk = fma((double)kv[j], (double)xk[j], sk);
                    sq = fmaf(kv[j], xq[j], sq);
                }
                if (KS) sk = row16_sum(sk) * P;
                sq = row16_sum(sq) * (float)P;
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    if (KS) acc_k[j] = fma(sk, (double)uv[j], acc_k[j]);
                    acc_q[j] = fmaf(sq, uv[j], acc_q[j]);
                }
                P *= (double)h2f((uint16_t)R.as[q]);
            }
        }
    };

    // ---- buffered records, newest first, up to PASS per pass ----------------------
    if (n > 0) {
        block_products();
        __syncthreads();
        scan(true);
        if (lo == 0) wait_vm_all();      // this wave's code copies have landed
        __syncthreads();
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            acc_k[j] = 0.0;
            acc_q[j] = 0.0f;
        }
        walk();
        while (lo > 0) {
            // older records: another pass.  Its first barrier orders this pass's
            // reads of the decay array before the next scan's writes.
            hi = lo;
            lo = hi > PASS ? hi - PASS : 0;
            d = (hi - lo + SLOTS - 1) / SLOTS;
            load_records<GATE>(a, rbase, lo, hi, d, ts, l16, R);
            block_products();
            __syncthreads();
            scan(false);
            if (lo == 0) wait_vm_all();
            __syncthreads();
            walk();
        }
    } else {
        // ---- no records: base read vectors only ----
        if (tid < D) base_vectors<CODE, KS>(sh, sh.yk[tid], kx, qx, cs, tid);
        wait_vm_all();
        __syncthreads();
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            acc_k[j] = 0.0;
            acc_q[j] = 0.0f;
        }
    }

    // ---- Compensator Tokens: token cj, same decay as the base -------------------
    if (cj < a.n_comp) {
        float kv[8], uv[8];
        unpack_h8(ck, kv);
        unpack_h8(cu, uv);
        double sk = 0.0;
        float sq = 0.0f;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            if (KS) sk = fma((double)kv[j], sh.yk[SW(l16, j)], sk);
            sq = fmaf(kv[j], sh.yq[SW(l16, j)], sq);
        }
        if (KS) sk = row16_sum(sk);
        sq = row16_sum(sq);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            if (KS) acc_k[j] = fma(sk, (double)uv[j], acc_k[j]);
            acc_q[j] = fmaf(sq, uv[j], acc_q[j]);
        }
    }

    // ---- quantized residual -------------------------------------------------------
    if (CODE == 1 || CODE == 4) {
        // thread (v, h) takes half h of code row v
        const int v = tid >> 1, h = tid & 1;
        double zk;
        float zq;
        if (CODE == 4) code_product_bf16<CODE, KS>(sh, v, h, zk, zq);
        else code_product_e4m3<CODE, KS>(sh, v, h, zk, zq);
        if (KS) zk += dpp<DPP_XOR1>(zk);
        zq += dpp<DPP_XOR1>(zq);
        if (h == 0) {
            const float dl = IsBF16<CODE>::value ? 1.0f : sh.dlt[v];
            if (KS) sh.zk[POS(v)] = (double)dl * zk;
            sh.zq[POS(v)] = dl * zq;
        }
    } else {
#ifdef LQ_CODE_PRODUCT_VALU
        const int v = tid >> 1, h = tid & 1;
        double zk;
        float zq;
        code_product_valu<CODE, KS>(sh, v, h, zk, zq);
        if (KS) zk += dpp<DPP_XOR1>(zk);
        zq += dpp<DPP_XOR1>(zq);
        if (h == 0) {
            if (KS) sh.zk[POS(v)] = (double)sh.dlt[v] * zk;
            sh.zq[POS(v)] = sh.dlt[v] * zq;
        }
#else
        code_product_mfma<CODE, KS>(sh, tid);
#endif
    }

    // sum over the wave's 4 slots in registers, then over the 4 waves in LDS:
    // lane (rho, l16) holds channels 8 l16 + 2 rho + e, e = 0, 1, stored at
    // [2 lane + e] of the wave's rows of the decay array (read only by its own
    // slots, all of which are past that read)
    {
        const int w = tid >> 6, lane = tid & 63;
        double *red_k = &sh.bp[4 * w][0];
        float *red_q = (float *)(red_k + D);
        if (KS) {
            double k0, k1;
            rows4_reduce_scatter(acc_k, k0, k1);
            red_k[2 * lane] = k0;
            red_k[2 * lane + 1] = k1;
        }
        float q0, q1;
        rows4_reduce_scatter(acc_q, q0, q1);
        *(float2 *)&red_q[2 * lane] = make_float2(q0, q1);
    }
    __syncthreads();

    // ---- combine, correction, output, record ------------------------------------
    if (tid < D) {
        // position t holds channel 8 (t & 15) + (t >> 4) = 8 l16 + 2 rho + e
        const int j = tid >> 4, e = j & 1;
        const int idx = 2 * (16 * (j >> 1) + (tid & 15)) + e;
        double ak = KS ? sh.zk[tid] : 0.0;
        float aq = sh.zq[tid];
#pragma unroll
        for (int w = 0; w < NT / 64; ++w) {
            const double *red_k = &sh.bp[4 * w][0];
            if (KS) ak += red_k[idx];
            aq += ((const float *)(red_k + D))[idx];
        }
        // u_t = fp16(v_t - A^T k_t) (general rule: v_t - S_{i-1}^T b_t), the
        // difference rounded to fp32 and then to FP16; the b_t = 0 rule reads
        // nothing (the k-side readouts above are then dead code and compiled out)
        const uint16_t uh = RULE == LQ_RULE_ADD ? f2h(vx) : d2h_via_f32((double)vx - ak);
        a.rec_u[(rbase + n) * D + ch] = uh;
        a.o[tvec + ch] = fmaf(h2f(uh), sh.kq[0] + sh.kq[1], aq);
        if (tid == 0) a.rec_len[tile] = n + 1;
    }
    return n;
}

inline DecodeArgs decode_args(const lq_dims &d, const StatePtrs &s, const TokenPtrs &t) {
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
    a.b = t.b;
    const uint64_t group = (uint64_t)(d.heads_v / d.heads_k);
    a.kv_mul = ((1ull << 32) + group - 1) / group;
    a.window = d.window;
    a.n_comp = d.n_comp;
    a.tiles = d.batch * d.heads_v;
    return a;
}

}  // namespace

}  // namespace lq
