// Device code of the whole-tile kernels (quantize, commit, dequantize), shared by
// their launches and by the decode step fused with the commit.
// Whole-tile kernels: quantize a given state, commit a window, dequantize.
//
// One 256-thread workgroup (4 waves) owns one 128 x 128 tile held in
// registers: thread (kb, vb) keeps the 8 x 8 block M[8kb .. 8kb+7][8vb .. 8vb+7]
// of the state in paper orientation (row = key channel).  kb is the lane's
// column inside its 16-lane DPP row, so sums over key channels stay inside a
// wave; sums over value channels go through LDS.  Three workgroups share a CU
// (168 VGPRs per lane, 50 KiB of LDS each): the 128 registers of the fp64
// block leave 40 for everything else, so the code below keeps few values
// live across phases (lane coordinates re-derived where used, records kept
// packed, the next pass's records copied straight into LDS).
//
//   commit   : reconstruct S_p = Gamma_{1:p}[C dequant(Z) + K~ U~^T]
//              + sum_j Gamma_{j+1:p} k~_j u_j^T  (Sec. 3.4 Eq. (smooth)),
//              then quantize it and reset the window (Sec. 3.3: the old
//              tokens are discarded and refitted);
//   quantize : load a given fp32 state and quantize it;
//   dequant  : reconstruct and write the fp32 state.
//
// Quantization (Sec. 3.3 Eq. (compensator-rank-r), Sec. 3.4, App. B.3): r
// Compensator Tokens fitted one after another by power iteration on the
// deflated residual (start: key-row l2 norms; each sweep y = M^T x, x = M y;
// the direction is normalised), each rounded to FP16 before it is
// subtracted; then the smoothing scales c_k = sqrt(max(mean_v |R_kv|, 1e-12)), the per-value-channel scale
// delta_v = max_k |R_kv / c_k| / qmax and the codes.
//
// Precision: the tile, the fit and the smoothing statistic are carried in
// fp64 (gfx950 runs fp64 FMA at the rate of unpacked fp32).  Each token is
// rounded to FP16 before it is deflated, so an fp32-level difference in the
// fit would flip a rounding and move every later token and the codes of whole
// rows; in fp64 the discrete decisions (FP16 tokens, fp32 scales, codes) are
// reproducible by any exact-enough implementation.  The code decision itself
// is taken in fp32 on the fp32-rounded residual.
#pragma once

#include "lq_device.hpp"
#include "lq_internal.hpp"

namespace lq {

namespace {

constexpr int TCH = 16;     // rank-one records staged per pass
constexpr int TT = 256;     // threads per tile
constexpr int NVB = 16;     // value blocks
constexpr int VPT = 8;      // value channels per thread

// Per-key-channel vectors in LDS are stored swizzled: channel 8kb+a sits at
// position 16a+kb, so the 16 lanes of a DPP row (kb = 0..15) touch 16
// consecutive 8-byte words and never share a bank.  A thread t < 128 that
// works on "position t" works on channel KCH(t).
__device__ __forceinline__ constexpr int KP(int kb, int a) { return 16 * a + kb; }
__device__ __forceinline__ constexpr int KCH(int t) { return 8 * (t & 15) + (t >> 4); }

// The 8 codes of row v (value channel), key channels 8kb..8kb+7: 8 bytes for
// the byte formats, 4 for INT4, 6 (three 16-bit words) for INT6, 16 (eight
// BF16 values) for the BF16 state.
template <int CODE> struct Codes8 { typedef uint2 type; };
template <> struct Codes8<4> { typedef uint4 type; };

template <int CODE>
__device__ __forceinline__ typename Codes8<CODE>::type load_codes8(const uint8_t *codes, int tile, int v, int kb) {
    constexpr int ROW = D * CodeFmt<CODE>::BITS / 8;
    const uint8_t *p = codes + ((size_t)tile * D + v) * ROW + kb * CodeFmt<CODE>::BITS;
    typename Codes8<CODE>::type w;
    if constexpr (CODE == 4) {
        w = *(const uint4 *)p;
    } else if constexpr (CODE <= 1) {
        w = *(const uint2 *)p;
    } else if constexpr (CODE == 2) {
        w = make_uint2(*(const uint32_t *)p, 0u);
    } else {
        const uint16_t *h = (const uint16_t *)p;
        w = make_uint2(h[0] | ((uint32_t)h[1] << 16), h[2]);
    }
    return w;
}

// Value a (0..7) of the 8 codes as a double (BF16 state: the value itself).
template <int CODE>
__device__ __forceinline__ double code8_value(const typename Codes8<CODE>::type &z, int a) {
    if constexpr (CODE == 4) {
        const uint32_t x = a < 2 ? z.x : a < 4 ? z.y : a < 6 ? z.z : z.w;
        return (double)bf2f((uint16_t)(x >> (16 * (a & 1))));
    } else {
        const uint32_t w[2] = {z.x, z.y};
        return (double)code_at<CODE>(w, a);
    }
}

template <int CODE>
__device__ __forceinline__ void store_codes8(uint8_t *codes, int tile, int v, int kb, uint2 w) {
    constexpr int ROW = D * CodeFmt<CODE>::BITS / 8;
    uint8_t *p = codes + ((size_t)tile * D + v) * ROW + kb * CodeFmt<CODE>::BITS;
    if (CODE <= 1) {
        *(uint2 *)p = w;
    } else if (CODE == 2) {
        *(uint32_t *)p = w.x;
    } else {
        uint16_t *h = (uint16_t *)p;
        h[0] = (uint16_t)w.x;
        h[1] = (uint16_t)(w.x >> 16);
        h[2] = (uint16_t)w.y;
    }
}

struct TileArgs {
    uint8_t *codes;
    float *scale;
    float *smooth;
    uint16_t *comp_k;
    uint16_t *comp_u;
    const uint16_t *rec_k;
    const uint16_t *rec_u;
    const uint16_t *rec_a;
    int32_t *rec_len;
    int32_t *err;
    const float *S_in;
    float *S_out;
    const int32_t *mask;
    int heads_v;
    int window;
    int n_comp;
    int power_iters;
    int smooth_on;
};

struct TileShared {
    union {
        double part[NVB][D];    // per-value-block partials of a sum over value channels
        double pre[TCH][D];     // record staging: decay of every newer record
    };
    double vec[D];          // broadcast vector
    double nrm[2];          // per-wave partial squared norms
    union {
        struct {            // reconstruction phase
            double key[TCH][D];     // staged record keys, decay folded in
            float val[TCH][D];      // staged record values
            float bp[TCH][D];       // decay of each staged record
            double tot[D];          // decay of a whole pass
        };
        double rowp[NVB][8 * 17];   // fit phase: per-row partials of sums over key blocks
    };
};

// Sums over value channels in two halves: each thread stores its value
// block's partial for channel 8kb+a as soon as it has it (put_part), then
// sum_parts adds the 16 value blocks; thread t < 128 gets channel KCH(t).
__device__ __forceinline__ void put_part(TileShared &sh, int a, double p, int kb, int vb) {
    sh.part[vb][KP(kb, a)] = p;
}
__device__ __forceinline__ double sum_parts(TileShared &sh) {
    __syncthreads();
    double s = 0.0;
    const int t = threadIdx.x;
    if (t < D) {
        double v[4] = {sh.part[0][t], sh.part[1][t], sh.part[2][t], sh.part[3][t]};
#pragma unroll
        for (int j = 4; j < NVB; ++j) v[j & 3] += sh.part[j][t];
        s = (v[0] + v[1]) + (v[2] + v[3]);
    }
    return s;
}

// Threads t < 128 publish x (channel KCH(t)) to sh.vec, which every thread
// then reads where it needs it (channel 8kb+a at KP(kb, a)); with_norm also
// returns the squared norm of the whole vector.  The barrier also ends every
// read of sh.part issued before the call.
__device__ __forceinline__ double publish(TileShared &sh, double x, bool with_norm) {
    const int t = threadIdx.x;
    if (t < D) {
        sh.vec[t] = x;
        if (with_norm) {
            const double s = wave_sum(x * x);
            if ((t & 63) == 0) sh.nrm[t >> 6] = s;
        }
    }
    __syncthreads();
    if (!with_norm) return 0.0;
    int z = 0;                           // a zero made where it is used (not held across the fit)
    asm volatile("v_mov_b32 %0, 0" : "=v"(z));
    return sh.nrm[z] + sh.nrm[z + 1];
}

// Sum v[b] (b = 0..7, this thread's value channels) over the 16 key blocks
// of its DPP row and return the 8 sums, times `scale`, in v.  The row's 16
// lanes belong to one wave, so a row-private LDS region needs no workgroup
// barrier: lane kb stores its partials at [b][kb] (rows of 17 words, so the
// words a read touches sit in distinct banks, and consecutive rows start 16
// banks apart); lane kb then sums channel kb & 7 over key blocks 8h .. 8h + 7
// (h = kb >> 3), adds lane kb ^ 8's half by a row rotation, and lanes kb < 8
// park the sums in the row's spare words, which every lane reads back.
__device__ __forceinline__ void row_sum8(TileShared &sh, double *v, int kb, int vb, double scale) {
    double *r = sh.rowp[vb];
#pragma unroll
    for (int b = 0; b < 8; ++b) r[17 * b + kb] = v[b];
    __builtin_amdgcn_wave_barrier();
    const int c = kb & 7, o = 17 * c + 8 * (kb >> 3);
    double t[4] = {r[o], r[o + 1], r[o + 2], r[o + 3]};
#pragma unroll
    for (int l = 4; l < 8; ++l) t[l & 3] += r[o + l];
    double h = (t[0] + t[1]) + (t[2] + t[3]);
    h += dpp<DPP_ROR8>(h);
    if (kb < 8) r[17 * c + 16] = h * scale;
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int b = 0; b < 8; ++b) v[b] = r[17 * b + 16];
    __builtin_amdgcn_wave_barrier();
}

// The whole-tile work of one workgroup.  p_given >= 0 (window commit only)
// is the number of buffered records, taken instead of the tile's rec_len and
// without the request mask: the decode step fused with the commit passes the
// count it has just made.
template <int GATE, int CODE, int MODE>
__device__ __forceinline__ void tile_body(const TileArgs &A, TileShared &sh, int tile, int p_given) {
    const int tid = threadIdx.x;
    int kb = tid & 15;                              // key block of 8 channels (DPP column)
    int vb = tid >> 4;                              // value block of VPT channels (0..15)
    // re-derive the lane coordinates from an opaque thread index, so that the
    // compiler recomputes the addresses built from them instead of holding
    // them in registers across phases
    auto refresh = [&]() {
        int t = (int)threadIdx.x;
        asm volatile("" : "+v"(t));
        kb = t & 15;
        vb = t >> 4;
    };
    const size_t tvec = (size_t)tile * D;
    const int r = A.n_comp;

    double m[8][VPT];                               // m[a][b] = M[8kb+a][VPT*vb+b]

    if (MODE == TILE_QUANTIZE) {
        const float *S = A.S_in + (size_t)tile * D * D;
#pragma unroll
        for (int b = 0; b < VPT; ++b) {
            const float4 *row = (const float4 *)(S + (size_t)(VPT * vb + b) * D + 8 * kb);
            const float4 lo = row[0], hi = row[1];
            m[0][b] = lo.x; m[1][b] = lo.y; m[2][b] = lo.z; m[3][b] = lo.w;
            m[4][b] = hi.x; m[5][b] = hi.y; m[6][b] = hi.z; m[7][b] = hi.w;
        }
    } else {
        // Every global load of the reconstruction is issued here, ahead of
        // its first use: rec_len, the codes and scales of this thread's
        // block, the compensators (one 16-byte segment per thread) and the
        // first pass of records.
        const int p = p_given >= 0 ? p_given : A.rec_len[tile];
        const int l16 = tid & 15, ts = tid >> 4;    // staging: segment, slot
        typename Codes8<CODE>::type zp[VPT];
#pragma unroll
        for (int b = 0; b < VPT; ++b) zp[b] = load_codes8<CODE>(A.codes, tile, VPT * vb + b, kb);
        // (the BF16 state has unit scales and no smoothing; its arrays are not read)
        const float4 one4 = make_float4(1.0f, 1.0f, 1.0f, 1.0f);
        const bool bf = IsBF16<CODE>::value;
        const float4 dl0 = bf ? one4 : *(const float4 *)(A.scale + tvec + VPT * vb);
        const float4 dl1 = bf ? one4 : *(const float4 *)(A.scale + tvec + VPT * vb + 4);
        const float4 c0 = bf ? one4 : *(const float4 *)(A.smooth + tvec + 8 * kb);
        const float4 c1 = bf ? one4 : *(const float4 *)(A.smooth + tvec + 8 * kb + 4);
        uint4 ck = make_uint4(0, 0, 0, 0), cu = ck;
        if (ts < r) {
            ck = *(const uint4 *)(A.comp_k + ((size_t)tile * r + ts) * D + 8 * l16);
            cu = *(const uint4 *)(A.comp_u + ((size_t)tile * r + ts) * D + 8 * l16);
        }
        if (p < 0 || p > A.window) {                                  // corrupt: tile untouched
            if (tid == 0) atomicOr(A.err, (int)LQ_DEVERR_BAD_REC_LEN);
            return;
        }
        if (MODE == TILE_COMMIT) {
            const int req = tile / A.heads_v;
            if (p == 0 || (p_given < 0 && A.mask && A.mask[req] == 0)) return;   // uniform: tile untouched
        }
        // records in passes of TCH, oldest pass first; slot ts of a pass takes
        // record lo+ts, lane l16 its 8-channel / 8-value segment.
        const size_t rbase = (size_t)tile * A.window;
        // the tile's record arrays as uniform bases, the lane's part as a 32-bit
        // offset (no per-lane 64-bit address is held across the passes)
        const uint16_t *rkb = A.rec_k + rbase * D, *rub = A.rec_u + rbase * D;
        const uint16_t *rab = A.rec_a + rbase * (GATE ? D : 1);
        // A pass's records are copied straight into LDS (the raw FP16 words,
        // in the record-staging area, which is idle while the previous pass's
        // records are applied), so no register holds them across a pass;
        // wave w copies records lo + 4w .. lo + 4w + 3.  The scalar gate's one
        // decay per record is loaded into a register.
        uint4 (*raw)[TCH][16] = (uint4 (*)[TCH][16])sh.pre;   // [key, corr, decay][record][segment]
        uint32_t ras = 0;
        auto load_pass = [&](int lo_, int hi_) {
            const int t = (int)threadIdx.x;
            const int w = __builtin_amdgcn_readfirstlane(t >> 6);
            const int rr = lo_ + 4 * w + ((t & 63) >> 4);
            const uint32_t off = (uint32_t)rr * D + 8u * (t & 15);
            if (rr < hi_) {
                dma16(rkb + off, lds_addr(&raw[0][4 * w][0]));
                dma16(rub + off, lds_addr(&raw[1][4 * w][0]));
                if (GATE) dma16(rab + off, lds_addr(&raw[2][4 * w][0]));
            }
            if (!GATE) {
                const int rs = lo_ + (t >> 4);
                if (rs < hi_) ras = rab[rs];
            }
        };
        if (p > 0) load_pass(0, p < TCH ? p : TCH);

        // window-start base C dequant(Z) (Sec. 3.4 Eq. (smooth))
        {
            const float dv[8] = {dl0.x, dl0.y, dl0.z, dl0.w, dl1.x, dl1.y, dl1.z, dl1.w};
            const float cv[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
#pragma unroll
            for (int b = 0; b < VPT; ++b) {
#pragma unroll
                for (int a = 0; a < 8; ++a) {
                    const double zf = code8_value<CODE>(zp[b], a);
                    m[a][b] = (double)cv[a] * (zf * (double)dv[b]);
                }
            }
        }
        // + its compensators K~ U~^T
        if (ts < r) {
            float kv[8], uv[8];
            unpack_h8(ck, kv);
            unpack_h8(cu, uv);
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                sh.key[ts][KP(l16, j)] = (double)kv[j];
                sh.val[ts][8 * l16 + j] = uv[j];
            }
        }
        __syncthreads();
#pragma unroll 1
        for (int h = 0; h < r; ++h) {
            refresh();
            double ud[VPT];
#pragma unroll
            for (int b = 0; b < VPT; ++b) ud[b] = (double)sh.val[h][VPT * vb + b];
#pragma unroll
            for (int a = 0; a < 8; ++a) {
                const double kd = sh.key[h][KP(kb, a)];
#pragma unroll
                for (int b = 0; b < VPT; ++b) m[a][b] = fma(kd, ud[b], m[a][b]);
            }
        }
        wait_vm_all();          // the first pass's records have landed in LDS
        __syncthreads();

        // Each pass: m <- Gamma_pass * m + sum_j Gamma_{j+1:hi} k~_j u_j^T, the
        // window recursion taken TCH records at a time; within the pass the
        // decay of every later record is an exclusive suffix product.
        for (int lo = 0; lo < p; lo += TCH) {
            refresh();
            const int hi = lo + TCH < p ? lo + TCH : p;
            const bool mine = lo + ts < hi;
            // the record (copied into LDS by this same thread) stays packed in
            // registers; halves are converted where stored
            uint4 rk = make_uint4(0, 0, 0, 0), ru = rk, ra = rk;
            if (mine) {
                rk = raw[0][ts][l16];
                ru = raw[1][ts][l16];
                if (GATE) ra = raw[2][ts][l16];
                else ra.x = ras;
            }
            auto h8 = [](const uint4 &w, int j) {
                const uint32_t x = j < 2 ? w.x : j < 4 ? w.y : j < 6 ? w.z : w.w;
                return h2f((uint16_t)(x >> (16 * (j & 1))));
            };
            if (GATE) {
#pragma unroll
                for (int j = 0; j < 8; ++j) sh.bp[ts][KP(l16, j)] = mine ? h8(ra, j) : 1.0f;
            } else if (l16 == 0) {
                sh.bp[ts][0] = mine ? h2f((uint16_t)ra.x) : 1.0f;
            }
            __syncthreads();
            if (tid < D) {
                const int ch = GATE ? tid : 0;
                double c = 1.0;
#pragma unroll
                for (int sl = TCH - 1; sl >= 0; --sl) {
                    const float bv = sh.bp[sl][ch];
                    if (GATE || tid == 0) sh.pre[sl][ch] = c;
                    c *= (double)bv;
                }
                if (GATE || tid == 0) sh.tot[ch] = c;
            }
            __syncthreads();
            if (mine) {
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const double P = sh.pre[ts][GATE ? KP(l16, j) : 0];
                    sh.key[ts][KP(l16, j)] = P * (double)h8(rk, j);
                    sh.val[ts][8 * l16 + j] = h8(ru, j);
                }
            } else {
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    sh.key[ts][KP(l16, j)] = 0.0;
                    sh.val[ts][8 * l16 + j] = 0.0f;
                }
            }
#pragma unroll
            for (int a = 0; a < 8; ++a) {
                const double T = sh.tot[GATE ? KP(kb, a) : 0];
#pragma unroll
                for (int b = 0; b < VPT; ++b) m[a][b] *= T;
            }
            __syncthreads();
            // sh.pre has been read by every thread: the next pass may land there
            if (hi < p) load_pass(hi, hi + TCH < p ? hi + TCH : p);
            // one record at a time, one key channel at a time, so only the
            // record's 8 values and one key are live beside the block
            const int nrec = hi - lo;
            // this lane's parts of the staging addresses, held across the pass
            refresh();
            const float *vrow = &sh.val[0][VPT * vb];
            const double *krow = &sh.key[0][kb];
#pragma unroll 1
            for (int j = 0; j < nrec; ++j) {
                double u0[VPT];
#pragma unroll
                for (int b = 0; b < VPT; ++b) u0[b] = (double)vrow[j * D + b];
#pragma unroll
                for (int a = 0; a < 8; ++a) {
                    const double k0 = krow[j * D + 16 * a];
#pragma unroll
                    for (int b = 0; b < VPT; ++b) m[a][b] = fma(k0, u0[b], m[a][b]);
                }
            }
            wait_vm_all();      // the next pass's records have landed in LDS
            __syncthreads();
        }

        if (MODE == TILE_DEQUANT) {
            float *S = A.S_out + (size_t)tile * D * D;
#pragma unroll
            for (int b = 0; b < VPT; ++b) {
                float4 *row = (float4 *)(S + (size_t)(VPT * vb + b) * D + 8 * kb);
                row[0] = make_float4((float)m[0][b], (float)m[1][b], (float)m[2][b], (float)m[3][b]);
                row[1] = make_float4((float)m[4][b], (float)m[5][b], (float)m[6][b], (float)m[7][b]);
            }
            return;
        }
    }

    // ------------------------------------------------------------------ quantize
    for (int h = 0; h < r; ++h) {
        refresh();
        // start vector: key-row l2 norms of the current residual
#pragma unroll
        for (int a = 0; a < 8; ++a) {
            double s = 0.0;
#pragma unroll
            for (int b = 0; b < VPT; ++b) s = fma(m[a][b], m[a][b], s);
            put_part(sh, a, s, kb, vb);
        }
        double x = sqrt(sum_parts(sh));
        double nrm = sqrt(publish(sh, x, true));
        bool ok = nrm > 0.0;
        // the published vector is read as sh.vec * xs: 1 / |x| after a
        // normalisation, 1 between sweeps
        double xs = ok ? 1.0 / nrm : 0.0;
        // Sweeps without per-sweep normalisation: each sweep is scaled by the
        // power of two sc ~ 1/|M|_F^2 (exact, so only the direction matters)
        // and the vector is normalised once after the last sweep.  A sweep
        // grows the norm by at most sc*sigma_1^2 < 2.
        const double sc = ok ? ldexp(1.0, -ilogb(nrm * nrm)) : 0.0;
        for (int it = 0; ok && it < A.power_iters; ++it) {
            refresh();
            // the eight reads of x issued together (one LDS round trip, not
            // one per pair of channels)
            double xv[8];
#pragma unroll
            for (int a = 0; a < 8; ++a) xv[a] = sh.vec[KP(kb, a)];
            asm volatile("" : "+v"(xv[0]), "+v"(xv[1]), "+v"(xv[2]), "+v"(xv[3]), "+v"(xv[4]), "+v"(xv[5]),
                         "+v"(xv[6]), "+v"(xv[7]));
            double y[VPT];
#pragma unroll
            for (int b = 0; b < VPT; ++b) y[b] = m[0][b] * xv[0];
#pragma unroll
            for (int a = 1; a < 8; ++a)
#pragma unroll
                for (int b = 0; b < VPT; ++b) y[b] = fma(m[a][b], xv[a], y[b]);
            row_sum8(sh, y, kb, vb, sc * xs);       // y_v = sc * sum_k M_kv (xs x_k)
#pragma unroll
            for (int a = 0; a < 8; ++a) {
                double s = 0.0;
#pragma unroll
                for (int b = 0; b < VPT; ++b) s = fma(m[a][b], y[b], s);
                put_part(sh, a, s, kb, vb);
            }
            x = sum_parts(sh);                      // x_k = sum_v M_kv y_v
            if (it + 1 < A.power_iters) {
                publish(sh, x, false);
                xs = 1.0;
            } else {
                nrm = sqrt(publish(sh, x, true));
                ok = nrm > 0.0;
                xs = ok ? 1.0 / nrm : 0.0;
            }
        }
        // the pair, FP16 bits packed two per word (zero when the residual is zero)
        // the pair, FP16 bits packed two per word, stored as soon as it is known
        // (zero when the residual is zero)
        refresh();
        if (ok) {
            float kf[8];
            uint32_t kw[4] = {0u, 0u, 0u, 0u};
#pragma unroll
            for (int a = 0; a < 8; ++a) {
                const uint16_t kh = d2h_via_f32(sh.vec[KP(kb, a)] * xs);   // rounded through fp32
                kw[a >> 1] |= (uint32_t)kh << (16 * (a & 1));
                kf[a] = h2f(kh);
            }
            if (vb == 0)
                *(uint4 *)(A.comp_k + ((size_t)tile * r + h) * D + 8 * kb) = make_uint4(kw[0], kw[1], kw[2], kw[3]);
            double us[VPT];
#pragma unroll
            for (int b = 0; b < VPT; ++b) {
                double s = 0.0;
#pragma unroll
                for (int a = 0; a < 8; ++a) s = fma(m[a][b], (double)kf[a], s);
                us[b] = s;
            }
            row_sum8(sh, us, kb, vb, 1.0);
            float uf[VPT];
            uint32_t uw[4] = {0u, 0u, 0u, 0u};
#pragma unroll
            for (int b = 0; b < VPT; ++b) {
                const uint16_t uh = d2h_via_f32(us[b]);      // u~_v = fp16(sum_k M_kv k~_k)
                uw[b >> 1] |= (uint32_t)uh << (16 * (b & 1));
                uf[b] = h2f(uh);
            }
            refresh();
            if (kb == 0)
                *(uint4 *)(A.comp_u + ((size_t)tile * r + h) * D + VPT * vb) = make_uint4(uw[0], uw[1], uw[2], uw[3]);
#pragma unroll
            for (int a = 0; a < 8; ++a)
#pragma unroll
                for (int b = 0; b < VPT; ++b) m[a][b] = fma(-(double)kf[a], (double)uf[b], m[a][b]);
        } else {
            if (vb == 0)
                *(uint4 *)(A.comp_k + ((size_t)tile * r + h) * D + 8 * kb) = make_uint4(0u, 0u, 0u, 0u);
            if (kb == 0)
                *(uint4 *)(A.comp_u + ((size_t)tile * r + h) * D + VPT * vb) = make_uint4(0u, 0u, 0u, 0u);
        }
    }

    if constexpr (IsBF16<CODE>::value) {
        // BF16 state: every entry rounded to nearest even through fp32 (the
        // window-end rounding of the per-window BF16 variant), unit scales
        refresh();
        constexpr int ROW = D * 2;
#pragma unroll
        for (int b = 0; b < VPT; ++b) {
            uint32_t w[4];
#pragma unroll
            for (int e = 0; e < 4; ++e)
                w[e] = (uint32_t)f2bf((float)m[2 * e][b]) | ((uint32_t)f2bf((float)m[2 * e + 1][b]) << 16);
            *(uint4 *)(A.codes + ((size_t)tile * D + VPT * vb + b) * ROW + 16 * kb) = make_uint4(w[0], w[1], w[2], w[3]);
        }
        if (tid < D) {
            A.smooth[tvec + tid] = 1.0f;
            A.scale[tvec + tid] = 1.0f;
        }
        if (tid == 0) A.rec_len[tile] = 0;
        return;
    }
    refresh();
    // residual smoothing over key rows: c_k = sqrt(max(mean_v |R_kv|, 1e-12)) in fp32
    {
#pragma unroll
        for (int a = 0; a < 8; ++a) {
            double s = 0.0;
#pragma unroll
            for (int b = 0; b < VPT; ++b) s += fabs(m[a][b]);
            put_part(sh, a, s, kb, vb);
        }
        const double s = sum_parts(sh);
        float c = 1.0f;
        if (A.smooth_on) c = (float)sqrt(fmax(s * (1.0 / (double)D), (double)1e-12f));
        if (tid < D) A.smooth[tvec + KCH(tid)] = c;
        publish(sh, (double)c, false);
    }
    refresh();
    // per-value-channel scale and codes, decided in fp32
    constexpr float QMAX = CodeFmt<CODE>::QMAX;
    float ic[8];
#pragma unroll
    for (int a = 0; a < 8; ++a) ic[a] = 1.0f / (float)sh.vec[KP(kb, a)];
#pragma unroll
    for (int b = 0; b < VPT; ++b) {
        float rc[8];
        float amax = 0.0f;
#pragma unroll
        for (int a = 0; a < 8; ++a) {
            rc[a] = (float)m[a][b] * ic[a];
            amax = fmaxf(amax, fabsf(rc[a]));
        }
        amax = row16_max(amax);
        const float dl = amax > 0.0f ? amax / QMAX : 0.0f;
        const float inv = amax > 0.0f ? QMAX / amax : 0.0f;
        uint32_t c8[8];
#pragma unroll
        for (int a = 0; a < 8; ++a) {
            if (CODE == 1) {
                const float t = fminf(fmaxf(rc[a] * inv, -QMAX), QMAX);
                c8[a] = f_to_e4m3(t);
            } else {
                const float t = fminf(fmaxf(rintf(rc[a] * inv), -QMAX), QMAX);
                c8[a] = (uint32_t)(int32_t)t;
            }
        }
        store_codes8<CODE>(A.codes, tile, VPT * vb + b, kb, encode8<CODE>(c8));
        if (kb == 0) A.scale[tvec + VPT * vb + b] = dl;
    }
    if (tid == 0) A.rec_len[tile] = 0;
}

inline TileArgs tile_args(const lq_dims &d, const StatePtrs &s, const float *S_in, float *S_out,
                          const int32_t *mask) {
    TileArgs a;
    a.codes = (uint8_t *)s.codes;
    a.scale = s.scale;
    a.smooth = s.smooth;
    a.comp_k = s.comp_k;
    a.comp_u = s.comp_u;
    a.rec_k = s.rec_k;
    a.rec_u = s.rec_u;
    a.rec_a = s.rec_a;
    a.rec_len = s.rec_len;
    a.err = s.err;
    a.S_in = S_in;
    a.S_out = S_out;
    a.mask = mask;
    a.heads_v = d.heads_v;
    a.window = d.window;
    a.n_comp = d.n_comp;
    a.power_iters = d.power_iters;
    a.smooth_on = d.smooth;
    return a;
}

}  // namespace

}  // namespace lq
