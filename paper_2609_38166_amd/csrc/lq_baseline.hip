// Per-step baseline with a dense fp32 or bf16 state (Sec. 4.1 "Baselines"):
//   A = D S,  u = v - A^T k,  S = A + (beta k) u^T,  o = S^T q   (Sec. 3.1)
// (u = v for the b_t = 0 rows of the instance table, u = v - S^T b with the
// read vector given for the general form, App. A)
// One 256-thread workgroup per tile; 16 lanes cover one 128-entry state row
// S^T[v][:] (8 key channels each), so both matvecs are DPP row reductions.
// The state is read once and written once; arithmetic is fp32, a bf16 state is
// rounded to nearest even after the update and the output reads the rounded
// state.
#include "lq_device.hpp"
#include "lq_internal.hpp"

namespace lq {

namespace {

// State accesses.  The bf16 state is streamed with non-temporal loads and
// stores (measured 6% faster per step than plain accesses at 8192 tiles); the
// fp32 state is faster with plain ones (non-temporal stores cost it 1.6x).
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
template <bool NT>
__device__ __forceinline__ uint4 ld_state16(const uint4 *p) {
    if (NT) {
        const u32x4_t v = __builtin_nontemporal_load((const u32x4_t *)p);
        return make_uint4(v.x, v.y, v.z, v.w);
    }
    return *p;
}
template <bool NT>
__device__ __forceinline__ void st_state16(uint4 *p, uint4 w) {
    if (NT) {
        const u32x4_t v = {w.x, w.y, w.z, w.w};
        __builtin_nontemporal_store(v, (u32x4_t *)p);
    } else {
        *p = w;
    }
}


struct BaseArgs {
    void *S;
    const float *q;
    const float *k;
    const float *v;
    const float *alpha;
    const float *beta;
    float *o;
    const float *b;   // read vectors [tiles][D] (general rule)
    int heads_v;
    int group;
};

template <int GATE, int BF16, int RULE>
__global__ __launch_bounds__(NT) void baseline_kernel(BaseArgs a) {
    const int tile = blockIdx.x;
    const int tid = threadIdx.x;
    const int l16 = tid & 15;
    const int r0 = tid >> 4;                  // rows r0 + 16 m
    const int b = tile / a.heads_v, hv = tile - b * a.heads_v;
    const size_t kvec = ((size_t)b * (a.heads_v / a.group) + hv / a.group) * D + 8 * l16;
    const size_t tvec = (size_t)tile * D;

    float kx[8], qx[8], al[8], bk[8], bx[8];
    const float4 *k4 = (const float4 *)(a.k + kvec);
    const float4 *q4 = (const float4 *)(a.q + kvec);
    {
        const float4 k0 = k4[0], k1 = k4[1], q0 = q4[0], q1 = q4[1];
        kx[0] = k0.x; kx[1] = k0.y; kx[2] = k0.z; kx[3] = k0.w;
        kx[4] = k1.x; kx[5] = k1.y; kx[6] = k1.z; kx[7] = k1.w;
        qx[0] = q0.x; qx[1] = q0.y; qx[2] = q0.z; qx[3] = q0.w;
        qx[4] = q1.x; qx[5] = q1.y; qx[6] = q1.z; qx[7] = q1.w;
    }
    if (GATE) {
        const float4 *a4 = (const float4 *)(a.alpha + tvec + 8 * l16);
        const float4 a0 = a4[0], a1 = a4[1];
        al[0] = a0.x; al[1] = a0.y; al[2] = a0.z; al[3] = a0.w;
        al[4] = a1.x; al[5] = a1.y; al[6] = a1.z; al[7] = a1.w;
    } else {
        const float s = a.alpha[tile];
#pragma unroll
        for (int j = 0; j < 8; ++j) al[j] = s;
    }
    if (RULE == LQ_RULE_GENERAL) {
        const float4 *b4 = (const float4 *)(a.b + tvec + 8 * l16);
        const float4 b0 = b4[0], b1 = b4[1];
        bx[0] = b0.x; bx[1] = b0.y; bx[2] = b0.z; bx[3] = b0.w;
        bx[4] = b1.x; bx[5] = b1.y; bx[6] = b1.z; bx[7] = b1.w;
    }
    const float beta = a.beta[tile];
#pragma unroll
    for (int j = 0; j < 8; ++j) bk[j] = beta * kx[j];

    float s[8][8];
    if (BF16) {
        const uint16_t *St = (const uint16_t *)a.S + (size_t)tile * D * D;
#pragma unroll
        for (int m = 0; m < 8; ++m) {
            const uint4 p = ld_state16<BF16 != 0>((const uint4 *)(St + (size_t)(r0 + 16 * m) * D + 8 * l16));
            const uint32_t w[4] = {p.x, p.y, p.z, p.w};
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                s[m][2 * i] = bf2f((uint16_t)(w[i] & 0xFFFFu));
                s[m][2 * i + 1] = bf2f((uint16_t)(w[i] >> 16));
            }
        }
    } else {
        const float *St = (const float *)a.S + (size_t)tile * D * D;
#pragma unroll
        for (int m = 0; m < 8; ++m) {
            const uint4 *row = (const uint4 *)(St + (size_t)(r0 + 16 * m) * D + 8 * l16);
            const uint4 lo_ = ld_state16<BF16 != 0>(row), hi_ = ld_state16<BF16 != 0>(row + 1);
            const float4 lo = make_float4(__uint_as_float(lo_.x), __uint_as_float(lo_.y), __uint_as_float(lo_.z), __uint_as_float(lo_.w));
            const float4 hi = make_float4(__uint_as_float(hi_.x), __uint_as_float(hi_.y), __uint_as_float(hi_.z), __uint_as_float(hi_.w));
            s[m][0] = lo.x; s[m][1] = lo.y; s[m][2] = lo.z; s[m][3] = lo.w;
            s[m][4] = hi.x; s[m][5] = hi.y; s[m][6] = hi.z; s[m][7] = hi.w;
        }
    }

#pragma unroll
    for (int m = 0; m < 8; ++m) {
        const int vrow = r0 + 16 * m;
        float p = 0.0f;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            if (RULE == LQ_RULE_GENERAL) p = fmaf(s[m][j], bx[j], p);   // S^T b (before the decay)
            s[m][j] *= al[j];                           // A = D S
            if (RULE == LQ_RULE_DELTA) p = fmaf(s[m][j], kx[j], p);     // A^T k
        }
        const float u = RULE == LQ_RULE_ADD ? a.v[tvec + vrow]
                                            : a.v[tvec + vrow] - row16_sum(p);  // u = v - A^T k (S^T b)
        float po = 0.0f;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            float x = fmaf(bk[j], u, s[m][j]);          // S = A + (beta k) u^T
            if (BF16) x = bf2f(f2bf(x));
            s[m][j] = x;
            po = fmaf(x, qx[j], po);
        }
        po = row16_sum(po);
        if (l16 == 0) a.o[tvec + vrow] = po;             // o = S^T q
    }

    if (BF16) {
        uint16_t *St = (uint16_t *)a.S + (size_t)tile * D * D;
#pragma unroll
        for (int m = 0; m < 8; ++m) {
            uint4 w;
            w.x = f2bf(s[m][0]) | ((uint32_t)f2bf(s[m][1]) << 16);
            w.y = f2bf(s[m][2]) | ((uint32_t)f2bf(s[m][3]) << 16);
            w.z = f2bf(s[m][4]) | ((uint32_t)f2bf(s[m][5]) << 16);
            w.w = f2bf(s[m][6]) | ((uint32_t)f2bf(s[m][7]) << 16);
            st_state16<BF16 != 0>((uint4 *)(St + (size_t)(r0 + 16 * m) * D + 8 * l16), w);
        }
    } else {
        float *St = (float *)a.S + (size_t)tile * D * D;
#pragma unroll
        for (int m = 0; m < 8; ++m) {
            uint4 *row = (uint4 *)(St + (size_t)(r0 + 16 * m) * D + 8 * l16);
            st_state16<BF16 != 0>(row, make_uint4(__float_as_uint(s[m][0]), __float_as_uint(s[m][1]), __float_as_uint(s[m][2]), __float_as_uint(s[m][3])));
            st_state16<BF16 != 0>(row + 1, make_uint4(__float_as_uint(s[m][4]), __float_as_uint(s[m][5]), __float_as_uint(s[m][6]), __float_as_uint(s[m][7])));
        }
    }
}

template <int GATE, int BF16>
hipError_t launch(const BaseArgs &a, int tiles, int rule, hipStream_t st) {
    if (rule == LQ_RULE_ADD)
        hipLaunchKernelGGL((baseline_kernel<GATE, BF16, LQ_RULE_ADD>), dim3(tiles), dim3(NT), 0, st, a);
    else if (rule == LQ_RULE_GENERAL)
        hipLaunchKernelGGL((baseline_kernel<GATE, BF16, LQ_RULE_GENERAL>), dim3(tiles), dim3(NT), 0, st, a);
    else
        hipLaunchKernelGGL((baseline_kernel<GATE, BF16, LQ_RULE_DELTA>), dim3(tiles), dim3(NT), 0, st, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_baseline(const lq_dims &d, void *S, int state_dtype, const TokenPtrs &t,
                           hipStream_t st) {
    BaseArgs a;
    a.S = S;
    a.q = t.q;
    a.k = t.k;
    a.v = t.v;
    a.alpha = t.alpha;
    a.beta = t.beta;
    a.o = t.o;
    a.b = t.b;
    a.heads_v = d.heads_v;
    a.group = d.heads_v / d.heads_k;
    const int tiles = d.batch * d.heads_v;
    const bool bf = state_dtype == LQ_STATE_BF16;
    if (d.gate == LQ_GATE_DIAG)
        return bf ? launch<1, 1>(a, tiles, d.rule, st) : launch<1, 0>(a, tiles, d.rule, st);
    return bf ? launch<0, 1>(a, tiles, d.rule, st) : launch<0, 0>(a, tiles, d.rule, st);
}

}  // namespace lq
