// Device helpers shared by the LeapQuant kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lq {

constexpr int D = 128;          // d_k = d_v
constexpr int NT = 256;         // threads per tile workgroup (4 waves)

// ---- DPP cross-lane moves (within a 16-lane row) ----------------------------
// quad_perm [1,0,3,2] / [2,3,0,1], row_ror:4 / row_ror:8, row_half_mirror.
enum : int {
    DPP_XOR1 = 0xB1,
    DPP_XOR2 = 0x4E,
    DPP_ROR4 = 0x124,
    DPP_ROR8 = 0x128,
    DPP_HALF_MIRROR = 0x141,
};

template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}

// Sum over the 16 lanes of a DPP row; every lane of the row receives the sum.
__device__ __forceinline__ float row16_sum(float x) {
    x += dpp<DPP_XOR1>(x);
    x += dpp<DPP_XOR2>(x);
    x += dpp<DPP_ROR4>(x);
    x += dpp<DPP_ROR8>(x);
    return x;
}

// Sum over an aligned group of 8 lanes; every lane of the group receives it.
__device__ __forceinline__ float row8_sum(float x) {
    x += dpp<DPP_XOR1>(x);
    x += dpp<DPP_XOR2>(x);
    x += dpp<DPP_HALF_MIRROR>(x);
    return x;
}

__device__ __forceinline__ float row16_max(float x) {
    x = fmaxf(x, dpp<DPP_XOR1>(x));
    x = fmaxf(x, dpp<DPP_XOR2>(x));
    x = fmaxf(x, dpp<DPP_ROR4>(x));
    x = fmaxf(x, dpp<DPP_ROR8>(x));
    return x;
}

// (every lane of the row has a source under these controls, so the moves need
// no old value: no register is cleared ahead of them)
template <int CTRL>
__device__ __forceinline__ double dpp(double x) {
    const int lo = __double2loint(x), hi = __double2hiint(x);
    return __hiloint2double(__builtin_amdgcn_mov_dpp(hi, CTRL, 0xF, 0xF, true),
                            __builtin_amdgcn_mov_dpp(lo, CTRL, 0xF, 0xF, true));
}

__device__ __forceinline__ double row16_sum(double x) {
    x += dpp<DPP_XOR1>(x);
    x += dpp<DPP_XOR2>(x);
    x += dpp<DPP_ROR4>(x);
    x += dpp<DPP_ROR8>(x);
    return x;
}

__device__ __forceinline__ double wave_sum(double x) {
    x = row16_sum(x);
    x += __shfl_xor(x, 16);
    x += __shfl_xor(x, 32);
    return x;
}

// Sum over the 64 lanes of a wave (result valid in every lane).
__device__ __forceinline__ float wave_sum(float x) {
    x = row16_sum(x);
    x += __shfl_xor(x, 16);
    x += __shfl_xor(x, 32);
    return x;
}

// ---- fp16 / bf16 / fp8 conversions ---------------------------------------------
__device__ __forceinline__ float h2f(uint16_t h) {
    return (float)__builtin_bit_cast(_Float16, h);
}
__device__ __forceinline__ uint16_t f2h(float f) {      // round to nearest even
    return __builtin_bit_cast(uint16_t, (_Float16)f);
}
__device__ __forceinline__ float f16_round(float f) { return h2f(f2h(f)); }

// fp16 of the fp32 product a * b: two roundings as written.  Without the empty
// asm the compiler emits one mixed-precision multiply (v_fma_mixlo_f16) that
// rounds the exact product straight to FP16, which decides some values
// differently.
__device__ __forceinline__ uint16_t f2h_mul(float a, float b) {
    float p = a * b;
    asm volatile("" : "+v"(p));
    return f2h(p);
}

// fp64 -> fp32 -> fp16, two roundings as written.  The empty asm keeps the
// compiler from fusing the two conversions into one direct fp64 -> fp16
// rounding, which decides ties differently.
__device__ __forceinline__ uint16_t d2h_via_f32(double d) {
    float f = (float)d;
    asm volatile("" : "+v"(f));
    return f2h(f);
}

__device__ __forceinline__ uint16_t f2bf(float f) {     // round to nearest even (finite f)
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}
__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// 8 packed fp16 values (one 16-byte load) to fp32.
__device__ __forceinline__ void unpack_h8(const uint4 &p, float *f) {
    const uint32_t w[4] = {p.x, p.y, p.z, p.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        f[2 * i] = h2f((uint16_t)(w[i] & 0xFFFFu));
        f[2 * i + 1] = h2f((uint16_t)(w[i] >> 16));
    }
}

// Byte `n` of a word as a signed int8 value, converted to fp32.
__device__ __forceinline__ float s8_to_f(uint32_t w, int n) {
    return (float)(int32_t)(int8_t)(uint8_t)(w >> (8 * n));
}

// OCP E4M3FN byte to fp32 (gfx950 converts the OCP format in hardware).
template <int SEL>
__device__ __forceinline__ float e4m3_to_f(uint32_t w) {
    return __builtin_amdgcn_cvt_f32_fp8((int)w, SEL);
}

// fp32 to OCP E4M3FN with round-to-nearest-even; |x| <= 448 on entry.
__device__ __forceinline__ uint8_t f_to_e4m3(float x) {
    return (uint8_t)(__builtin_amdgcn_cvt_pk_fp8_f32(x, x, 0, false) & 0xFF);
}

// ---- code formats -------------------------------------------------------------
// CODE 0: INT8 byte; 1: E4M3FN byte; 2: INT4, two codes per byte (even channel in
// the low nibble); 3: INT6, four codes per three bytes (channel 4i+q at bits
// 6q..6q+5 of the little-endian 24-bit group i).  Codes are two's complement.
template <int CODE> struct CodeFmt;
template <> struct CodeFmt<0> { static constexpr int BITS = 8; static constexpr float QMAX = 127.0f; };
template <> struct CodeFmt<1> { static constexpr int BITS = 8; static constexpr float QMAX = 448.0f; };
template <> struct CodeFmt<2> { static constexpr int BITS = 4; static constexpr float QMAX = 7.0f; };
template <> struct CodeFmt<3> { static constexpr int BITS = 6; static constexpr float QMAX = 31.0f; };
// CODE 4: the state itself in BF16 (the per-window BF16 variant): unit scales,
// no smoothing, no Compensator Tokens.
template <> struct CodeFmt<4> { static constexpr int BITS = 16; static constexpr float QMAX = 1.0f; };

// CODE 4 stores BF16 state values; every other code is an integer or an E4M3 byte.
template <int CODE> struct IsBF16 { static constexpr bool value = CODE == 4; };

// Signed field of `bits` bits at bit `off` of w (off + bits <= 32).
__device__ __forceinline__ int32_t sfield(uint32_t w, int off, int bits) {
    return (int32_t)(w << (32 - off - bits)) >> (32 - bits);
}

// Value of code j of a run of consecutive codes packed from bit 0 of the
// little-endian words w[] (j, CODE compile-time after unrolling).
template <int CODE>
__device__ __forceinline__ float code_at(const uint32_t *w, int j) {
    if (CODE == 0) return (float)sfield(w[j >> 2], 8 * (j & 3), 8);
    if (CODE == 1) {
        switch (j & 3) {
            case 0: return e4m3_to_f<0>(w[j >> 2]);
            case 1: return e4m3_to_f<1>(w[j >> 2]);
            case 2: return e4m3_to_f<2>(w[j >> 2]);
            default: return e4m3_to_f<3>(w[j >> 2]);
        }
    }
    if (CODE == 2) return (float)sfield(w[j >> 3], 4 * (j & 7), 4);
    const int bit = 6 * j, wi = bit >> 5, off = bit & 31;   // CODE == 3
    if (off + 6 <= 32) return (float)sfield(w[wi], off, 6);
    const uint32_t span = __builtin_amdgcn_alignbit(w[wi + 1], w[wi], off);
    return (float)sfield(span, 0, 6);
}

// 16 consecutive codes (the first 4 * BITS / 8 words of p) to fp32.
template <int CODE>
__device__ __forceinline__ void decode16(const uint4 &p, float *f) {
    const uint32_t w[4] = {p.x, p.y, p.z, p.w};
    if (CODE == 0) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            f[4 * i + 0] = s8_to_f(w[i], 0);
            f[4 * i + 1] = s8_to_f(w[i], 1);
            f[4 * i + 2] = s8_to_f(w[i], 2);
            f[4 * i + 3] = s8_to_f(w[i], 3);
        }
    } else {
#pragma unroll
        for (int j = 0; j < 16; ++j) f[j] = code_at<CODE>(w, j);
    }
}

// Pack 8 codes (integers, or E4M3 bytes) into the words of their format.
template <int CODE>
__device__ __forceinline__ uint2 encode8(const uint32_t *c) {
    if (CODE <= 1) {
        return make_uint2((c[0] & 0xFFu) | ((c[1] & 0xFFu) << 8) | ((c[2] & 0xFFu) << 16) | (c[3] << 24),
                          (c[4] & 0xFFu) | ((c[5] & 0xFFu) << 8) | ((c[6] & 0xFFu) << 16) | (c[7] << 24));
    }
    if (CODE == 2) {
        uint32_t x = 0;
#pragma unroll
        for (int a = 0; a < 8; ++a) x |= (c[a] & 0xFu) << (4 * a);
        return make_uint2(x, 0u);
    }
    uint64_t v = 0;                                          // CODE == 3: 48 bits
#pragma unroll
    for (int a = 0; a < 8; ++a) v |= (uint64_t)(c[a] & 0x3Fu) << (6 * a);
    return make_uint2((uint32_t)v, (uint32_t)(v >> 32));
}

// Non-temporal-free plain vector loads/stores through the vector memory path.
template <typename T>
__device__ __forceinline__ T ld(const T *p) { return *p; }

// LDS byte address of a __shared__ object.
__device__ __forceinline__ uint32_t lds_addr(const void *p) {
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void *)p;
}

// Copy 16 bytes per lane from global memory straight into LDS: lane L of the
// wave writes lds_base + 16 L (lds_base uniform).  Issued from asm so that the
// compiler does not treat it as an LDS store that every later LDS access must
// wait for; the reader waits with wait_vm_all() and a barrier.  M0 is set here
// and not declared clobbered (the compiler reserves it): the kernels that call
// this use M0 for nothing else, which their generated code shows.
__device__ __forceinline__ void dma16(const void *g, uint32_t lds_base) {
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" :: "v"(g), "s"(lds_base) : "memory");
}
__device__ __forceinline__ void wait_vm_all() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

}  // namespace lq
