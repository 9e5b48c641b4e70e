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

template <int CTRL>
__device__ __forceinline__ double dpp(double x) {
    const int lo = __double2loint(x), hi = __double2hiint(x);
    return __hiloint2double(__builtin_amdgcn_update_dpp(0, hi, CTRL, 0xF, 0xF, false),
                            __builtin_amdgcn_update_dpp(0, lo, CTRL, 0xF, 0xF, false));
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

template <int CODE>
__device__ __forceinline__ void decode16(const uint4 &p, float *f) {
    const uint32_t w[4] = {p.x, p.y, p.z, p.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        if (CODE == 0) {
            f[4 * i + 0] = s8_to_f(w[i], 0);
            f[4 * i + 1] = s8_to_f(w[i], 1);
            f[4 * i + 2] = s8_to_f(w[i], 2);
            f[4 * i + 3] = s8_to_f(w[i], 3);
        } else {
            f[4 * i + 0] = e4m3_to_f<0>(w[i]);
            f[4 * i + 1] = e4m3_to_f<1>(w[i]);
            f[4 * i + 2] = e4m3_to_f<2>(w[i]);
            f[4 * i + 3] = e4m3_to_f<3>(w[i]);
        }
    }
}

template <int CODE>
__device__ __forceinline__ void decode8(const uint2 &p, float *f) {
    const uint32_t w[2] = {p.x, p.y};
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        if (CODE == 0) {
            f[4 * i + 0] = s8_to_f(w[i], 0);
            f[4 * i + 1] = s8_to_f(w[i], 1);
            f[4 * i + 2] = s8_to_f(w[i], 2);
            f[4 * i + 3] = s8_to_f(w[i], 3);
        } else {
            f[4 * i + 0] = e4m3_to_f<0>(w[i]);
            f[4 * i + 1] = e4m3_to_f<1>(w[i]);
            f[4 * i + 2] = e4m3_to_f<2>(w[i]);
            f[4 * i + 3] = e4m3_to_f<3>(w[i]);
        }
    }
}

// Non-temporal-free plain vector loads/stores through the vector memory path.
template <typename T>
__device__ __forceinline__ T ld(const T *p) { return *p; }

}  // namespace lq
