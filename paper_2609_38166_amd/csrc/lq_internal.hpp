// Launchers shared between the C ABI layer and the kernel translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "leapquant.h"

namespace lq {

struct StatePtrs {
    void *codes;
    float *scale;
    float *smooth;
    uint16_t *comp_k;
    uint16_t *comp_u;
    uint16_t *rec_k;
    uint16_t *rec_u;
    uint16_t *rec_a;
    int32_t *rec_len;
    int32_t *err;
};

struct TokenPtrs {
    const float *q;
    const float *k;
    const float *v;
    const float *alpha;
    const float *beta;
    float *o;
    const float *b;     // read vectors [tiles][d_k] (general rule only, else null)
};

hipError_t launch_decode(const lq_dims &d, const StatePtrs &s, const TokenPtrs &t, hipStream_t st);

// decode step, then the window commit of every tile whose window it filled
hipError_t launch_decode_commit(const lq_dims &d, const StatePtrs &s, const TokenPtrs &t, hipStream_t st);

// mode: 0 = quantize given fp32 states, 1 = window commit, 2 = dequantize (read only)
enum TileMode { TILE_QUANTIZE = 0, TILE_COMMIT = 1, TILE_DEQUANT = 2 };
hipError_t launch_tile(const lq_dims &d, const StatePtrs &s, int mode, const float *S_in,
                       float *S_out, const int32_t *mask, hipStream_t st);

hipError_t launch_baseline(const lq_dims &d, void *S, int state_dtype, const TokenPtrs &t,
                           hipStream_t st);

}  // namespace lq
