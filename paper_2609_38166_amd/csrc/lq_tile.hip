// Launches of the whole-tile kernels: quantize a given state, commit a window,
// dequantize.
#include "lq_tile.hpp"

namespace lq {

namespace {

template <int GATE, int CODE, int MODE>
__global__ __launch_bounds__(TT, 3) void tile_kernel(TileArgs A) {
    __shared__ TileShared sh;
    tile_body<GATE, CODE, MODE>(A, sh, blockIdx.x, -1);
}

template <int GATE, int CODE, int MODE>
hipError_t launch3(const TileArgs &a, int tiles, hipStream_t st) {
    hipLaunchKernelGGL((tile_kernel<GATE, CODE, MODE>), dim3(tiles), dim3(TT), 0, st, a);
    return hipGetLastError();
}

template <int GATE, int CODE>
hipError_t launch2(const TileArgs &a, int tiles, int mode, hipStream_t st) {
    switch (mode) {
        case TILE_QUANTIZE: return launch3<GATE, CODE, TILE_QUANTIZE>(a, tiles, st);
        case TILE_COMMIT: return launch3<GATE, CODE, TILE_COMMIT>(a, tiles, st);
        default: return launch3<GATE, CODE, TILE_DEQUANT>(a, tiles, st);
    }
}

}  // namespace

hipError_t launch_tile(const lq_dims &d, const StatePtrs &s, int mode, const float *S_in,
                       float *S_out, const int32_t *mask, hipStream_t st) {
    const TileArgs a = tile_args(d, s, S_in, S_out, mask);
    const int tiles = d.batch * d.heads_v;
    if (d.gate == LQ_GATE_DIAG) {
        switch (d.code) {
            case LQ_CODE_E4M3: return launch2<1, 1>(a, tiles, mode, st);
            case LQ_CODE_INT4: return launch2<1, 2>(a, tiles, mode, st);
            case LQ_CODE_INT6: return launch2<1, 3>(a, tiles, mode, st);
            case LQ_CODE_BF16: return launch2<1, 4>(a, tiles, mode, st);
            default: return launch2<1, 0>(a, tiles, mode, st);
        }
    }
    switch (d.code) {
        case LQ_CODE_E4M3: return launch2<0, 1>(a, tiles, mode, st);
        case LQ_CODE_INT4: return launch2<0, 2>(a, tiles, mode, st);
        case LQ_CODE_INT6: return launch2<0, 3>(a, tiles, mode, st);
        case LQ_CODE_BF16: return launch2<0, 4>(a, tiles, mode, st);
        default: return launch2<0, 0>(a, tiles, mode, st);
    }
}

}  // namespace lq
