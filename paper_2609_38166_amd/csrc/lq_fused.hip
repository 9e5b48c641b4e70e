// Decode step fused with the window-end commit.
//
// The paper refits a tile whose window ends inside the decode launch, where
// the refit's arithmetic runs beside the other tiles' state reads (Sec. 3.3,
// Sec. 4.1 "Implementation").  Here one workgroup per tile runs the decode
// step of lq_decode.hpp and, when this token filled the tile's window
// (rec_len reached W), the window commit of lq_tile.hpp for the same tile in
// the same launch: reconstruction from the base and all W records (the one
// just written included), refit, smoothing, requantization, rec_len := 0.
// Requests may sit at different window positions, so one launch can hold
// decode-only and decode-and-commit tiles (staggered windows, where every step
// commits the group of requests whose window ends there).
//
// Resources are those of the larger body: the commit holds a 128 x 128 fp64
// tile in registers, so the kernel runs three workgroups per CU (the plain
// decode runs four); with the BF16 state, whose decode stages 32 KiB of state
// per tile in LDS, two.
#include "lq_decode.hpp"
#include "lq_tile.hpp"

namespace lq {

namespace {

template <int CODE>
union FusedShared {
    DecodeShared<CODE> d;
    TileShared t;
};

template <int CODE> struct FusedOcc { static constexpr int value = IsBF16<CODE>::value ? 2 : 3; };

template <int GATE, int CODE, int RULE>
__global__ __launch_bounds__(NT, FusedOcc<CODE>::value) void decode_commit_kernel(DecodeArgs a, TileArgs c) {
    __shared__ FusedShared<CODE> sh;
    const int tile = blockIdx.x;
    const int n = decode_body<GATE, CODE, RULE>(a, sh.d, tile);
    if (n + 1 != a.window) return;       // uniform: the window is not full (or the tile untouched)
    // The token's record and rec_len are stored; make them visible to the
    // commit's loads (device-scope release and acquire, which also drops any
    // cached copy) and end every use of the decode's LDS.
    __threadfence();
    __syncthreads();
    tile_body<GATE, CODE, TILE_COMMIT>(c, sh.t, tile, n + 1);
}

template <int GATE, int CODE>
hipError_t launch(const DecodeArgs &a, const TileArgs &c, int rule, hipStream_t st) {
    if (rule == LQ_RULE_ADD)
        hipLaunchKernelGGL((decode_commit_kernel<GATE, CODE, LQ_RULE_ADD>), dim3(a.tiles), dim3(NT), 0, st, a, c);
    else
        hipLaunchKernelGGL((decode_commit_kernel<GATE, CODE, LQ_RULE_DELTA>), dim3(a.tiles), dim3(NT), 0, st, a, c);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_decode_commit(const lq_dims &d, const StatePtrs &s, const TokenPtrs &t, hipStream_t st) {
    const DecodeArgs a = decode_args(d, s, t);
    const TileArgs c = tile_args(d, s, nullptr, nullptr, nullptr);
    if (d.gate == LQ_GATE_DIAG) {
        switch (d.code) {
            case LQ_CODE_E4M3: return launch<1, 1>(a, c, d.rule, st);
            case LQ_CODE_INT4: return launch<1, 2>(a, c, d.rule, st);
            case LQ_CODE_INT6: return launch<1, 3>(a, c, d.rule, st);
            case LQ_CODE_BF16: return launch<1, 4>(a, c, d.rule, st);
            default: return launch<1, 0>(a, c, d.rule, st);
        }
    }
    switch (d.code) {
        case LQ_CODE_E4M3: return launch<0, 1>(a, c, d.rule, st);
        case LQ_CODE_INT4: return launch<0, 2>(a, c, d.rule, st);
        case LQ_CODE_INT6: return launch<0, 3>(a, c, d.rule, st);
        case LQ_CODE_BF16: return launch<0, 4>(a, c, d.rule, st);
        default: return launch<0, 0>(a, c, d.rule, st);
    }
}

}  // namespace lq
