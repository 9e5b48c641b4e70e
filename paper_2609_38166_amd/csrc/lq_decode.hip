// Launch of the decode step: one workgroup per tile.
#include "lq_decode.hpp"

namespace lq {

namespace {

// Four workgroups per CU; the BF16 state's 32 KiB of codes per tile in LDS
// leave room for two.
template <int CODE> struct DecodeOcc { static constexpr int value = IsBF16<CODE>::value ? 2 : 4; };

template <int GATE, int CODE, int RULE>
__global__ __launch_bounds__(NT, DecodeOcc<CODE>::value) void decode_kernel(DecodeArgs a) {
    __shared__ DecodeShared<CODE> sh;
    decode_body<GATE, CODE, RULE>(a, sh, blockIdx.x);
}

template <int GATE, int CODE>
hipError_t launch(const DecodeArgs &args, int rule, hipStream_t st) {
    if (rule == LQ_RULE_ADD)
        hipLaunchKernelGGL((decode_kernel<GATE, CODE, LQ_RULE_ADD>), dim3(args.tiles), dim3(NT), 0, st, args);
    else if (rule == LQ_RULE_GENERAL)
        hipLaunchKernelGGL((decode_kernel<GATE, CODE, LQ_RULE_GENERAL>), dim3(args.tiles), dim3(NT), 0, st, args);
    else
        hipLaunchKernelGGL((decode_kernel<GATE, CODE, LQ_RULE_DELTA>), dim3(args.tiles), dim3(NT), 0, st, args);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_decode(const lq_dims &d, const StatePtrs &s, const TokenPtrs &t, hipStream_t st) {
    const DecodeArgs a = decode_args(d, s, t);
    if (d.gate == LQ_GATE_DIAG) {
        switch (d.code) {
            case LQ_CODE_E4M3: return launch<1, 1>(a, d.rule, st);
            case LQ_CODE_INT4: return launch<1, 2>(a, d.rule, st);
            case LQ_CODE_INT6: return launch<1, 3>(a, d.rule, st);
            case LQ_CODE_BF16: return launch<1, 4>(a, d.rule, st);
            default: return launch<1, 0>(a, d.rule, st);
        }
    }
    switch (d.code) {
        case LQ_CODE_E4M3: return launch<0, 1>(a, d.rule, st);
        case LQ_CODE_INT4: return launch<0, 2>(a, d.rule, st);
        case LQ_CODE_INT6: return launch<0, 3>(a, d.rule, st);
        case LQ_CODE_BF16: return launch<0, 4>(a, d.rule, st);
        default: return launch<0, 0>(a, d.rule, st);
    }
}

}  // namespace lq
