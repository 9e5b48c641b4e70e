// Memory and undefined-behaviour check of the C ABI's host code (test
// infrastructure).
//
// tests/test_sanitizers.py compiles the library's host-side layer
// (lq_api.hip, host pass only) with AddressSanitizer and
// UndefinedBehaviorSanitizer and links it with this driver, which stands in
// for the kernel launchers: each stub records that it was reached and returns
// the status the driver chooses.  Every entry point is then called with valid
// arguments (the stub must be reached with the caller's sizes) and with each
// kind of invalid argument (NULL, misaligned, out-of-range enums and sizes,
// overflowing shapes), which must be rejected before any launch.  No device
// memory is touched: pointers are plain addresses that are never dereferenced.
#include <cstdio>
#include <cstring>
#include <string>
#include <thread>

#include "leapquant.h"
#include "lq_internal.hpp"

namespace {
int launches = 0;
hipError_t next_status = hipSuccess;
lq_dims last_dims;
}  // namespace

namespace lq {
hipError_t launch_decode(const lq_dims &d, const StatePtrs &, const TokenPtrs &, hipStream_t) {
    ++launches;
    last_dims = d;
    return next_status;
}
hipError_t launch_decode_commit(const lq_dims &d, const StatePtrs &, const TokenPtrs &, hipStream_t) {
    ++launches;
    last_dims = d;
    return next_status;
}
hipError_t launch_tile(const lq_dims &d, const StatePtrs &, int, const float *, float *, const int32_t *,
                       hipStream_t) {
    ++launches;
    last_dims = d;
    return next_status;
}
hipError_t launch_baseline(const lq_dims &d, void *, int, const TokenPtrs &, hipStream_t) {
    ++launches;
    last_dims = d;
    return next_status;
}
}  // namespace lq

namespace {

int failures = 0;

void expect(bool ok, const char *what, int line) {
    if (!ok) {
        std::fprintf(stderr, "line %d: %s\n", line, what);
        ++failures;
    }
}
#define EXPECT(c) expect((c), #c, __LINE__)

char *P(uintptr_t a) { return reinterpret_cast<char *>(a); }

lq_dims dims(int gate = LQ_GATE_SCALAR, int code = LQ_CODE_INT8, int rule = LQ_RULE_DELTA) {
    lq_dims d;
    std::memset(&d, 0, sizeof(d));
    d.batch = 3;
    d.heads_v = 4;
    d.heads_k = 2;
    d.d_k = 128;
    d.d_v = 128;
    d.window = 16;
    d.n_comp = code == LQ_CODE_BF16 ? 0 : 4;
    d.power_iters = 4;
    d.gate = gate;
    d.code = code;
    d.smooth = code == LQ_CODE_BF16 ? 0 : 1;
    d.rule = rule;
    return d;
}

lq_state state() {
    lq_state s;
    uintptr_t base = 0x100000;
    void **f[] = {&s.codes, (void **)&s.scale, (void **)&s.smooth, (void **)&s.comp_k, (void **)&s.comp_u,
                  (void **)&s.rec_k, (void **)&s.rec_u, (void **)&s.rec_a, (void **)&s.rec_len, (void **)&s.err};
    for (void **p : f) {
        *p = P(base);
        base += 0x10000;
    }
    return s;
}

// one call of every launching entry point with the given arguments; returns
// the statuses in a fixed order
struct Tok {
    float *q = (float *)P(0x900000), *k = (float *)P(0x910000), *v = (float *)P(0x920000);
    float *a = (float *)P(0x930000), *b = (float *)P(0x940000), *o = (float *)P(0x950000);
    float *rv = (float *)P(0x960000);
};

int call(int which, const lq_dims *d, lq_state *s, const Tok &t) {
    float *S = (float *)P(0xA00000);
    switch (which) {
        case 0: return leapquant_quantize_state(d, S, s, nullptr);
        case 1: return leapquant_decode_step(d, s, t.q, t.k, t.v, t.a, t.b, t.o, nullptr);
        case 2: return leapquant_decode_step_commit(d, s, t.q, t.k, t.v, t.a, t.b, t.o, nullptr);
        case 3: return leapquant_decode_step_general(d, s, t.q, t.k, t.rv, t.v, t.a, t.b, t.o, nullptr);
        case 4: return leapquant_window_commit(d, s, nullptr, nullptr);
        case 5: return leapquant_baseline_step(d, S, LQ_STATE_F32, t.q, t.k, t.v, t.a, t.b, t.o, nullptr);
        case 6: return leapquant_baseline_step_general(d, S, LQ_STATE_BF16, t.q, t.k, t.rv, t.v, t.a, t.b,
                                                       t.o, nullptr);
        default: return leapquant_dequantize_state(d, s, S, nullptr);
    }
}
constexpr int N_CALLS = 8;
bool general_only(int which) { return which == 3 || which == 6; }
bool needs_read(int which) { return which == 1 || which == 2 || which == 5; }

// every call rejects `d` with status `want`, before any launch
void all_reject(const lq_dims &d, int want, int line) {
    Tok t;
    for (int w = 0; w < N_CALLS; ++w) {
        lq_state s = state();
        const int before = launches;
        const int got = call(w, &d, &s, t);
        if (got != want || launches != before) {
            std::fprintf(stderr, "line %d: call %d returned %d (want %d), launches %d\n", line, w, got, want,
                         launches - before);
            ++failures;
        }
    }
}

void test_valid_calls_launch() {
    for (int gate = 0; gate < 2; ++gate)
        for (int code = 0; code < 5; ++code)
            for (int rule = 0; rule < 3; ++rule) {
                lq_dims d = dims(gate, code, rule);
                Tok t;
                for (int w = 0; w < N_CALLS; ++w) {
                    lq_state s = state();
                    const int before = launches;
                    const int got = call(w, &d, &s, t);
                    const bool rule_ok = !(general_only(w) && rule != LQ_RULE_GENERAL) &&
                                         !(needs_read(w) && rule == LQ_RULE_GENERAL);
                    if (rule_ok) {
                        EXPECT(got == LQ_OK);
                        EXPECT(launches == before + 1);
                        EXPECT(std::memcmp(&last_dims, &d, sizeof(d)) == 0);
                    } else {
                        EXPECT(got == LQ_EINVAL);
                        EXPECT(launches == before);
                    }
                }
            }
}

void test_rejections() {
    Tok t;
    // NULL dims and state
    for (int w = 0; w < N_CALLS; ++w) {
        lq_state s = state();
        const int before = launches;
        EXPECT(call(w, nullptr, &s, t) == LQ_EINVAL);
        if (w != 5 && w != 6) {
            lq_dims d = dims(LQ_GATE_SCALAR, LQ_CODE_INT8, general_only(w) ? LQ_RULE_GENERAL : LQ_RULE_DELTA);
            EXPECT(call(w, &d, nullptr, t) == LQ_EINVAL);
        }
        EXPECT(launches == before);
    }
    struct Bad {
        void (*edit)(lq_dims &);
        int want;
    };
    const Bad bad[] = {
        {[](lq_dims &d) { d.batch = 0; }, LQ_EINVAL},
        {[](lq_dims &d) { d.heads_v = -1; }, LQ_EINVAL},
        {[](lq_dims &d) { d.heads_k = 3; }, LQ_EINVAL},
        {[](lq_dims &d) { d.window = 0; }, LQ_EINVAL},
        {[](lq_dims &d) { d.n_comp = -1; }, LQ_EINVAL},
        {[](lq_dims &d) { d.power_iters = -1; }, LQ_EINVAL},
        {[](lq_dims &d) { d.gate = 2; }, LQ_EINVAL},
        {[](lq_dims &d) { d.code = 5; }, LQ_EINVAL},
        {[](lq_dims &d) { d.code = -1; }, LQ_EINVAL},
        {[](lq_dims &d) { d.smooth = 2; }, LQ_EINVAL},
        {[](lq_dims &d) { d.rule = 3; }, LQ_EINVAL},
        {[](lq_dims &d) { d.d_k = 64; }, LQ_EUNSUPPORTED},
        {[](lq_dims &d) { d.d_v = 256; }, LQ_EUNSUPPORTED},
        {[](lq_dims &d) { d.n_comp = LQ_MAX_COMP + 1; }, LQ_EUNSUPPORTED},
        {[](lq_dims &d) { d.power_iters = 0; }, LQ_EUNSUPPORTED},
        {[](lq_dims &d) { d.power_iters = LQ_MAX_POWER_ITERS + 1; }, LQ_EUNSUPPORTED},
        {[](lq_dims &d) { d.window = LQ_MAX_WINDOW_GDN + 1; }, LQ_EUNSUPPORTED},
        {[](lq_dims &d) { d.gate = LQ_GATE_DIAG; d.window = LQ_MAX_WINDOW_KDA + 1; }, LQ_EUNSUPPORTED},
        {[](lq_dims &d) { d.code = LQ_CODE_BF16; }, LQ_EUNSUPPORTED},   // BF16 state with tokens
        // shapes whose tile index or key-head mapping would overflow the kernels' integers
        {[](lq_dims &d) { d.batch = 1 << 30; d.heads_v = 2; d.heads_k = 2; }, LQ_EUNSUPPORTED},
        {[](lq_dims &d) { d.batch = 1 << 22; d.heads_v = 1 << 8; d.heads_k = 1; }, LQ_EUNSUPPORTED},
        {[](lq_dims &d) { d.batch = 0x7FFFFFFF; d.heads_v = 0x7FFFFFFF; d.heads_k = 1; }, LQ_EUNSUPPORTED},
    };
    for (const Bad &b : bad) {
        lq_dims d = dims();
        b.edit(d);
        all_reject(d, b.want, __LINE__);
    }
    // misaligned and NULL state fields, per field
    for (int f = 0; f < 10; ++f)
        for (int kind = 0; kind < 2; ++kind) {
            for (int w = 0; w < N_CALLS; ++w) {
                if (w == 5 || w == 6) continue;     // the baselines take no lq_state
                lq_dims d = dims(LQ_GATE_SCALAR, LQ_CODE_INT8, general_only(w) ? LQ_RULE_GENERAL : LQ_RULE_DELTA);
                lq_state s = state();
                char **fields = reinterpret_cast<char **>(&s);
                fields[f] = kind == 0 ? nullptr : fields[f] + 1;
                const int before = launches;
                const int got = call(w, &d, &s, t);
                EXPECT(launches == before);
                EXPECT(got == (kind == 0 ? LQ_EINVAL : LQ_EALIGN));
            }
        }
    // misaligned token buffers: 16 bytes for q, k, v, o, the read vector and the
    // per-channel alpha; 4 bytes for beta and the scalar alpha
    for (int gate = 0; gate < 2; ++gate)
        for (int f = 0; f < 7; ++f)
            for (int off : {2, 4, 8}) {
                Tok t2;
                float **fs[] = {&t2.q, &t2.k, &t2.v, &t2.a, &t2.b, &t2.o, &t2.rv};
                *fs[f] = (float *)(P((uintptr_t)*fs[f]) + off);
                const bool four = f == 4 || (f == 3 && gate == LQ_GATE_SCALAR);
                for (int w = 1; w < N_CALLS - 1; ++w) {
                    if (w == 4) continue;            // the window commit takes no tokens
                    const bool general = general_only(w);
                    if (f == 6 && !general) continue;
                    lq_dims d = dims(gate, LQ_CODE_INT8, general ? LQ_RULE_GENERAL : LQ_RULE_DELTA);
                    lq_state s = state();
                    const int before = launches;
                    const int got = call(w, &d, &s, t2);
                    const bool ok = four && off % 4 == 0;
                    EXPECT(got == (ok ? LQ_OK : LQ_EALIGN));
                    EXPECT(launches == before + (ok ? 1 : 0));
                }
            }
    // a misaligned commit mask, an unknown baseline state type
    {
        lq_dims d = dims();
        lq_state s = state();
        EXPECT(leapquant_window_commit(&d, &s, (const int32_t *)P(0xB00002), nullptr) == LQ_EALIGN);
        EXPECT(leapquant_window_commit(&d, &s, (const int32_t *)P(0xB00004), nullptr) == LQ_OK);
        EXPECT(leapquant_baseline_step(&d, P(0xA00000), 2, t.q, t.k, t.v, t.a, t.b, t.o, nullptr) == LQ_EINVAL);
    }
}

void test_state_bytes() {
    size_t out[10];
    lq_dims d = dims(LQ_GATE_DIAG, LQ_CODE_INT6);
    d.window = 256;
    EXPECT(leapquant_state_bytes(&d, out) == LQ_OK);
    const size_t t = 12;
    EXPECT(out[0] == t * 128 * 128 * 6 / 8);
    EXPECT(out[7] == t * 256 * 128 * 2);
    EXPECT(leapquant_state_bytes(&d, nullptr) == LQ_EINVAL);
    EXPECT(leapquant_state_bytes(nullptr, out) == LQ_EINVAL);
    d.code = LQ_CODE_BF16;
    d.n_comp = 0;
    EXPECT(leapquant_state_bytes(&d, out) == LQ_OK && out[0] == t * 128 * 128 * 2);
}

void test_errors_and_strings() {
    // a launch failure becomes LQ_EHIP with the runtime's text, kept per thread
    lq_dims d = dims();
    lq_state s = state();
    next_status = hipErrorInvalidValue;
    EXPECT(leapquant_window_commit(&d, &s, nullptr, nullptr) == LQ_EHIP);
    next_status = hipSuccess;
    const char *msg = leapquant_last_hip_error();
    EXPECT(msg != nullptr && std::strlen(msg) > 0 && std::strlen(msg) < 256);
    std::string other = "unset";
    std::thread th([&] { other = leapquant_last_hip_error(); });
    th.join();
    EXPECT(other.empty());
    for (int st = -2; st < 10; ++st) EXPECT(leapquant_strerror(st) != nullptr);
    EXPECT(leapquant_check_error(nullptr, nullptr, nullptr) == LQ_EINVAL);
    lq_state s2 = state();
    s2.err = nullptr;
    EXPECT(leapquant_check_error(&s2, nullptr, nullptr) == LQ_EINVAL);
}

}  // namespace

int main() {
    test_valid_calls_launch();
    test_rejections();
    test_state_bytes();
    test_errors_and_strings();
    if (failures) {
        std::fprintf(stderr, "%d failures\n", failures);
        return 1;
    }
    std::printf("api sanitizer check ok (%d launches)\n", launches);
    return 0;
}
