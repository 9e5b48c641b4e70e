// Streaming ceilings for the benchmark (measurement helpers, not part of the
// method's ABI): read a device buffer once with coalesced non-temporal 16-byte
// loads and nothing else, to give a measured HBM read rate next to the
// decode's (non-temporal loads stream about 13% faster than plain ones here,
// so they set the ceiling); and read and write back a buffer in place, the
// access pattern of the dense baselines.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr int NT = 256;
constexpr int UNROLL = 8;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint4 ld_nt(const uint4 *p) {
    const u32x4 v = __builtin_nontemporal_load((const u32x4 *)p);
    return make_uint4(v.x, v.y, v.z, v.w);
}

// Thread t of the grid reads 16-byte words t, t + stride, ... (stride = grid
// threads), UNROLL at a time, and folds them into one word per workgroup so the
// loads are not removed.
__global__ __launch_bounds__(NT) void stream_read(const uint4 *p, size_t words, uint32_t *sink) {
    const size_t stride = (size_t)gridDim.x * NT;
    size_t i = (size_t)blockIdx.x * NT + threadIdx.x;
    uint32_t acc = 0;
    for (; i + (UNROLL - 1) * stride < words; i += UNROLL * stride) {
        uint4 w[UNROLL];
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) w[u] = ld_nt(p + i + u * stride);
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) acc ^= w[u].x ^ w[u].y ^ w[u].z ^ w[u].w;
    }
    for (; i < words; i += stride) {
        const uint4 w = ld_nt(p + i);
        acc ^= w.x ^ w.y ^ w.z ^ w.w;
    }
    __shared__ uint32_t red[NT];
    red[threadIdx.x] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t x = 0;
        for (int t = 0; t < NT; ++t) x ^= red[t];
        sink[blockIdx.x] = x;
    }
}

// In-place read-modify-write of a buffer, the access pattern of a dense state
// update: thread t of the grid loads 16-byte words t, t + stride, ... (plain
// loads), adds 1 to the first lane of each and stores it back (plain stores).
__global__ __launch_bounds__(NT) void stream_rw(uint4 *p, size_t words) {
    const size_t stride = (size_t)gridDim.x * NT;
    size_t i = (size_t)blockIdx.x * NT + threadIdx.x;
    for (; i + (UNROLL - 1) * stride < words; i += UNROLL * stride) {
        uint4 w[UNROLL];
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) w[u] = p[i + u * stride];
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) {
            w[u].x += 1u;
            p[i + u * stride] = w[u];
        }
    }
    for (; i < words; i += stride) {
        uint4 w = p[i];
        w.x += 1u;
        p[i] = w;
    }
}

}  // namespace

// Read and write back `bytes` (a multiple of 16, 16-byte aligned) at device
// pointer p on `stream`.  Returns 0, or a hipError_t value.
extern "C" int lqb_stream_rw(void *p, size_t bytes, int grid, void *stream) {
    if (!p || grid <= 0 || (bytes & 15) || ((uintptr_t)p & 15)) return (int)hipErrorInvalidValue;
    hipLaunchKernelGGL(stream_rw, dim3(grid), dim3(NT), 0, (hipStream_t)stream, (uint4 *)p, bytes / 16);
    return (int)hipGetLastError();
}

// Read `bytes` (a multiple of 16, 16-byte aligned) from device pointer p on
// `stream`; `sink` needs `grid` words.  Returns 0, or a hipError_t value.
extern "C" int lqb_stream_read(const void *p, size_t bytes, uint32_t *sink, int grid, void *stream) {
    if (!p || !sink || grid <= 0 || (bytes & 15) || ((uintptr_t)p & 15)) return (int)hipErrorInvalidValue;
    hipLaunchKernelGGL(stream_read, dim3(grid), dim3(NT), 0, (hipStream_t)stream, (const uint4 *)p,
                       bytes / 16, sink);
    return (int)hipGetLastError();
}
