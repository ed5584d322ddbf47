// stream_read.hip -- a plain HBM stream read (the measured read ceiling).
//
// Work group b reads part b of the buffer: ceil(units / blocks) contiguous
// 16-byte units, each thread every 256th unit, eight loads in flight per
// thread, with the non-temporal hint (data read once should not displace
// anything).  The XOR of everything a work group read goes to its sink word,
// which keeps the loads alive and lets a test check what was read.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "splice_calib.h"

namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 8;

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(kThreads) void stream_read_kernel(const u32x4_t *buf, uint64_t units, uint32_t *sink) {
    const uint64_t per = (units + gridDim.x - 1) / gridDim.x;
    const uint64_t lo = min(units, per * blockIdx.x);
    const uint64_t hi = min(units, lo + per);
    u32x4_t acc = {0u, 0u, 0u, 0u};
    uint64_t i = lo + threadIdx.x;
    for (; i + (uint64_t)(kUnroll - 1) * kThreads < hi; i += (uint64_t)kUnroll * kThreads) {
        u32x4_t v[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) v[u] = __builtin_nontemporal_load(buf + i + (uint64_t)u * kThreads);
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) acc ^= v[u];
    }
    for (; i < hi; i += kThreads) acc ^= __builtin_nontemporal_load(buf + i);
    uint32_t x = acc.x ^ acc.y ^ acc.z ^ acc.w;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) x ^= (uint32_t)__shfl_xor((int)x, o);
    __shared__ uint32_t waves[kThreads / 64];
    if ((threadIdx.x & 63) == 0) waves[threadIdx.x >> 6] = x;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t y = 0;
#pragma unroll
        for (int w = 0; w < kThreads / 64; ++w) y ^= waves[w];
        sink[blockIdx.x] = y;
    }
}

}  // namespace

extern "C" SPLICE_CALIB_API int32_t splice_calib_stream_read(const void *buf, uint64_t bytes, uint32_t *sink,
                                                             int32_t blocks, void *stream) {
    if (!buf || !sink || ((uintptr_t)buf & 15u) || bytes == 0 || (bytes & 15u) || blocks < 1 ||
        blocks > SPLICE_CALIB_MAX_BLOCKS)
        return SPLICE_CALIB_EINVAL;
    hipLaunchKernelGGL(stream_read_kernel, dim3((unsigned)blocks), dim3(kThreads), 0, (hipStream_t)stream,
                       (const u32x4_t *)buf, bytes / 16, sink);
    return hipGetLastError() == hipSuccess ? SPLICE_CALIB_OK : SPLICE_CALIB_EHIP;
}
