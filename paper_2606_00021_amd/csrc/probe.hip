// Plain streaming read of a device buffer: the practical HBM read ceiling of
// the device, measured beside its published peak.  Grid-stride over 16-byte
// words, 8 non-temporal loads in flight per thread, 8 blocks of 256 threads
// per compute unit.
#include "internal.h"

namespace sense {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void stream_read_kernel(const u32x4* __restrict__ p,
                                                          int64_t n16, uint32_t* __restrict__ sink) {
    constexpr int U = 8;
    uint32_t acc = 0;
    const int64_t stride = (int64_t)gridDim.x * 256 * U;
    for (int64_t base = (int64_t)blockIdx.x * 256 * U + threadIdx.x; base < n16; base += stride) {
        u32x4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t i = base + (int64_t)u * 256;
            v[u] = (i < n16) ? __builtin_nontemporal_load(p + i) : u32x4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint32_t a = v[u][0], b = v[u][1], c = v[u][2], d = v[u][3];
            acc ^= a ^ b ^ c ^ d;
        }
    }
    if (acc == 0x9E3779B9u) sink[0] = acc;   // keeps the loads alive
}

}  // namespace

hipError_t launch_stream_read(const void* buf, size_t bytes, uint32_t* sink, hipStream_t stream) {
    const int64_t n16 = (int64_t)(bytes / 16);
    hipLaunchKernelGGL(stream_read_kernel, dim3((unsigned)(device_cus() * 8)), dim3(256), 0, stream,
                       (const u32x4*)buf, n16, sink);
    return hipGetLastError();
}

}  // namespace sense
