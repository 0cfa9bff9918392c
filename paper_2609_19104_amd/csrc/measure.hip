// Measurement kernel: a plain streaming read of a device buffer.  The benchmark times it on the same box as the
// hot path, so the hot path's bandwidth can be stated as a fraction of what a bare read reaches there, beside the
// fraction of the HBM specification.
//
// Each lane reads 16-byte pieces in a grid-stride loop, eight loads in flight before their values are combined;
// consecutive lanes read consecutive pieces (whole 128-byte lines per 8 lanes).  The values are XOR-ed into one
// word per lane, which is stored only if it equals a magic number: the loads cannot be dropped, and in practice
// nothing is written.
#include "rm_internal.h"

namespace {

constexpr int kThreads = 512;
constexpr int kInFlight = 8;
constexpr uint32_t kMagic = 0x9e3779b9u;

__global__ __launch_bounds__(kThreads) void stream_read_kernel(const uint4 *__restrict__ p, size_t n16,
                                                               uint32_t *__restrict__ sink) {
    const size_t stride = static_cast<size_t>(gridDim.x) * kThreads;
    size_t i = static_cast<size_t>(blockIdx.x) * kThreads + threadIdx.x;
    uint32_t acc = 0;
    for (; i + (kInFlight - 1) * stride < n16; i += kInFlight * stride) {
        uint4 v[kInFlight];
#pragma unroll
        for (int k = 0; k < kInFlight; ++k) v[k] = p[i + k * stride];
#pragma unroll
        for (int k = 0; k < kInFlight; ++k) acc ^= v[k].x ^ v[k].y ^ v[k].z ^ v[k].w;
    }
    for (; i < n16; i += stride) {
        const uint4 v = p[i];
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    if (acc == kMagic) sink[static_cast<size_t>(blockIdx.x) * kThreads + threadIdx.x] = acc;
}

}  // namespace

namespace rm {

hipError_t launch_stream_read(const void *buf, size_t bytes, int workgroups, uint32_t *sink, hipStream_t st) {
    hipLaunchKernelGGL(stream_read_kernel, dim3(workgroups), dim3(kThreads), 0, st, static_cast<const uint4 *>(buf),
                       bytes / 16, sink);
    return hipGetLastError();
}

}  // namespace rm
