// Layer epilogue: y = x + sum over K-slices of the down projection's partials, then (inside a stack) the next
// layer's FFN input xn = y * g in the FFN kernels' input dtype and the row's sum of squares, from which the
// next gate/up kernel forms the RMSNorm factor 1 / sqrt(mean(y^2) + eps).
//
// One workgroup per token row.  Each thread owns float4 groups of the row; the slices are added in slice order
// 0, 1, 2, ... (loads issued sixteen at a time, additions in order), so the result is bitwise reproducible.
// Slices past the end of a sample's list were not written by the down projection and are skipped; with no
// listed neuron at all y = x exactly.  The row's sum of squares is reduced in a fixed order (lane butterfly,
// then the four waves in order).  A separate launch, rather than the last K-slice workgroup of each column
// tile, does this: a device-wide release from every such workgroup costs more than one kernel boundary.
#include "rm_internal.h"

namespace {

constexpr int kThreads = 256;
constexpr int kKeep = 4;  // float4 groups per thread kept in registers for the norm (d <= 4096)

__device__ __forceinline__ float4 add4(float4 a, float4 b) {
    return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w);
}

__device__ __forceinline__ float4 ld4(const float *p) { return *reinterpret_cast<const float4 *>(p); }

__device__ __forceinline__ float4 reduce_column(const float *P, size_t stride, int used, const float *xr, int c) {
    const float4 xv = ld4(xr + c);
    if (used == 0) return xv;
    float4 acc = ld4(P + c);
    for (int s = 1; s < used; s += 16) {
        float4 v[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) v[i] = ld4(P + min(s + i, used - 1) * stride + c);  // unconditional: no waits
#pragma unroll
        for (int i = 0; i < 16; ++i)
            if (s + i < used) acc = add4(acc, v[i]);
    }
    return add4(xv, acc);
}

template <bool kBf16Xn>
__device__ __forceinline__ void store_xn(void *xn, size_t o, float4 v) {
    if constexpr (kBf16Xn) {
        uint2 packed;
        packed.x = rm_f32_to_bf16_bits(v.x) | (rm_f32_to_bf16_bits(v.y) << 16);
        packed.y = rm_f32_to_bf16_bits(v.z) | (rm_f32_to_bf16_bits(v.w) << 16);
        *reinterpret_cast<uint2 *>(static_cast<uint16_t *>(xn) + o) = packed;
    } else {
        *reinterpret_cast<float4 *>(static_cast<float *>(xn) + o) = v;
    }
}

template <bool kBf16Xn>
__global__ __launch_bounds__(kThreads) void epilogue_kernel(const float *__restrict__ part, int slices,
                                                            int slice_neurons, const int32_t *__restrict__ count,
                                                            int max_count, const float *x,
                                                            float *y, int T, int d, void *__restrict__ xn_next,
                                                            const float *__restrict__ g_next,
                                                            float *__restrict__ ssq) {
    const int row = blockIdx.x;
    const int b = row / T;
    const int t = row - b * T;
    const int tid = threadIdx.x;
    int cnt = count[b];
    cnt = cnt < 0 ? 0 : (cnt > max_count ? max_count : cnt);
    const int used = (cnt + slice_neurons - 1) / slice_neurons;
    const size_t stride = static_cast<size_t>(T) * d;
    const float *P = part + static_cast<size_t>(b) * slices * stride + static_cast<size_t>(t) * d;
    const float *xr = x + static_cast<size_t>(row) * d;
    float *yr = y + static_cast<size_t>(row) * d;

    float4 keep[kKeep];
    float ss = 0.0f;
#pragma unroll
    for (int k = 0; k < kKeep; ++k) {
        const int c = (tid + k * kThreads) * 4;
        if (c < d) {
            const float4 out = reduce_column(P, stride, used, xr, c);
            *reinterpret_cast<float4 *>(yr + c) = out;
            keep[k] = out;
            ss = fmaf(out.x, out.x, ss);
            ss = fmaf(out.y, out.y, ss);
            ss = fmaf(out.z, out.z, ss);
            ss = fmaf(out.w, out.w, ss);
        }
    }
    for (int c = (tid + kKeep * kThreads) * 4; c < d; c += kThreads * 4) {
        const float4 out = reduce_column(P, stride, used, xr, c);
        *reinterpret_cast<float4 *>(yr + c) = out;
        ss = fmaf(out.x, out.x, ss);
        ss = fmaf(out.y, out.y, ss);
        ss = fmaf(out.z, out.z, ss);
        ss = fmaf(out.w, out.w, ss);
    }
    if (xn_next == nullptr) return;

    if (g_next != nullptr) {
        for (int off = 32; off >= 1; off >>= 1) ss += __shfl_xor(ss, off);
        __shared__ float wave_ss[kThreads / 64];
        if ((tid & 63) == 0) wave_ss[tid >> 6] = ss;
        __syncthreads();
        if (tid == 0) ssq[row] = (wave_ss[0] + wave_ss[1]) + (wave_ss[2] + wave_ss[3]);
    }
    const size_t ro = static_cast<size_t>(row) * d;
#pragma unroll
    for (int k = 0; k < kKeep; ++k) {
        const int c = (tid + k * kThreads) * 4;
        if (c < d) {
            float4 v = keep[k];
            if (g_next != nullptr) {
                const float4 g = ld4(g_next + c);
                v = make_float4(v.x * g.x, v.y * g.y, v.z * g.z, v.w * g.w);
            }
            store_xn<kBf16Xn>(xn_next, ro + c, v);
        }
    }
    for (int c = (tid + kKeep * kThreads) * 4; c < d; c += kThreads * 4) {
        float4 v = ld4(yr + c);
        if (g_next != nullptr) {
            const float4 g = ld4(g_next + c);
            v = make_float4(v.x * g.x, v.y * g.y, v.z * g.z, v.w * g.w);
        }
        store_xn<kBf16Xn>(xn_next, ro + c, v);
    }
}

}  // namespace

namespace rm {

hipError_t launch_epilogue(const Plan &p, const int32_t *count, const float *x, float *y, const float *g_next,
                           bool emit_xn, void *ws, hipStream_t st) {
    char *base = static_cast<char *>(ws);
    const float *part = reinterpret_cast<const float *>(base + p.off_part);
    void *xn = emit_xn ? static_cast<void *>(base + p.off_xn) : nullptr;
    float *ssq = reinterpret_cast<float *>(base + p.off_ssq);
    const int rows = p.B * p.T;
    const int slice_neurons = p.wdtype == RM_BF16 ? p.slice_units * kBfChunk : p.slice_units;
    const float *g = emit_xn ? g_next : nullptr;
    if (p.wdtype == RM_BF16)
        hipLaunchKernelGGL(epilogue_kernel<true>, dim3(rows), dim3(kThreads), 0, st, part, p.slices, slice_neurons,
                           count, p.max_count, x, y, p.T, p.d, xn, g, ssq);
    else
        hipLaunchKernelGGL(epilogue_kernel<false>, dim3(rows), dim3(kThreads), 0, st, part, p.slices, slice_neurons,
                           count, p.max_count, x, y, p.T, p.d, xn, g, ssq);
    return hipGetLastError();
}

}  // namespace rm
