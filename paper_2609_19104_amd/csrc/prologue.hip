// First layer's FFN input: xn = x * g (or x without a norm) in the FFN kernels' input dtype, plus the row's
// sum of squares for the RMSNorm factor.  Also the identity index lists with which the dense reference runs the
// sparse kernels.
//
// The action expert normalizes each FFN input (the layer is x + FFN(RMSNorm(x)) with RMSNorm(x) =
// x / sqrt(mean(x^2) + eps) * g).  The per-token factor is applied by the gate/up kernel after its matrix-core
// products, so xn itself stays unscaled; the row's sum of squares is reduced here in a fixed order (lane
// butterfly, then waves 0..3).  One workgroup per token row.
#include <algorithm>

#include "rm_internal.h"

namespace {

constexpr int kThreads = 256;

template <bool kBf16Out>
__global__ __launch_bounds__(kThreads) void prologue_kernel(const float *__restrict__ x,
                                                            const float *__restrict__ g, int d,
                                                            void *__restrict__ xn, float *__restrict__ ssq) {
    const int row = blockIdx.x;
    const int tid = threadIdx.x;

    const float *xr = x + static_cast<size_t>(row) * d;
    float ss = 0.0f;
    for (int c = tid * 4; c < d; c += kThreads * 4) {
        float4 v = *reinterpret_cast<const float4 *>(xr + c);
        if (g != nullptr) {
            ss = fmaf(v.x, v.x, ss);
            ss = fmaf(v.y, v.y, ss);
            ss = fmaf(v.z, v.z, ss);
            ss = fmaf(v.w, v.w, ss);
            const float4 gv = *reinterpret_cast<const float4 *>(g + c);
            v.x *= gv.x;
            v.y *= gv.y;
            v.z *= gv.z;
            v.w *= gv.w;
        }
        const size_t o = static_cast<size_t>(row) * d + c;
        if constexpr (kBf16Out) {
            uint2 packed;
            packed.x = rm_f32_to_bf16_bits(v.x) | (rm_f32_to_bf16_bits(v.y) << 16);
            packed.y = rm_f32_to_bf16_bits(v.z) | (rm_f32_to_bf16_bits(v.w) << 16);
            *reinterpret_cast<uint2 *>(static_cast<uint16_t *>(xn) + o) = packed;
        } else {
            *reinterpret_cast<float4 *>(static_cast<float *>(xn) + o) = v;
        }
    }
    if (g == nullptr) return;
    for (int off = 32; off >= 1; off >>= 1) ss += __shfl_xor(ss, off);
    __shared__ float wave_ss[kThreads / 64];
    if ((tid & 63) == 0) wave_ss[tid >> 6] = ss;
    __syncthreads();
    if (tid == 0) ssq[row] = (wave_ss[0] + wave_ss[1]) + (wave_ss[2] + wave_ss[3]);
}

__global__ __launch_bounds__(kThreads) void identity_lists_kernel(int32_t *idx, int32_t *count, int d_ff, int B) {
    const size_t n = static_cast<size_t>(B) * d_ff;
    for (size_t i = static_cast<size_t>(blockIdx.x) * kThreads + threadIdx.x; i < n;
         i += static_cast<size_t>(gridDim.x) * kThreads)
        idx[i] = static_cast<int32_t>(i % d_ff);
    if (blockIdx.x == 0 && threadIdx.x < B) count[threadIdx.x] = d_ff;
    for (int b = kThreads + threadIdx.x; blockIdx.x == 0 && b < B; b += kThreads) count[b] = d_ff;
}

}  // namespace

namespace rm {

hipError_t launch_identity_lists(const Plan &p, void *ws, hipStream_t st) {
    char *base = static_cast<char *>(ws);
    int32_t *idx = reinterpret_cast<int32_t *>(base + p.off_ident);
    int32_t *count = reinterpret_cast<int32_t *>(base + p.off_ident_count);
    const size_t n = static_cast<size_t>(p.B) * p.d_ff;
    const int blocks = static_cast<int>(std::min<size_t>((n + kThreads - 1) / kThreads, 1024));
    hipLaunchKernelGGL(identity_lists_kernel, dim3(blocks), dim3(kThreads), 0, st, idx, count, p.d_ff, p.B);
    return hipGetLastError();
}

hipError_t launch_prologue(const Plan &p, const float *x, const float *norm_g, void *ws, hipStream_t st) {
    char *base = static_cast<char *>(ws);
    void *xn = base + p.off_xn;
    float *ssq = reinterpret_cast<float *>(base + p.off_ssq);
    const int rows = p.B * p.T;
    if (p.wdtype == RM_BF16)
        hipLaunchKernelGGL(prologue_kernel<true>, dim3(rows), dim3(kThreads), 0, st, x, norm_g, p.d, xn, ssq);
    else
        hipLaunchKernelGGL(prologue_kernel<false>, dim3(rows), dim3(kThreads), 0, st, x, norm_g, p.d, xn, ssq);
    return hipGetLastError();
}

}  // namespace rm
