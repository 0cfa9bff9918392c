// First layer's FFN input: xn = x * g (or x without a norm) in the FFN kernels' input dtype, plus the row's
// sums of squares for the RMSNorm factor.  Also the identity index lists with which the dense reference runs the
// sparse kernels.
//
// The action expert normalizes each FFN input (the layer is x + FFN(RMSNorm(x)) with RMSNorm(x) =
// x / sqrt(mean(x^2) + eps) * g).  The per-token factor is applied by the gate/up kernel after its matrix-core
// products, so xn itself stays unscaled.  One wave per (token row, block of 256 columns), each lane a float4:
// the row's sum of squares is kept as one partial per column block (lane butterfly, fixed order), which the
// gate/up kernel adds in block order.
#include <algorithm>

#include "rm_internal.h"

namespace {

constexpr int kThreads = 64;

template <bool kBf16Out>
__global__ __launch_bounds__(kThreads) void prologue_kernel(const float *__restrict__ x,
                                                            const float *__restrict__ g, int d, int nblk,
                                                            void *__restrict__ xn, float *__restrict__ ssq) {
    const int row = blockIdx.x / nblk;
    const int blk = blockIdx.x - row * nblk;
    const int c = blk * rm::kRowBlock + static_cast<int>(threadIdx.x) * 4;
    const size_t o = static_cast<size_t>(row) * d + c;
    float ss = 0.0f;
    if (c < d) {
        float4 v = *reinterpret_cast<const float4 *>(x + o);
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
    if (threadIdx.x == 0) ssq[blockIdx.x] = ss;  // [row][blk]
}

__global__ __launch_bounds__(256) void identity_lists_kernel(int32_t *idx, int32_t *count, int d_ff, int B) {
    const size_t n = static_cast<size_t>(B) * d_ff;
    const size_t step = static_cast<size_t>(gridDim.x) * 256;
    for (size_t i = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x; i < n; i += step)
        idx[i] = static_cast<int32_t>(i % d_ff);
    for (int b = threadIdx.x; blockIdx.x == 0 && b < B; b += 256) count[b] = d_ff;
}

}  // namespace

namespace rm {

hipError_t launch_identity_lists(const Plan &p, void *ws, hipStream_t st) {
    char *base = static_cast<char *>(ws);
    int32_t *idx = reinterpret_cast<int32_t *>(base + p.off_ident);
    int32_t *count = reinterpret_cast<int32_t *>(base + p.off_ident_count);
    const size_t n = static_cast<size_t>(p.B) * p.d_ff;
    const int blocks = static_cast<int>(std::min<size_t>((n + 255) / 256, 1024));
    hipLaunchKernelGGL(identity_lists_kernel, dim3(blocks), dim3(256), 0, st, idx, count, p.d_ff, p.B);
    return hipGetLastError();
}

hipError_t launch_prologue(const Plan &p, const float *x, const float *norm_g, void *ws, hipStream_t st) {
    char *base = static_cast<char *>(ws);
    void *xn = base + p.off_xn;
    float *ssq = reinterpret_cast<float *>(base + p.off_ssq);
    const int nblk = (p.d + kRowBlock - 1) / kRowBlock;
    const dim3 grid(p.B * p.T * nblk);
    if (p.wdtype == RM_BF16)
        hipLaunchKernelGGL(prologue_kernel<true>, grid, dim3(kThreads), 0, st, x, norm_g, p.d, nblk, xn, ssq);
    else
        hipLaunchKernelGGL(prologue_kernel<false>, grid, dim3(kThreads), 0, st, x, norm_g, p.d, nblk, xn, ssq);
    return hipGetLastError();
}

}  // namespace rm
