// First layer's FFN input: xn = x * g (or x without a norm) in the FFN kernels' input dtype, plus the row's
// sums of squares for the RMSNorm factor.  Also the identity index lists with which the dense reference runs the
// sparse kernels, and the launch that runs the mask compaction beside the prologue (the calls that take masks).
//
// The action expert normalizes each FFN input (the layer is x + FFN(RMSNorm(x)) with RMSNorm(x) =
// x / sqrt(mean(x^2) + eps) * g).  The per-token factor is applied by the gate/up kernel after its matrix-core
// products, so xn itself stays unscaled.  One wave per (token row, block of 256 columns), each lane a float4:
// the row's sum of squares is kept as one partial per column block (lane butterfly, fixed order), which the
// gate/up kernel adds in block order.
#include <algorithm>

#include "rm_units.h"

namespace {

constexpr int kThreads = 64;

template <bool kBf16Out>
__global__ __launch_bounds__(kThreads) void prologue_kernel(const float *__restrict__ x,
                                                            const float *__restrict__ g, int d, int nblk,
                                                            void *__restrict__ xn, float *__restrict__ ssq) {
    rm_units::prologue_unit<kBf16Out>(x, g, d, nblk, xn, ssq, blockIdx.x, threadIdx.x);
}

// Compaction and prologue in one launch (they are independent): workgroups [0, n_compact) each compact one
// (mask, segment) unit; each later workgroup runs the prologue of four (row, column block) units, one per wave.
template <bool kBf16Out>
__global__ __launch_bounds__(rm_units::kCompactThreads) void compact_prologue_kernel(
    const uint8_t *__restrict__ mask, int d_ff, int nseg, int n_compact, int32_t *__restrict__ idx,
    int32_t *__restrict__ count, const float *__restrict__ x, const float *__restrict__ g, int d, int nblk,
    int units, void *__restrict__ xn, float *__restrict__ ssq) {
    const int w = static_cast<int>(blockIdx.x);
    if (w < n_compact) {
        const int m = w / nseg;
        rm_units::compact_segment(mask, d_ff, m, w - m * nseg, idx, count);
        return;
    }
    const int unit = (w - n_compact) * (rm_units::kCompactThreads / 64) + static_cast<int>(threadIdx.x >> 6);
    if (unit < units) rm_units::prologue_unit<kBf16Out>(x, g, d, nblk, xn, ssq, unit, threadIdx.x & 63);
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

hipError_t launch_compact_prologue(const Plan &p, const uint8_t *mask, int n_masks, int32_t *idx, int32_t *count,
                                   const float *x, const float *norm_g, void *ws, hipStream_t st) {
    char *base = static_cast<char *>(ws);
    void *xn = base + p.off_xn;
    float *ssq = reinterpret_cast<float *>(base + p.off_ssq);
    const int nblk = (p.d + kRowBlock - 1) / kRowBlock;
    const int nseg = (p.d_ff + rm_units::kSeg - 1) / rm_units::kSeg;
    const int n_compact = nseg * n_masks;
    const int units = p.B * p.T * nblk;
    const int per = rm_units::kCompactThreads / 64;
    const dim3 grid(n_compact + (units + per - 1) / per);
    const dim3 block(rm_units::kCompactThreads);
    if (p.wdtype == RM_BF16)
        hipLaunchKernelGGL(compact_prologue_kernel<true>, grid, block, 0, st, mask, p.d_ff, nseg, n_compact, idx,
                           count, x, norm_g, p.d, nblk, units, xn, ssq);
    else
        hipLaunchKernelGGL(compact_prologue_kernel<false>, grid, block, 0, st, mask, p.d_ff, nseg, n_compact, idx,
                           count, x, norm_g, p.d, nblk, units, xn, ssq);
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
