// Layer epilogue: y = x + sum over K-slices of the down projection's partials, then (inside a stack) the next
// layer's FFN input xn = y * g in the FFN kernels' input dtype and the row's partial sums of squares, from which
// the next gate/up kernel forms the RMSNorm factor 1 / sqrt(mean(y^2) + eps).
//
// One wave per (token row, block of 256 columns), each lane a float4, so the launch has B T d / 256 waves.  The
// slices are added in slice order 0, 1, 2, ... (their loads issued in one batch when the launch has at most 12
// slices, else sixteen at a time; the additions in order), so the result is bitwise reproducible.  Slices past the end of a sample's list are skipped (their partials hold
// zeros or are stale); with no listed neuron at all y = x exactly.  The block's sum of squares is reduced in a
// fixed order (lane butterfly).  A separate launch, rather than the last K-slice workgroup of each column tile,
// does this: a device-wide release from every such workgroup costs more than one kernel boundary.
#include "rm_internal.h"

namespace {

constexpr int kThreads = 64;

__device__ __forceinline__ float4 add4(float4 a, float4 b) {
    return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w);
}

__device__ __forceinline__ float4 ld4(const float *p) { return *reinterpret_cast<const float4 *>(p); }

template <bool kBf16Xn>
__global__ __launch_bounds__(kThreads) void epilogue_kernel(const float *__restrict__ part, int slices,
                                                            int slice_neurons, const int32_t *__restrict__ count,
                                                            int max_count, const float *x, float *y, int T, int d,
                                                            int nblk, void *__restrict__ xn_next,
                                                            const float *__restrict__ g_next,
                                                            float *__restrict__ ssq, const float *__restrict__ ya_in,
                                                            float *__restrict__ ya_out,
                                                            const float *__restrict__ out_gate) {
    const int row = blockIdx.x / nblk;
    const int blk = blockIdx.x - row * nblk;
    const int b = row / T;
    const int t = row - b * T;
    int cnt = count[b];
    cnt = cnt < 0 ? 0 : (cnt > max_count ? max_count : cnt);
    const int used = (cnt + slice_neurons - 1) / slice_neurons;
    const size_t stride = static_cast<size_t>(T) * d;
    const int c = blk * rm::kRowBlock + static_cast<int>(threadIdx.x) * 4;
    const bool ok = c < d;
    const int cc = ok ? c : d - 4;  // lanes past d read a valid column and store nothing
    const float *P = part + static_cast<size_t>(b) * slices * stride + static_cast<size_t>(t) * d + cc;
    const size_t ro = static_cast<size_t>(row) * d + cc;

    float4 out = ld4(x + ro);
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    if (slices <= 12) {
        // All the launch's slices in one batch, addressed by the slice count of the launch (not by `used`,
        // which waits for the count to arrive): the loads go out with x's, and only the additions depend on
        // the count.  Slices at or past `used` are read (they lie inside the partials) and not added.
        float4 v[12];
        if (slices <= 4) {  // several samples per call: 4 loads, not 12 mostly repeated
#pragma unroll
            for (int i = 0; i < 4; ++i) v[i] = ld4(P + min(i, slices - 1) * stride);
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (i < used) acc = i == 0 ? v[0] : add4(acc, v[i]);
        } else {
#pragma unroll
            for (int i = 0; i < 12; ++i) v[i] = ld4(P + min(i, slices - 1) * stride);
#pragma unroll
            for (int i = 0; i < 12; ++i)
                if (i < used) acc = i == 0 ? v[0] : add4(acc, v[i]);
        }
    } else if (used > 0) {
        acc = ld4(P);
        for (int s = 1; s < used; s += 16) {
            float4 v[16];
#pragma unroll
            for (int i = 0; i < 16; ++i) v[i] = ld4(P + min(s + i, used - 1) * stride);  // unconditional
#pragma unroll
            for (int i = 0; i < 16; ++i)
                if (s + i < used) acc = add4(acc, v[i]);
        }
    }
    if (ya_in != nullptr || used > 0) {  // an empty list without an anchor leaves y = x bit for bit
        float4 f = acc;
        if (ya_in != nullptr) f = add4(ld4(ya_in + ro), acc);  // Eq. 4: the FFN output is y_a + (h - h_a) W_down
        if (out_gate != nullptr) {  // the adaptive output gate, before the residual
            const float4 g = ld4(out_gate + static_cast<size_t>(b) * d + cc);
            f = make_float4(f.x * g.x, f.y * g.y, f.z * g.z, f.w * g.w);
        }
        out = add4(out, f);
    }
    if (ok) {
        *reinterpret_cast<float4 *>(y + ro) = out;
        if (ya_out != nullptr) *reinterpret_cast<float4 *>(ya_out + ro) = acc;
    }
    if (xn_next == nullptr) return;

    if (g_next != nullptr) {  // partial sums of squares of the row's 32-column blocks (lane 8 j: block 8 blk + j)
        const float ss = rm_ssq32(out, ok);
        const int part = blk * 8 + static_cast<int>(threadIdx.x >> 3);
        if ((threadIdx.x & 7) == 0 && part < rm::ssq_parts(d))
            ssq[static_cast<size_t>(row) * rm::ssq_stride(d) + part] = ss;
        if (ok) {
            const float4 g = ld4(g_next + cc);
            out = make_float4(out.x * g.x, out.y * g.y, out.z * g.z, out.w * g.w);
        }
    }
    if (!ok) return;
    if constexpr (kBf16Xn) {
        uint2 packed;
        packed.x = rm_f32_to_bf16_bits(out.x) | (rm_f32_to_bf16_bits(out.y) << 16);
        packed.y = rm_f32_to_bf16_bits(out.z) | (rm_f32_to_bf16_bits(out.w) << 16);
        *reinterpret_cast<uint2 *>(static_cast<uint16_t *>(xn_next) + ro) = packed;
    } else {
        *reinterpret_cast<float4 *>(static_cast<float *>(xn_next) + ro) = out;
    }
}

}  // namespace

namespace rm {

hipError_t launch_epilogue(const Plan &p, const int32_t *count, const float *x, float *y, const float *g_next,
                           bool emit_xn, const float *ya_in, float *ya_out, const float *out_gate, void *ws,
                           hipStream_t st) {
    char *base = static_cast<char *>(ws);
    const float *part = reinterpret_cast<const float *>(base + p.off_part);
    void *xn = emit_xn ? static_cast<void *>(base + p.off_xn) : nullptr;
    float *ssq = reinterpret_cast<float *>(base + p.off_ssq);
    const int nblk = (p.d + kRowBlock - 1) / kRowBlock;
    const dim3 grid(p.B * p.T * nblk);
    const int slice_neurons = p.wdtype == RM_BF16 ? p.slice_units * kBfChunk : p.slice_units;
    const float *g = emit_xn ? g_next : nullptr;
    if (p.wdtype == RM_BF16)
        hipLaunchKernelGGL(epilogue_kernel<true>, grid, dim3(kThreads), 0, st, part, p.slices, slice_neurons, count,
                           p.max_count, x, y, p.T, p.d, nblk, xn, g, ssq, ya_in, ya_out, out_gate);
    else
        hipLaunchKernelGGL(epilogue_kernel<false>, grid, dim3(kThreads), 0, st, part, p.slices, slice_neurons,
                           count, p.max_count, x, y, p.T, p.d, nblk, xn, g, ssq, ya_in, ya_out, out_gate);
    return hipGetLastError();
}

}  // namespace rm
