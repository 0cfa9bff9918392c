// float32 masked SwiGLU FFN on the vector ALU (for float32 weights; float32 end to end).
//
// With float32 weights the arithmetic intensity is T/2 FLOP per weight byte, a few FLOP/B at the small token
// counts of an action chunk, so the vector ALU keeps up with HBM and no input rounding is needed.
//
// gate/up (gateup_f32_kernel): one wave per 8 listed neurons; 8 lanes per neuron row, each lane reading
//   16 contiguous bytes (128 contiguous bytes per row per step).  8 tokens per register block; the 8 lanes'
//   partial dot products are combined with a fixed xor butterfly, then lane j forms h for token j.
// down (down_f32_kernel): one wave per (256-column tile, K-slice of listed neurons, sample); a lane owns
//   4 columns, loops over its slice's neurons (one 1 KB coalesced row segment per neuron and wave) and keeps
//   8 tokens x 4 columns of float32 sums.  The slice's float32 partial is stored; the epilogue kernel adds
//   the slices in order to the residual (no float atomics).
// The FFN input xn is x * g; the per-token RMSNorm factor multiplies the gate and up sums (see ffn_bf16.hip).
#include "rm_internal.h"

namespace {

constexpr int kWave = 64;

__device__ __forceinline__ int clamp_neuron(int n, int d_ff) { return n < 0 ? 0 : (n >= d_ff ? d_ff - 1 : n); }

__global__ __launch_bounds__(kWave) void gateup_f32_kernel(
    const float *__restrict__ wg, const float *__restrict__ wu, const float *__restrict__ xn,
    const int32_t *__restrict__ idx, const int32_t *__restrict__ count, int max_count, int d_ff, int d, int T,
    int tpad, float *__restrict__ H, int kcap, const float *__restrict__ ssq, float eps,
    const float *__restrict__ h_anchor, float *__restrict__ h_out, int act) {
    const int b = blockIdx.y;
    const int slot0 = blockIdx.x * rm::kF32NeurPerBlk;
    const int lane = threadIdx.x;
    int cnt = count[b];
    cnt = cnt < 0 ? 0 : (cnt > max_count ? max_count : cnt);
    if (slot0 >= cnt) return;  // the down projection never reads slots past the list

    const int r = lane >> 3;  // neuron of the block
    const int cl = lane & 7;  // 16-byte column group of each 128-byte step
    const int slot = slot0 + r;
    const bool valid = slot < cnt;
    const int n = valid ? clamp_neuron(idx[static_cast<size_t>(b) * d_ff + slot], d_ff) : 0;
    const float *grow = wg + static_cast<size_t>(n) * d;
    const float *urow = wu + static_cast<size_t>(n) * d;
    const float *xb = xn + static_cast<size_t>(b) * T * d;
    float *Hb = H + static_cast<size_t>(b) * tpad * kcap;

    for (int t0 = 0; t0 < T; t0 += rm::kF32TokBlock) {
        const int nt = min(rm::kF32TokBlock, T - t0);
        float ag[rm::kF32TokBlock], au[rm::kF32TokBlock];
#pragma unroll
        for (int t = 0; t < rm::kF32TokBlock; ++t) ag[t] = au[t] = 0.0f;
        // No branch around the loads (a branch lets the compiler wait for each load before the next): a slot past
        // the list reads neuron 0 and tokens past T re-read the last token; neither sum is ever stored.
        for (int c = cl * 4; c < d; c += 32) {
            const float4 g4 = *reinterpret_cast<const float4 *>(grow + c);
            const float4 u4 = *reinterpret_cast<const float4 *>(urow + c);
            float4 xv[rm::kF32TokBlock];
#pragma unroll
            for (int t = 0; t < rm::kF32TokBlock; ++t)
                xv[t] = *reinterpret_cast<const float4 *>(xb + static_cast<size_t>(min(t0 + t, T - 1)) * d + c);
#pragma unroll
            for (int t = 0; t < rm::kF32TokBlock; ++t) {
                ag[t] = fmaf(g4.x, xv[t].x, ag[t]);
                ag[t] = fmaf(g4.y, xv[t].y, ag[t]);
                ag[t] = fmaf(g4.z, xv[t].z, ag[t]);
                ag[t] = fmaf(g4.w, xv[t].w, ag[t]);
                au[t] = fmaf(u4.x, xv[t].x, au[t]);
                au[t] = fmaf(u4.y, xv[t].y, au[t]);
                au[t] = fmaf(u4.z, xv[t].z, au[t]);
                au[t] = fmaf(u4.w, xv[t].w, au[t]);
            }
        }
        // Combine the 8 lanes of each neuron row (lanes 8r .. 8r+7): fixed butterfly.
#pragma unroll
        for (int t = 0; t < rm::kF32TokBlock; ++t) {
#pragma unroll
            for (int off = 1; off < 8; off <<= 1) {
                ag[t] += __shfl_xor(ag[t], off);
                au[t] += __shfl_xor(au[t], off);
            }
        }
        float gs = 0.f, us = 0.f;
#pragma unroll
        for (int t = 0; t < rm::kF32TokBlock; ++t) {
            if (t == cl) {
                gs = ag[t];
                us = au[t];
            }
        }
        if (t0 + cl < tpad && valid) {
            float h = 0.0f;
            if (cl < nt) {
                float rn = 1.0f;
                if (ssq != nullptr) rn = rm_token_rnorm(ssq, b * T + t0 + cl, d, eps);
                h = rm_glu_act(act, gs * rn) * (us * rn);
            }
            // Eq. 4: the anchor step keeps h of the listed slots; a delta step stores h - h_anchor.
            const size_t ai = (static_cast<size_t>(b) * max_count + slot) * T + t0 + cl;
            if (h_out != nullptr) {
                if (cl < nt) h_out[ai] = h;
            } else {
                if (h_anchor != nullptr && cl < nt) h -= h_anchor[ai];
                Hb[static_cast<size_t>(t0 + cl) * kcap + slot] = h;
            }
        }
    }
}

__global__ __launch_bounds__(kWave) void down_f32_kernel(
    const float *__restrict__ H, const float *__restrict__ wd, const int32_t *__restrict__ idx,
    const int32_t *__restrict__ count, int max_count, int d_ff, int d, int T, int tpad, int kcap, int slices,
    int slice_neurons, float *__restrict__ part) {
    const int ct = blockIdx.x;
    const int s = blockIdx.y;
    const int b = blockIdx.z;
    const int lane = threadIdx.x;
    int cnt = count[b];
    cnt = cnt < 0 ? 0 : (cnt > max_count ? max_count : cnt);
    const int k_begin = s * slice_neurons;
    const int k_end = min(k_begin + slice_neurons, cnt);
    const int col0 = ct * rm::kF32ColTile;
    const int c = col0 + lane * 4;
    const bool colok = c < d;
    const float *Hb = H + static_cast<size_t>(b) * tpad * kcap;
    const int32_t *idxb = idx + static_cast<size_t>(b) * d_ff;
    float *P = part + (static_cast<size_t>(b) * slices + s) * static_cast<size_t>(T) * d;

    if (k_begin < k_end) {
        for (int t0 = 0; t0 < T; t0 += rm::kF32TokBlock) {
            const int nt = min(rm::kF32TokBlock, T - t0);
            float4 acc[rm::kF32TokBlock];
#pragma unroll
            for (int t = 0; t < rm::kF32TokBlock; ++t) acc[t] = make_float4(0.f, 0.f, 0.f, 0.f);
            for (int k = k_begin; k < k_end; ++k) {
                const int n = clamp_neuron(idxb[k], d_ff);
                float4 w4 = make_float4(0.f, 0.f, 0.f, 0.f);
                if (colok) w4 = *reinterpret_cast<const float4 *>(wd + static_cast<size_t>(n) * d + c);
#pragma unroll
                for (int t = 0; t < rm::kF32TokBlock; ++t) {
                    const float h = Hb[static_cast<size_t>(t0 + t) * kcap + k];
                    acc[t].x = fmaf(h, w4.x, acc[t].x);
                    acc[t].y = fmaf(h, w4.y, acc[t].y);
                    acc[t].z = fmaf(h, w4.z, acc[t].z);
                    acc[t].w = fmaf(h, w4.w, acc[t].w);
                }
            }
            if (colok) {
#pragma unroll
                for (int t = 0; t < rm::kF32TokBlock; ++t)
                    if (t < nt)
                        *reinterpret_cast<float4 *>(P + static_cast<size_t>(t0 + t) * d + c) = acc[t];
            }
        }
    }

}

}  // namespace

namespace rm {

hipError_t launch_gateup_f32(const Plan &p, const void *w_gate, const void *w_up, const int32_t *idx,
                             const int32_t *count, bool norm, const float *h_anchor, float *h_out, void *ws,
                             hipStream_t st) {
    char *base = static_cast<char *>(ws);
    const float *xn = reinterpret_cast<const float *>(base + p.off_xn);
    float *H = reinterpret_cast<float *>(base + p.off_h);
    const float *ssq = norm ? reinterpret_cast<const float *>(base + p.off_ssq) : nullptr;
    const hipError_t e =
        launch_timed(RM_KERNEL_GATEUP, gateup_f32_kernel, dim3(p.gate_blocks, p.B), dim3(kWave), st,
                     static_cast<const float *>(w_gate), static_cast<const float *>(w_up), xn, idx, count, p.max_count,
                     p.d_ff, p.d, p.T, p.tpad, H, p.kcap, ssq, p.eps, h_anchor, h_out, p.act);
    return e != hipSuccess ? e : hipGetLastError();
}

hipError_t launch_down_f32(const Plan &p, const void *w_down, const int32_t *idx, const int32_t *count, void *ws,
                           hipStream_t st) {
    char *base = static_cast<char *>(ws);
    const float *H = reinterpret_cast<const float *>(base + p.off_h);
    float *part = reinterpret_cast<float *>(base + p.off_part);
    const hipError_t e = launch_timed(RM_KERNEL_DOWN, down_f32_kernel, dim3(p.ncol, p.slices, p.B), dim3(kWave), st,
                                      H, static_cast<const float *>(w_down), idx, count, p.max_count, p.d_ff, p.d,
                                      p.T, p.tpad, p.kcap, p.slices, p.slice_units, part);
    return e != hipSuccess ? e : hipGetLastError();
}

}  // namespace rm
