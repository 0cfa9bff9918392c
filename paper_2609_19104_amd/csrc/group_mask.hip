// Group neuron masks from reference activations (paper section 5, "Constructing Group Neuron Masks", with the
// contribution score of Eq. 1 from section 3.4).
//
// Per layer l of a group of S steps: c[s][n] = (sum over t of |h[s][n][t]|) * ||W_down[n]||_2 (Eq. 1); each
// step's K best neurons are candidates; the mask is the K candidates with the largest sum over the steps of c.
// Top-K is an integer decision on floating-point scores, so every sum here has a fixed order and single
// rounding per operation (no contraction into fused multiply-adds): |h| over t = 0 .. T-1, w^2 over columns
// j = 0 .. d-1 (each square rounded), the steps' scores over s = 0 .. S-1, a correctly rounded square root and
// a rounded product.  Ties at the K-th place go to the lower neuron index.
//
// Kernels:
//   neuron_norms_kernel:  one wave per 64 neurons; a 64 x 64 weight tile at a time goes through LDS (coalesced
//                         row loads), then each lane adds its own row's 64 squares in column order.
//   scores_kernel:        one wave per (step, layer, 64 neurons): the rows go through LDS with coalesced loads,
//                         then lane n adds row n in token order.
//   step_select_kernel:   one workgroup per (step, layer), 16 neurons per thread (256 threads up to d_ff = 4096,
//                         else 1024, d_ff <= 16384): the step's top K sets the layer's mask bytes (their union over
//                         the steps).
//   group_rerank_kernel:  one workgroup per layer (same size): the union's top K by summed score.
// Top K is an MSB-first radix select over the scores' bit patterns (non-negative floats order like their bits):
// four 8-bit passes, each a histogram (per-wave LDS histograms with integer atomics, so the counts are exact,
// then added) and a suffix scan that finds the digit of the K-th largest key; then the keys above that
// threshold plus the lowest-index keys equal to it, found with a workgroup prefix sum.
#include "rm_select.h"

namespace {

using rm_sel::kSelPerThread;
using rm_sel::kSelThreads;
using rm_sel::kSelThreadsSmall;
using rm_sel::mul_rounded;
using rm_sel::select_top_k;
using rm_sel::SelLds;

// ------------------------------------------------------------------------------------------ norms

template <bool kBf16>
__global__ __launch_bounds__(64) void neuron_norms_kernel(const void *__restrict__ w, int d_ff, int d,
                                                          float *__restrict__ norms) {
    __shared__ float tile[64][65];  // 64 rows x 64 columns, padded: lane n reads row n without bank conflicts
    const int lane = threadIdx.x;
    const int n0 = blockIdx.x * 64;
    float s = 0.0f;
    for (int c0 = 0; c0 < d; c0 += 64) {
        // 64 rows x 64 columns: each lane loads 8 pieces of 8 columns, 8 lanes per row.
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const int piece = lane + 64 * k;  // 0 .. 511
            const int r = piece >> 3;
            const int cc = (piece & 7) * 8;
            const int row = min(n0 + r, d_ff - 1);
            // d is a multiple of 32, so a piece is wholly inside or outside the row.  A piece outside reads the
            // row's first piece and contributes +0 (no change to a non-negative sum): no branch around the load,
            // which would let the compiler wait for each load before issuing the next.
            const bool in = c0 + cc < d;
            const int col = in ? c0 + cc : 0;
            float v[8];
            if constexpr (kBf16) {
                const uint4 p = *reinterpret_cast<const uint4 *>(static_cast<const uint16_t *>(w) +
                                                                 static_cast<size_t>(row) * d + col);
                const uint32_t q[4] = {p.x, p.y, p.z, p.w};
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    v[2 * i] = __uint_as_float(q[i] << 16);
                    v[2 * i + 1] = __uint_as_float(q[i] & 0xffff0000u);
                }
            } else {
                const float *src = static_cast<const float *>(w) + static_cast<size_t>(row) * d + col;
                const float4 a = *reinterpret_cast<const float4 *>(src);
                const float4 b = *reinterpret_cast<const float4 *>(src + 4);
                v[0] = a.x, v[1] = a.y, v[2] = a.z, v[3] = a.w, v[4] = b.x, v[5] = b.y, v[6] = b.z, v[7] = b.w;
            }
#pragma unroll
            for (int i = 0; i < 8; ++i) v[i] = in ? v[i] : 0.0f;
#pragma unroll
            for (int i = 0; i < 8; ++i) tile[r][cc + i] = v[i];
        }
        __syncthreads();
        for (int j = 0; j < 64; ++j) s = __fadd_rn(s, mul_rounded(tile[lane][j], tile[lane][j]));
        __syncthreads();
    }
    if (n0 + lane < d_ff) norms[n0 + lane] = __builtin_sqrtf(s);
}

// ------------------------------------------------------------------------------------------ scores

// One wave per (step and layer, 64 neurons).  The 64 rows of T floats are contiguous in h: the wave loads them
// (or 64-token slices of them) with consecutive lanes on consecutive addresses into LDS, then lane n adds |h| of
// row n in token order.  The mask bytes of the layer are cleared here (step 0), before the selections set them.
constexpr int kScoreRows = 64;
constexpr int kScoreChunk = 64;
#ifndef RM_SCORE_BATCH
#define RM_SCORE_BATCH 32
#endif
constexpr int kScoreBatch = RM_SCORE_BATCH;  // loads in flight per lane

// s + the n staged values added in index order, one rounding per addition (the chain continues across chunks),
// with the LDS reads of 8 values issued before their additions.
__device__ __forceinline__ float row_abs_sum(float s, const float *row, int n) {
    int t = 0;
    for (; t + 8 <= n; t += 8) {
        float q[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) q[i] = row[t + i];
#pragma unroll
        for (int i = 0; i < 8; ++i) s = __fadd_rn(s, q[i]);
    }
    for (; t < n; ++t) s = __fadd_rn(s, row[t]);
    return s;
}

__global__ __launch_bounds__(64) void scores_kernel(const float *__restrict__ h, int d_ff, int T,
                                                    const float *__restrict__ norms, int L,
                                                    float *__restrict__ scores, uint8_t *__restrict__ mask) {
    __shared__ float tile[kScoreRows * (kScoreChunk + 1)];
    const int lane = threadIdx.x;
    const int n0 = blockIdx.x * kScoreRows;
    const int sl = blockIdx.y;  // step * L + layer
    const int rows = min(kScoreRows, d_ff - n0);
    const float *base = h + (static_cast<size_t>(sl) * d_ff + n0) * T;
    float s = 0.0f;
    if (T <= kScoreChunk && (T & 1)) {
        // Fast path (one chunk, odd T): the rows are one contiguous run of rows * T floats, staged as they lie
        // (row n at n T: an odd pitch, so lane n's reads of row n fall in distinct banks); element e = lane + 64 k
        // is a fixed offset from the lane's first, so the address arithmetic is one clamp per load.
        const int total = rows * T;
        const float *p = base + lane;
        for (int k0 = 0; k0 * 64 < total; k0 += kScoreBatch) {
            float v[kScoreBatch];
#pragma unroll
            for (int k = 0; k < kScoreBatch; ++k) v[k] = p[min(64 * (k0 + k), total - 1 - lane)];
#pragma unroll
            for (int k = 0; k < kScoreBatch; ++k)
                if (lane + 64 * (k0 + k) < total) tile[lane + 64 * (k0 + k)] = fabsf(v[k]);
        }
        __syncthreads();
        if (lane < rows) s = row_abs_sum(s, tile + lane * T, T);
    } else {
        for (int t0 = 0; t0 < T; t0 += kScoreChunk) {
            const int C = min(kScoreChunk, T - t0);
            const int stride = C | 1;  // odd row pitch: lane n's reads of row n fall in distinct banks
            const int total = rows * C;  // <= 64 x 64: at most 64 elements per lane
            // The lane's elements e = lane + 64 k, (row r, token t) with e = r C + t stepped without a division,
            // in batches of kScoreBatch loads issued before any is used (elements past the chunk re-read its last
            // one and are not stored).
            const int dr = 64 / C, dt = 64 - dr * C;
            int r = lane / C, t = lane - r * C;
            for (int k0 = 0; k0 * 64 < total; k0 += kScoreBatch) {
                float v[kScoreBatch];
                int rs = r, ts = t;
#pragma unroll
                for (int k = 0; k < kScoreBatch; ++k) {
                    const bool in = lane + 64 * (k0 + k) < total;
                    v[k] = base[static_cast<size_t>(in ? r : rows - 1) * T + t0 + (in ? t : C - 1)];
                    r += dr;
                    t += dt;
                    if (t >= C) {
                        t -= C;
                        ++r;
                    }
                }
#pragma unroll
                for (int k = 0; k < kScoreBatch; ++k) {
                    if (lane + 64 * (k0 + k) < total) tile[rs * stride + ts] = fabsf(v[k]);
                    rs += dr;
                    ts += dt;
                    if (ts >= C) {
                        ts -= C;
                        ++rs;
                    }
                }
            }
            __syncthreads();
            if (lane < rows) s = row_abs_sum(s, tile + lane * stride, C);
            __syncthreads();
        }
    }
    if (lane < rows) {
        const int l = sl % L;
        const float nrm = norms[static_cast<size_t>(l) * d_ff + n0 + lane];
        scores[static_cast<size_t>(sl) * d_ff + n0 + lane] = __fmul_rn(s, nrm);
        if (sl < L) mask[static_cast<size_t>(l) * d_ff + n0 + lane] = 0;
    }
}

// ------------------------------------------------------------------------------------------ selection

// Each step's K best neurons of one layer (workgroup = step * L + layer) set their mask bytes to 1: the mask
// holds the union of the steps' candidates when the rerank runs.
template <int kThreads>
__global__ __launch_bounds__(kThreads) void step_select_kernel(const float *__restrict__ scores, int L, int d_ff,
                                                               int k, uint8_t *__restrict__ mask) {
    __shared__ SelLds<kThreads> l;
    const int sl = blockIdx.x;
    const int n0 = threadIdx.x * kSelPerThread;
    const float *c = scores + static_cast<size_t>(sl) * d_ff;
    uint32_t valid = 0, key[kSelPerThread];
#pragma unroll
    for (int i = 0; i < kSelPerThread; ++i) {
        const bool ok = n0 + i < d_ff;
        if (ok) valid |= 1u << i;
        key[i] = ok ? __float_as_uint(c[n0 + i]) : 0u;  // c >= 0: its bits order like its value
    }
    const uint32_t sel = select_top_k(key, valid, k, d_ff, l);
    uint8_t *m = mask + static_cast<size_t>(sl % L) * d_ff;
#pragma unroll
    for (int i = 0; i < kSelPerThread; ++i)
        if ((sel >> i) & 1u) m[n0 + i] = 1;  // several steps may set the same byte to the same value
}

// The layer's mask: the K members of the union (mask bytes set by step_select_kernel) with the largest score
// summed over the steps in step order.  Neurons outside the union get the smallest key and are never taken
// (the union holds at least K neurons).
template <int kThreads>
__global__ __launch_bounds__(kThreads) void group_rerank_kernel(const float *__restrict__ scores, int S, int L,
                                                                int d_ff, int k, uint8_t *__restrict__ mask) {
    __shared__ SelLds<kThreads> l;
    const int layer = blockIdx.x;
    const int n0 = threadIdx.x * kSelPerThread;
    uint8_t *m = mask + static_cast<size_t>(layer) * d_ff;
    uint32_t valid = 0, key[kSelPerThread];
    float summed[kSelPerThread];
#pragma unroll
    for (int i = 0; i < kSelPerThread; ++i) {
        summed[i] = 0.0f;
        if (n0 + i < d_ff) valid |= 1u << i;
    }
    // The loads of a step are all issued before its sums, with no branch between them (a branch would let the
    // compiler sink each load to its use, one round trip per neuron); slots past d_ff read the last neuron and
    // are not used.
    const int last = d_ff - 1;
    for (int s = 0; s < S; ++s) {
        const float *c = scores + (static_cast<size_t>(s) * L + layer) * d_ff;
        float v[kSelPerThread];
#pragma unroll
        for (int i = 0; i < kSelPerThread; ++i) v[i] = c[min(n0 + i, last)];
#pragma unroll
        for (int i = 0; i < kSelPerThread; ++i) summed[i] = __fadd_rn(summed[i], v[i]);
    }
    uint8_t in_union[kSelPerThread];
#pragma unroll
    for (int i = 0; i < kSelPerThread; ++i) in_union[i] = m[min(n0 + i, last)];
#pragma unroll
    for (int i = 0; i < kSelPerThread; ++i)
        key[i] = ((valid >> i) & 1u) && in_union[i] != 0 ? __float_as_uint(summed[i]) + 1u : 0u;
    const uint32_t sel = select_top_k(key, valid, k, d_ff, l);
#pragma unroll
    for (int i = 0; i < kSelPerThread; ++i)
        if ((valid >> i) & 1u) m[n0 + i] = static_cast<uint8_t>((sel >> i) & 1u);
}

}  // namespace

namespace rm {

hipError_t launch_neuron_norms(const void *w_down, int d_ff, int d, int wdtype, float *norms, hipStream_t st) {
    const dim3 grid((d_ff + 63) / 64);
    if (wdtype == RM_BF16)
        hipLaunchKernelGGL(neuron_norms_kernel<true>, grid, dim3(64), 0, st, w_down, d_ff, d, norms);
    else
        hipLaunchKernelGGL(neuron_norms_kernel<false>, grid, dim3(64), 0, st, w_down, d_ff, d, norms);
    return hipGetLastError();
}

hipError_t launch_group_masks(const float *h, int S, int L, int d_ff, int T, const float *norms, int k,
                              float *scores, uint8_t *mask, hipStream_t st) {
    hipError_t e = launch_timed(RM_KERNEL_SCORES, scores_kernel, dim3((d_ff + kScoreRows - 1) / kScoreRows, S * L),
                                dim3(64), st, h, d_ff, T, norms, L, scores, mask);
    if (e == hipSuccess) e = hipGetLastError();
    if (e != hipSuccess) return e;
    const float *sc = scores;
    // A workgroup of 256 threads while the layer's neurons fit (fewer waves meet at each barrier), else 1024.
    if (d_ff <= kSelThreadsSmall * kSelPerThread) {
        e = launch_timed(RM_KERNEL_GROUP_SELECT, step_select_kernel<kSelThreadsSmall>, dim3(S * L),
                         dim3(kSelThreadsSmall), st, sc, L, d_ff, k, mask);
        if (e == hipSuccess) e = hipGetLastError();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(group_rerank_kernel<kSelThreadsSmall>, dim3(L), dim3(kSelThreadsSmall), 0, st, sc, S, L,
                           d_ff, k, mask);
        return hipGetLastError();
    }
    e = launch_timed(RM_KERNEL_GROUP_SELECT, step_select_kernel<kSelThreads>, dim3(S * L), dim3(kSelThreads), st, sc,
                     L, d_ff, k, mask);
    if (e == hipSuccess) e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(group_rerank_kernel<kSelThreads>, dim3(L), dim3(kSelThreads), 0, st, sc, S, L, d_ff, k, mask);
    return hipGetLastError();
}

}  // namespace rm
