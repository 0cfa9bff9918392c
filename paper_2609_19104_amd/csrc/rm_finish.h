// Deterministic finish of the down projection: fixed-order sum of K-slice partials + residual.
//
// The down projection y = x + sum_k h[:,k] W_down[idx[k], :] is split over K (the listed neurons) into
// `slices` workgroups per output column tile; each writes its float32 partial for the tile.  Every workgroup
// then takes an integer ticket for its tile; the one that takes the last ticket adds the partials in slice
// order 0, 1, 2, ... to x and writes y.  The order of the sum does not depend on which workgroup finishes last,
// so results are bitwise reproducible, and no floating-point atomics are used.  That workgroup also resets the
// ticket to 0 for the next launch.
#pragma once

#include "rm_internal.h"

// part_tile: [slices][T][CT] floats of this (sample, column tile).  used_slices: how many of them were written
// (slices past the end of the sample's list hold no neurons and are skipped).  If none were, y = x exactly.
template <int CT>
__device__ __forceinline__ void rm_finish_column_tile(const float *part_tile, int slices, int used_slices,
                                                      int *ticket, const float *x, float *y, int T, int d,
                                                      int col0) {
    __shared__ int s_is_last;
    __threadfence();  // release this workgroup's partial to the whole device
    __syncthreads();
    if (threadIdx.x == 0) s_is_last = (atomicAdd(ticket, 1) == slices - 1) ? 1 : 0;
    __syncthreads();
    if (!s_is_last) return;
    __threadfence();  // acquire the other workgroups' partials

    constexpr int kVec = CT / 4;
    for (int e = threadIdx.x; e < T * kVec; e += blockDim.x) {
        const int t = e / kVec;
        const int c = (e % kVec) * 4;
        if (col0 + c >= d) continue;
        const size_t o = static_cast<size_t>(t) * d + col0 + c;
        const float4 xv = *reinterpret_cast<const float4 *>(x + o);
        if (used_slices == 0) {
            *reinterpret_cast<float4 *>(y + o) = xv;
            continue;
        }
        float4 acc = *reinterpret_cast<const float4 *>(part_tile + static_cast<size_t>(t) * CT + c);
        for (int s = 1; s < used_slices; ++s) {
            const float4 v =
                *reinterpret_cast<const float4 *>(part_tile + (static_cast<size_t>(s) * T + t) * CT + c);
            acc.x += v.x;
            acc.y += v.y;
            acc.z += v.z;
            acc.w += v.w;
        }
        float4 out;
        out.x = xv.x + acc.x;
        out.y = xv.y + acc.y;
        out.z = xv.z + acc.z;
        out.w = xv.w + acc.w;
        *reinterpret_cast<float4 *>(y + o) = out;
    }
    if (threadIdx.x == 0) *ticket = 0;
}
