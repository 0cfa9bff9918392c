// Mask -> ascending active-neuron index list (rm_mask_compact).
//
// A reference execution's neuron mask is stored as the indices of its selected neurons and shared by every
// step of a denoising group (paper section 4.1, "Group-Shared Neuron Masks"; section 5 builds one mask per
// layer and group).  The kernel turns a uint8 mask into that list.
//
// Grid: one workgroup per (mask, segment of 1024 neurons).  Every workgroup first counts the active neurons of
// its mask before its segment and in total, reading the whole mask (at most a few KB, from L2): the workgroups
// need no communication, so one launch of many small workgroups replaces a serial sweep by one.  It then scans its
// segment (4 neurons per thread: wave inclusive scan, prefix over the four waves) and writes the positions of
// its active neurons, in order, from list slot `before` on; and it fills the slots of its own index range that
// lie past the total with -1.  The list is ascending by construction, and the result is bit-exact and
// independent of scheduling.
#include "rm_internal.h"

namespace {

constexpr int kThreads = 256;
constexpr int kSeg = 4 * kThreads;  // neurons per workgroup

__device__ __forceinline__ uint32_t nonzero_bytes(uint32_t v) {
    return ((v & 0x000000ffu) ? 1u : 0u) | ((v & 0x0000ff00u) ? 2u : 0u) | ((v & 0x00ff0000u) ? 4u : 0u) |
           ((v & 0xff000000u) ? 8u : 0u);
}

// Sum of v over the workgroup.
__device__ __forceinline__ int block_sum(int v, int *lds) {
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
    const int wave = threadIdx.x >> 6;
    __syncthreads();  // lds may still be read by a previous call
    if ((threadIdx.x & 63) == 0) lds[wave] = v;
    __syncthreads();
    return lds[0] + lds[1] + lds[2] + lds[3];
}

__global__ __launch_bounds__(kThreads) void mask_compact_kernel(const uint8_t *__restrict__ mask, int d_ff,
                                                                int nseg, int32_t *__restrict__ idx,
                                                                int32_t *__restrict__ count) {
    const int m = blockIdx.x / nseg;
    const int s = blockIdx.x - m * nseg;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const uint8_t *row = mask + static_cast<size_t>(m) * d_ff;
    int32_t *out = idx + static_cast<size_t>(m) * d_ff;
    const int seg0 = s * kSeg;
    const int seg1 = min(seg0 + kSeg, d_ff);
    __shared__ int lds[kThreads / 64];
    // This segment's mask bytes, kept as they pass through step 1.
    __shared__ __attribute__((aligned(16))) uint32_t seg_bytes[kSeg / 4];

    // 1. Active neurons before the segment and in the whole mask.
    int before = 0, total = 0;
    const bool al16 = (reinterpret_cast<uintptr_t>(row) & 15u) == 0;
    const int n16 = al16 ? d_ff / 16 : 0;  // whole 16-byte units (they never straddle a segment boundary)
    // Four units per thread are loaded before any is counted (one wait per 16 KB of mask); units past the end
    // re-read the last unit and are not counted.
    constexpr int kBatch = 4;
    for (int u0 = tid; u0 < n16; u0 += kBatch * kThreads) {
        uint4 v[kBatch];
#pragma unroll
        for (int i = 0; i < kBatch; ++i)
            v[i] = *reinterpret_cast<const uint4 *>(row + min(u0 + i * kThreads, n16 - 1) * 16);
#pragma unroll
        for (int i = 0; i < kBatch; ++i) {
            const int u = u0 + i * kThreads;
            const int c = __popc(nonzero_bytes(v[i].x)) + __popc(nonzero_bytes(v[i].y)) +
                          __popc(nonzero_bytes(v[i].z)) + __popc(nonzero_bytes(v[i].w));
            if (u < n16) {
                total += c;
                if (u * 16 < seg0) before += c;
                if (u * 16 >= seg0 && u * 16 < seg1)
                    *reinterpret_cast<uint4 *>(&seg_bytes[(u * 16 - seg0) / 4]) = v[i];
            }
        }
    }
    for (int p = n16 * 16 + tid; p < d_ff; p += kThreads) {  // unaligned rows and the ragged end, bytewise
        const uint8_t m8 = row[p];
        const int c = m8 != 0;
        total += c;
        if (p < seg0) before += c;
        if (p >= seg0 && p < seg1) reinterpret_cast<uint8_t *>(seg_bytes)[p - seg0] = m8;
    }
    before = block_sum(before, lds);
    total = block_sum(total, lds);

    // 2. This thread's 4 neurons of the segment (from LDS: every byte of [seg0, seg1) was stored in step 1, and
    //    block_sum's barriers made it visible), their exclusive prefix within the segment, and the writes.
    const int p0 = seg0 + 4 * tid;
    uint32_t bits = 0;
    if (p0 < seg1) {
        bits = nonzero_bytes(seg_bytes[tid]);
        if (p0 + 4 > seg1) bits &= (1u << (seg1 - p0)) - 1u;  // bytes past the mask are not neurons
    }
    const int mine = __popc(bits);
    int incl = mine;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int v = __shfl_up(incl, off);
        if (lane >= off) incl += v;
    }
    __syncthreads();  // lds was read by block_sum
    if (lane == 63) lds[wave] = incl;
    __syncthreads();
    int before_wave = 0;
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) before_wave += (w < wave) ? lds[w] : 0;
    int pos = before + before_wave + incl - mine;
    while (bits) {
        const int j = __builtin_ctz(bits);
        out[pos++] = p0 + j;
        bits &= bits - 1;
    }

    // 3. The -1 tail inside this workgroup's index range, and the count.
    for (int p = max(total, seg0) + tid; p < seg1; p += kThreads) out[p] = -1;
    if (s == 0 && tid == 0) count[m] = total;
}

}  // namespace

namespace rm {

hipError_t launch_mask_compact(const uint8_t *mask, int n_masks, int d_ff, int32_t *idx, int32_t *count,
                               hipStream_t st) {
    const int nseg = (d_ff + kSeg - 1) / kSeg;
    hipLaunchKernelGGL(mask_compact_kernel, dim3(nseg * n_masks), dim3(kThreads), 0, st, mask, d_ff, nseg, idx,
                       count);
    return hipGetLastError();
}

}  // namespace rm
