// Device bodies shared by the mask-compaction, prologue and fused compaction + prologue kernels: one
// workgroup's compaction of a (mask, segment) unit and one wave's prologue of a (token row, column block) unit.
// See mask_compact.hip and prologue.hip for what they compute.
#pragma once

#include "rm_internal.h"
#include "rm_select.h"

namespace rm_units {

constexpr int kCompactThreads = 256;
constexpr int kSeg = 4 * kCompactThreads;  // neurons per compaction workgroup

__device__ __forceinline__ uint32_t nonzero_bytes(uint32_t v) {
    return ((v & 0x000000ffu) ? 1u : 0u) | ((v & 0x0000ff00u) ? 2u : 0u) | ((v & 0x00ff0000u) ? 4u : 0u) |
           ((v & 0xff000000u) ? 8u : 0u);
}

// Sums of u and v over the workgroup (kCompactThreads threads), one pair of barriers for both.
__device__ __forceinline__ void block_sum2(int &u, int &v, int *lds) {
    for (int off = 32; off >= 1; off >>= 1) {
        u += __shfl_xor(u, off);
        v += __shfl_xor(v, off);
    }
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
        lds[wave] = u;
        lds[4 + wave] = v;
    }
    __syncthreads();
    u = lds[0] + lds[1] + lds[2] + lds[3];
    v = lds[4] + lds[5] + lds[6] + lds[7];
}

// Mask m, segment s (neurons [s * kSeg, (s + 1) * kSeg)) -> the segment's part of idx[m] and, for s == 0,
// count[m].  All kCompactThreads threads of the workgroup take part.
__device__ __forceinline__ void compact_segment(const uint8_t *__restrict__ mask, int d_ff, int m, int s,
                                                int32_t *__restrict__ idx, int32_t *__restrict__ count) {
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const uint8_t *row = mask + static_cast<size_t>(m) * d_ff;
    int32_t *out = idx + static_cast<size_t>(m) * d_ff;
    const int seg0 = s * kSeg;
    const int seg1 = min(seg0 + kSeg, d_ff);
    static_assert(kCompactThreads == 256, "block_sum2 adds four waves");
    __shared__ int lds[2 * kCompactThreads / 64];
    // This segment's mask bytes, kept as they pass through step 1.
    __shared__ __attribute__((aligned(16))) uint32_t seg_bytes[kSeg / 4];

    // 1. Active neurons before the segment and in the whole mask.
    int before = 0, total = 0;
    const bool al16 = (reinterpret_cast<uintptr_t>(row) & 15u) == 0;
    const int n16 = al16 ? d_ff / 16 : 0;  // whole 16-byte units (they never straddle a segment boundary)
    // Four units per thread are loaded before any is counted (one wait per 16 KB of mask); units past the end
    // re-read the last unit and are not counted.
    constexpr int kBatch = 4;
    for (int u0 = tid; u0 < n16; u0 += kBatch * kCompactThreads) {
        uint4 v[kBatch];
#pragma unroll
        for (int i = 0; i < kBatch; ++i)
            v[i] = *reinterpret_cast<const uint4 *>(row + min(u0 + i * kCompactThreads, n16 - 1) * 16);
#pragma unroll
        for (int i = 0; i < kBatch; ++i) {
            const int u = u0 + i * kCompactThreads;
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
    for (int p = n16 * 16 + tid; p < d_ff; p += kCompactThreads) {  // unaligned rows, the ragged end: bytewise
        const uint8_t m8 = row[p];
        const int c = m8 != 0;
        total += c;
        if (p < seg0) before += c;
        if (p >= seg0 && p < seg1) reinterpret_cast<uint8_t *>(seg_bytes)[p - seg0] = m8;
    }
    block_sum2(before, total, lds);

    // 2. This thread's 4 neurons of the segment (from LDS: every byte of [seg0, seg1) was stored in step 1, and
    //    block_sum2's barrier made it visible), their exclusive prefix within the segment, and the writes.
    const int p0 = seg0 + 4 * tid;
    uint32_t bits = 0;
    if (p0 < seg1) {
        bits = nonzero_bytes(seg_bytes[tid]);
        if (p0 + 4 > seg1) bits &= (1u << (seg1 - p0)) - 1u;  // bytes past the mask are not neurons
    }
    const int mine = __popc(bits);
    const int incl = rm_sel::wave_incl_scan(mine);  // every lane of the wave takes part
    __shared__ int wave_tot[kCompactThreads / 64];   // its own array: no barrier against block_sum2's reads
    if (lane == 63) wave_tot[wave] = incl;
    __syncthreads();
    int before_wave = 0;
#pragma unroll
    for (int w = 0; w < kCompactThreads / 64; ++w) before_wave += (w < wave) ? wave_tot[w] : 0;
    int pos = before + before_wave + incl - mine;
    while (bits) {
        const int j = __builtin_ctz(bits);
        out[pos++] = p0 + j;
        bits &= bits - 1;
    }

    // 3. The -1 tail inside this workgroup's index range, and the count.
    for (int p = max(total, seg0) + tid; p < seg1; p += kCompactThreads) out[p] = -1;
    if (s == 0 && tid == 0) count[m] = total;
}

// Prologue of unit = row * nblk + blk (token row, block of 256 columns) by one wave; lane = the thread's lane.
template <bool kBf16Out>
__device__ __forceinline__ void prologue_unit(const float *__restrict__ x, const float *__restrict__ g, int d,
                                              int nblk, void *__restrict__ xn, float *__restrict__ ssq, int unit,
                                              int lane) {
    const int row = unit / nblk;
    const int blk = unit - row * nblk;
    const int c = blk * rm::kRowBlock + lane * 4;
    const size_t o = static_cast<size_t>(row) * d + c;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (c < d) v = *reinterpret_cast<const float4 *>(x + o);
    if (g != nullptr) {  // partial sums of squares of the row's 32-column blocks (lane 8 j: block 8 blk + j)
        const float ss = rm_ssq32(v, c < d);
        const int part = blk * 8 + (lane >> 3);
        if ((lane & 7) == 0 && part < rm::ssq_parts(d))
            ssq[static_cast<size_t>(row) * rm::ssq_stride(d) + part] = ss;
    }
    if (c < d) {
        if (g != nullptr) {
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
}

}  // namespace rm_units
