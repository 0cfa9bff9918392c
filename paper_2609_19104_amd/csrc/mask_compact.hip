// Mask -> ascending active-neuron index list (rm_mask_compact).
//
// A reference execution's neuron mask is stored as the indices of its selected neurons and shared by every
// step of a denoising group (paper section 4.1, "Group-Shared Neuron Masks"; section 5 builds one mask per
// layer and group).  The kernel turns a uint8 mask into that list.
//
// One 256-thread workgroup per mask.  A thread owns 16 consecutive bytes of each 4096-byte chunk, and up to
// four chunks are loaded before any is processed, so the workgroup waits for memory once per 16 KB.  Per
// chunk, the thread's active-byte count goes through a wave inclusive scan and a prefix over the four waves;
// the thread then writes its active positions in order.  The list is ascending by construction, and the
// result is bit-exact and independent of scheduling.  Slots after the count are filled with -1.
#include "rm_internal.h"

namespace {

constexpr int kThreads = 256;
constexpr int kBytes = 16;                  // bytes per thread and chunk
constexpr int kChunk = kThreads * kBytes;   // 4096 neurons
constexpr int kBatch = 4;                   // chunks loaded together

__device__ __forceinline__ uint32_t nonzero_bytes(uint32_t v) {
    return ((v & 0x000000ffu) ? 1u : 0u) | ((v & 0x0000ff00u) ? 2u : 0u) | ((v & 0x00ff0000u) ? 4u : 0u) |
           ((v & 0xff000000u) ? 8u : 0u);
}

__global__ __launch_bounds__(kThreads) void mask_compact_kernel(const uint8_t *__restrict__ mask, int d_ff,
                                                                int32_t *__restrict__ idx,
                                                                int32_t *__restrict__ count) {
    const int m = blockIdx.x;
    const uint8_t *row = mask + static_cast<size_t>(m) * d_ff;
    int32_t *out = idx + static_cast<size_t>(m) * d_ff;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const bool row_aligned = (reinterpret_cast<uintptr_t>(row) & 15u) == 0;

    __shared__ int wave_total[kThreads / 64];
    int running = 0;  // active neurons before the current chunk (uniform across the workgroup)

    for (int base = 0; base < d_ff; base += kBatch * kChunk) {
        uint32_t bits[kBatch];  // bit j: byte j of this thread's 16 is nonzero
#pragma unroll
        for (int c = 0; c < kBatch; ++c) {
            const int p0 = base + c * kChunk + tid * kBytes;
            bits[c] = 0;
            if (row_aligned && p0 + kBytes <= d_ff) {
                const uint4 v = *reinterpret_cast<const uint4 *>(row + p0);
                bits[c] = nonzero_bytes(v.x) | (nonzero_bytes(v.y) << 4) | (nonzero_bytes(v.z) << 8) |
                          (nonzero_bytes(v.w) << 12);
            } else {
                for (int j = 0; j < kBytes; ++j)
                    if (p0 + j < d_ff && row[p0 + j] != 0) bits[c] |= 1u << j;
            }
        }
#pragma unroll
        for (int c = 0; c < kBatch; ++c) {
            const int p0 = base + c * kChunk + tid * kBytes;
            if (base + c * kChunk >= d_ff) break;  // uniform
            const int mine = __popc(bits[c]);
            int incl = mine;
#pragma unroll
            for (int off = 1; off < 64; off <<= 1) {
                const int v = __shfl_up(incl, off);
                if (lane >= off) incl += v;
            }
            if (lane == 63) wave_total[wave] = incl;
            __syncthreads();
            int before_wave = 0, chunk_total = 0;
#pragma unroll
            for (int w = 0; w < kThreads / 64; ++w) {
                before_wave += (w < wave) ? wave_total[w] : 0;
                chunk_total += wave_total[w];
            }
            int pos = running + before_wave + incl - mine;
            uint32_t rest = bits[c];
            while (rest) {
                const int j = __builtin_ctz(rest);
                out[pos++] = p0 + j;
                rest &= rest - 1;
            }
            running += chunk_total;
            __syncthreads();  // wave_total is rewritten by the next chunk
        }
    }
    for (int p = running + tid; p < d_ff; p += kThreads) out[p] = -1;
    if (tid == 0) count[m] = running;
}

}  // namespace

namespace rm {

hipError_t launch_mask_compact(const uint8_t *mask, int n_masks, int d_ff, int32_t *idx, int32_t *count,
                               hipStream_t st) {
    hipLaunchKernelGGL(mask_compact_kernel, dim3(n_masks), dim3(kThreads), 0, st, mask, d_ff, idx, count);
    return hipGetLastError();
}

}  // namespace rm
