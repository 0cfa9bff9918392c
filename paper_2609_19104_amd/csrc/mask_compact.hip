// Mask -> ascending active-neuron index list (rm_mask_compact).
//
// A reference execution's neuron mask is stored as the indices of its selected neurons and shared by every
// step of a denoising group (paper section 4.1, "Group-Shared Neuron Masks"; section 5 builds one mask per
// layer and group).  The kernel turns a uint8 mask into that list.
//
// One 256-thread workgroup per mask.  The mask is walked in chunks of 1024 neurons; a lane owns 4 consecutive
// bytes.  The wave ballots each of the 4 byte positions, so a lane's first output slot is
//   (active neurons in earlier chunks) + (active in earlier waves of this chunk)
//   + (active in lower lanes of this wave: mbcnt of the 4 ballots)
// and its own active bytes follow in order.  The list is therefore ascending by construction and the result
// is bit-exact and independent of scheduling.  Slots after the count are filled with -1.
#include "rm_internal.h"

namespace {

constexpr int kThreads = 256;
constexpr int kChunk = kThreads * 4;

__device__ __forceinline__ int lanes_below(uint64_t ballot) {
    // Number of set bits of `ballot` in lanes below this one.
    return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(ballot >> 32),
                                     __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(ballot), 0u));
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
    const bool row_aligned = (reinterpret_cast<uintptr_t>(row) & 3u) == 0;

    __shared__ int wave_total[kThreads / 64];
    int running = 0;  // active neurons before the current chunk (uniform across the workgroup)

    for (int base = 0; base < d_ff; base += kChunk) {
        const int p0 = base + tid * 4;
        uint32_t act = 0;  // bit j set <=> neuron p0 + j is active
        if (row_aligned && p0 + 4 <= d_ff) {
            const uint32_t v = *reinterpret_cast<const uint32_t *>(row + p0);
            act = ((v & 0x000000ffu) ? 1u : 0u) | ((v & 0x0000ff00u) ? 2u : 0u) |
                  ((v & 0x00ff0000u) ? 4u : 0u) | ((v & 0xff000000u) ? 8u : 0u);
        } else {
            for (int j = 0; j < 4; ++j)
                if (p0 + j < d_ff && row[p0 + j] != 0) act |= 1u << j;
        }
        const uint64_t b0 = __ballot(act & 1u);
        const uint64_t b1 = __ballot(act & 2u);
        const uint64_t b2 = __ballot(act & 4u);
        const uint64_t b3 = __ballot(act & 8u);
        const int below = lanes_below(b0) + lanes_below(b1) + lanes_below(b2) + lanes_below(b3);
        if (lane == 0) wave_total[wave] = __popcll(b0) + __popcll(b1) + __popcll(b2) + __popcll(b3);
        __syncthreads();
        int before_wave = 0, chunk_total = 0;
        for (int w = 0; w < kThreads / 64; ++w) {
            before_wave += (w < wave) ? wave_total[w] : 0;
            chunk_total += wave_total[w];
        }
        int pos = running + before_wave + below;
        for (int j = 0; j < 4; ++j)
            if (act & (1u << j)) out[pos++] = p0 + j;
        running += chunk_total;
        __syncthreads();  // wave_total is rewritten by the next chunk
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
