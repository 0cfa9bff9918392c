// Compact copies of a group's selected weight rows (paper section 4.1, last paragraph; section 5 builds one mask
// per layer and group): each layer's listed rows copied once, contiguously, for all the steps of the group.
//
// gather_rows_kernel: one wave per output row, 16-byte loads and stores (a bf16 row of d = 1024 is 2 KB, two
// passes of the wave).  Output rows past a layer's count are filled with zeros: the FFN kernels read those rows
// for list slots past the count (with h = 0 there), and 0 * finite must stay 0.
#include <algorithm>

#include "rm_internal.h"

namespace {

constexpr int kGatherThreads = 256;  // four rows per workgroup
constexpr int kGatherLayers = 64;    // layers per launch: their 3 * 64 matrix pointers travel as kernel arguments

struct GatherSrc {
    const void *p[kGatherLayers * 3];  // layer-major: w_gate, w_up, w_down of each layer
};

__global__ __launch_bounds__(kGatherThreads) void gather_rows_kernel(GatherSrc src, const int32_t *__restrict__ idx,
                                                                     const int32_t *__restrict__ count, int d_ff,
                                                                     int max_count, int row_units, int L,
                                                                     rm_u32x4 *__restrict__ out) {
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const long long row = static_cast<long long>(blockIdx.x) * (kGatherThreads / 64) + wave;
    const long long rows = static_cast<long long>(L) * 3 * max_count;
    if (row >= rows) return;
    const int i = static_cast<int>(row % max_count);  // slot in the layer's list
    const int lm = static_cast<int>(row / max_count);  // layer * 3 + matrix
    const int l = lm / 3;
    int cnt = count[l];
    cnt = cnt < 0 ? 0 : (cnt > max_count ? max_count : cnt);
    rm_u32x4 *dst = out + row * row_units;
    if (i >= cnt) {
        for (int u = lane; u < row_units; u += 64) dst[u] = rm_u32x4{0u, 0u, 0u, 0u};
        return;
    }
    int n = idx[static_cast<size_t>(l) * d_ff + i];
    n = n < 0 ? 0 : (n >= d_ff ? d_ff - 1 : n);
    const rm_u32x4 *s = static_cast<const rm_u32x4 *>(src.p[lm]) + static_cast<size_t>(n) * row_units;
    for (int u = lane; u < row_units; u += 64) dst[u] = s[u];
}

}  // namespace

namespace rm {

hipError_t launch_gather_rows(const rm_ffn_layer_weights *w, const int32_t *idx, const int32_t *count, int d_ff,
                              int d, int wdtype, int max_count, int L, void *out, hipStream_t st) {
    const int row_units = d * (wdtype == RM_BF16 ? 2 : 4) / 16;
    for (int l0 = 0; l0 < L; l0 += kGatherLayers) {
        const int nl = std::min(kGatherLayers, L - l0);
        GatherSrc src{};
        for (int l = 0; l < nl; ++l) {
            src.p[3 * l] = w[l0 + l].w_gate;
            src.p[3 * l + 1] = w[l0 + l].w_up;
            src.p[3 * l + 2] = w[l0 + l].w_down;
        }
        const long long rows = static_cast<long long>(nl) * 3 * max_count;
        const long long blocks = (rows + kGatherThreads / 64 - 1) / (kGatherThreads / 64);
        rm_u32x4 *dst = static_cast<rm_u32x4 *>(out) + static_cast<size_t>(l0) * 3 * max_count * row_units;
        hipLaunchKernelGGL(gather_rows_kernel, dim3(static_cast<unsigned>(blocks)), dim3(kGatherThreads), 0, st, src,
                           idx + static_cast<size_t>(l0) * d_ff, count + l0, d_ff, max_count, row_units, nl, dst);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace rm
