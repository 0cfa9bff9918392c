// Device helpers shared by the kernels that rank float32 scores: an exactly rounded product, a workgroup prefix
// sum, and the top-K selection of a workgroup of 256 or 1024 threads (group_mask.hip, context_cache.hip).
//
// Top K is an MSB-first radix select over the scores' bit patterns (non-negative floats order like their bits):
// four 8-bit passes, each a histogram (per-wave LDS histograms with integer atomics, so the counts are exact,
// then added) and a suffix scan that finds the digit of the K-th largest key; then the keys above that
// threshold plus the lowest-index keys equal to it, found with a workgroup prefix sum.
#pragma once

#include "rm_internal.h"

namespace rm_sel {

constexpr int kSelThreads = 1024;      // the largest workgroup: 16384 keys
constexpr int kSelThreadsSmall = 256;  // up to 4096 keys: a quarter of the waves at each barrier
constexpr int kSelPerThread = 16;      // keys per thread

// a * b rounded to float32 on its own: the empty asm statement hides the product from the optimizer, so it
// cannot be fused with the sum it feeds into one multiply-add (HIP compiles with contraction allowed).
__device__ __forceinline__ float mul_rounded(float a, float b) {
    float p = a * b;
    asm volatile("" : "+v"(p));
    return p;
}

template <int kThreads>
struct SelLds {
    // One histogram per wave (atomics only contend within a wave), two sets: a pass counts into one while the
    // other is cleared for the next pass.
    uint32_t whist[2][kThreads / 64][256];
    int wave_sum[kThreads / 64];
    int digit, need;
};

// Inclusive prefix sum over the 64 lanes of a wave (every lane active), with DPP moves instead of LDS
// permutes: scans within rows of 16 lanes (row_shr 1, 2, 4, 8, a source outside the row adding 0), then row 0's
// total into row 1 and row 2's into row 3 (row_bcast:15), then rows 0-1's into rows 2-3 (row_bcast:31).
__device__ __forceinline__ int wave_incl_scan(int x) {
    x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xF, 0xF, true);
    x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xF, 0xF, true);
    x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xF, 0xF, true);
    x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xF, 0xF, true);
    x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xA, 0xF, false);
    x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xC, 0xF, false);
    return x;
}

// Exclusive prefix sum of v over the workgroup, in thread order.
template <int kThreads>
__device__ __forceinline__ int block_excl_scan(int v, SelLds<kThreads> &l) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int incl = wave_incl_scan(v);
    __syncthreads();  // wave_sum may still be read by a previous call
    if (lane == 63) l.wave_sum[wave] = incl;
    __syncthreads();
    int before = 0;
    for (int w = 0; w < wave; ++w) before += l.wave_sum[w];
    return before + incl - v;
}

// Selection bits (bit i: item tid * 16 + i) of the k largest keys among the thread's valid ones (bit i of
// `valid`), ties to the lower item index.  0 <= k; every thread of the workgroup calls it.
template <int kThreads>
__device__ inline uint32_t select_top_k(const uint32_t (&key)[kSelPerThread], uint32_t valid, int k, int n_valid,
                                        SelLds<kThreads> &l) {
    static_assert(kThreads >= 256, "wave 0 finds the digit while at least three other waves clear histograms");
    if (k <= 0) return 0u;
    if (k >= n_valid) return valid;
    constexpr int kWaves = kThreads / 64;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    uint32_t prefix = 0, hi = 0;
    int need = k;
    for (int b = lane; b < 256; b += 64) l.whist[0][wave][b] = 0u;
    __syncthreads();
    // Two barriers per pass: after the counts, and after wave 0 has found the digit (meanwhile the other waves
    // clear the other histogram set for the next pass).
    for (int pass = 0; pass < 4; ++pass) {
        const int shift = 24 - 8 * pass, buf = pass & 1;
#pragma unroll
        for (int i = 0; i < kSelPerThread; ++i)
            if (((valid >> i) & 1u) && (key[i] & hi) == prefix)
                atomicAdd(&l.whist[buf][wave][(key[i] >> shift) & 255u], 1u);
        __syncthreads();
        if (wave == 0) {  // lane j holds digits 4j .. 4j+3; find the digit holding the need-th largest key
            uint32_t b[4] = {0u, 0u, 0u, 0u};
#pragma unroll
            for (int w = 0; w < kWaves; ++w)
#pragma unroll
                for (int q = 0; q < 4; ++q) b[q] += l.whist[buf][w][4 * lane + q];
            const int own = static_cast<int>(b[0] + b[1] + b[2] + b[3]);
            const int incl = wave_incl_scan(own);
            const int above = __builtin_amdgcn_readlane(incl, 63) - incl;  // keys in digits above 4j + 3
            int cum = above;
#pragma unroll
            for (int q = 3; q >= 0; --q) {
                const int c = static_cast<int>(b[q]);
                if (cum < need && cum + c >= need) {
                    l.digit = 4 * lane + q;
                    l.need = need - cum;
                }
                cum += c;
            }
        } else {
            for (int w = wave - 1; w < kWaves; w += kWaves - 1)
                for (int b = lane; b < 256; b += 64) l.whist[buf ^ 1][w][b] = 0u;
        }
        __syncthreads();  // l.digit / l.need are rewritten by wave 0 only after the next pass's first barrier
        prefix |= static_cast<uint32_t>(l.digit) << shift;
        hi |= 255u << shift;
        need = l.need;
    }
    // prefix is the k-th largest key; take every larger key and the `need` lowest-index keys equal to it.
    uint32_t sel = 0, eq = 0;
#pragma unroll
    for (int i = 0; i < kSelPerThread; ++i) {
        if (!((valid >> i) & 1u)) continue;
        if (key[i] > prefix) sel |= 1u << i;
        if (key[i] == prefix) eq |= 1u << i;
    }
    int rank = block_excl_scan(__popc(eq), l);
#pragma unroll
    for (int i = 0; i < kSelPerThread; ++i) {
        if ((eq >> i) & 1u) {
            if (rank < need) sel |= 1u << i;
            ++rank;
        }
    }
    return sel;
}

}  // namespace rm_sel
