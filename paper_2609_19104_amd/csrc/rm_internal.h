// Internal declarations shared by the HIP sources of the rmuscle library (gfx950 only).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <tuple>

#include "rmuscle.h"

namespace rm {

// ---------------------------------------------------------------------------------------------------------
// Launch plan and workspace layout.  One plan is derived on the host from (shape, B, T, max_count); the same
// function sizes the workspace and every launch, so they always agree.
// ---------------------------------------------------------------------------------------------------------

// The spread gate/up kernel for long single-sample lists (set to 0 at build time to compare without it).
#ifndef RM_GATEUP_SPREAD
#define RM_GATEUP_SPREAD 1
#endif

// One launch for the gate/up and down projections of one sample's long list at d = 2048, its workgroups meeting
// per XCD between the two (set to 0 at build time to compare with the separate launches).
#ifndef RM_LAYER_XCD
#define RM_LAYER_XCD 1
#endif
// The meetings of that launch: one uint64 flag per workgroup (8 XCDs x 32), then one counter per XCD, each on
// its own 256-byte line.
constexpr int kXcdFlagBytes = 8 * 32 * 8;
constexpr int kXcdCtrBytes = 8 * 256;
// How long a workgroup of that launch waits for the rest of its XCD before it gives up (100 MHz clock ticks).
constexpr long long kXcdSpinTicks = 20000000;  // 200 ms

// bf16 path: 16x16x32 bf16 matrix-core tiles.
constexpr int kBfTokBlock = 64;     // tokens per accumulator block (4 tiles of 16)
constexpr int kBfNeurPerBlk = 8;    // neurons per gate/up workgroup (8 gate rows + 8 up rows = one 16-row tile)
constexpr int kBfChunk = 32;        // neurons per down-projection matrix-core step (K of the 16x16x32 tile)
constexpr int kBfColTile = 64;      // output columns per down workgroup (16 lanes x 4 columns)
constexpr int kBfWaves = 4;
constexpr int kBfMaxChunksPerSlice = 32;  // down: a slice's indices (32 x 32) are staged in 4 KB of LDS
constexpr int kDfWaves = 8;        // fused down: waves per workgroup
constexpr int kDfMaxCpw = 8;       // fused down: at most 8 chunks per wave
constexpr int kDfMaxChunks = kDfWaves * kDfMaxCpw;  // lists of up to 64 chunks (2048 neurons)

// Prologue / epilogue: one wave per (token row, block of 256 columns).
constexpr int kRowBlock = 256;
// RMSNorm sums of squares are kept as partial sums over blocks of kSsqCols columns, [row][ssq_stride(d)] with
// ssq_parts(d) partials per row (the rest of the row is padding, never read into a sum).  d is a multiple of 32,
// so every block is whole.
constexpr int kSsqCols = 32;
__host__ __device__ constexpr int ssq_parts(int d) { return (d + kSsqCols - 1) / kSsqCols; }
__host__ __device__ constexpr int ssq_stride(int d) { return (ssq_parts(d) + 3) / 4 * 4; }

// f32 path: vector ALU.
constexpr int kF32TokBlock = 8;     // tokens per register block
constexpr int kF32NeurPerBlk = 8;   // neurons per gate/up wave (8 lanes per neuron row)
constexpr int kF32ColTile = 256;    // output columns per down wave (64 lanes x 4 columns)
constexpr int kF32SliceNeur = 16;   // neurons per down K-slice

struct Plan {
    int d = 0, d_ff = 0, wdtype = 0, B = 0, T = 0, max_count = 0, act = RM_ACT_SILU;
    float eps = 1e-6f;
    int tpad = 0;        // T rounded up to the token block (rows of H)
    int kcap = 0;        // row length of H (neuron slots), max_count rounded up
    int gate_groups = 1; // bf16 gate/up: groups of 8 neurons per workgroup (1 = direct, 2/4/8 = LDS-staged)
    int gate_blocks = 0; // gate/up workgroups per sample
    // bf16, one sample, 257 .. 768 groups of 8 listed slots: the spread gate/up kernel, gate_blocks (= one per
    // compute unit) workgroups taking quads of 4 slots round-robin, in at most gate_spread 16-row tiles each (0 =
    // not used).
    int gate_spread = 0;
    int col_tile = 0;    // output columns per down workgroup
    int ncol = 0;        // column tiles
    int slices = 0;      // K-slices per column tile (down partial sums)
    int slice_units = 0; // bf16: 32-neuron chunks per slice; f32: neurons per slice
    // bf16, lists of at most kDfMaxChunks chunks: the down projection runs fused (one workgroup per column tile and token tile sums the whole list and applies the residual
    // itself: no partials, no epilogue launch).
    bool fused_down = false;
    int dn_cpw = 0;      // fused down: chunks per wave (the kernel's unrolled pipeline depth)
    int df_nt = 1;       // fused down: 16-token tiles per workgroup (4 with several samples)
    int df_cw = 4;       // fused down: columns per lane (2 for one sample, 4 with several)
    int df_ncol = 0;     // fused down: column tiles of 16 df_cw columns
    int ntt = 0;         // fused down: token tiles of 16 df_nt tokens
    // bf16, one sample, d = 2048, the spread plan's list lengths, 256 compute units: gate/up and down in one
    // launch (layer_xcd_kernel) that reads the float32 input itself, slices = the 8 XCDs' slices of slice_units
    // chunks; no prologue launch, the epilogue follows.
    bool xcd_layer = false;
    // Workspace: xn [B][T][d] (bf16 or f32); H (bf16: [B][kcap / 32][tpad][32], chunk-major; f32:
    // [B][tpad][kcap]); partials f32 [B][slices][T][d]; ssq f32 [B][T][ssq_stride(d)]
    // (per-token sums of squares of the FFN input by 32-column block, for the RMSNorm factor); and, for the dense
    // reference, the lists 0 .. d_ff-1 int32 [B][d_ff] and their counts int32 [B].
    // With xcd_layer, also the XCDs' own copies of the FFN input, bf16 [8][T][d], and of its partial sums of
    // squares, f32 [8][T][ssq_stride(d)], and the meetings' flags and counters (kXcdFlagBytes + kXcdCtrBytes; no
    // initialization needed).
    size_t off_xn = 0, off_h = 0, off_part = 0, off_ssq = 0, off_ident = 0, off_ident_count = 0, off_xn8 = 0,
           off_ssq8 = 0, off_sync = 0, total = 0;
};

// form: the kind of call the plan is for, 0 (a single layer on given lists) or a sum of the flags below; it
// decides whether the one-launch layer form pays (the workspace size does not depend on it).
constexpr unsigned kFormStack = 1;  // several layers
constexpr unsigned kFormMask = 2;   // the call compacts masks
rm_status make_plan(const rm_ffn_shape *s, int B, int T, int max_count, Plan *p, unsigned form = 0);

// ---------------------------------------------------------------------------------------------------------
// Launchers (enqueue only; all arguments already validated).
// ---------------------------------------------------------------------------------------------------------

hipError_t launch_mask_compact(const uint8_t *mask, int n_masks, int d_ff, int32_t *idx, int32_t *count,
                               hipStream_t st);

// Compact copies of the listed rows of L layers' three matrices: out [L][3][max_count][d] (gather_rows.hip).
hipError_t launch_gather_rows(const rm_ffn_layer_weights *w, const int32_t *idx, const int32_t *count, int d_ff,
                              int d, int wdtype, int max_count, int L, void *out, hipStream_t st);

// Context Cache (context_cache.hip).  Workspace plan: the gathered rows as bf16 [m_pad][d], then H bf16
// [m_pad][d_ff] (both in the GEMMs' blocked layout), then the down GEMM's K-slice partials; m_pad = max_rows
// rounded up to the row tile.  GEMM tiles: 256 rows by 8 waves (4 along the rows x 2 along the columns), each wave
// 64 rows x 64 columns per weight matrix; the gate/up tile spans 128 neurons of both matrices, the down tile 128
// output columns (64 when d is not a multiple of 128).  The stage counts and the down GEMM's workgroup target can
// be set at build time (RM_CTX_GLU_STAGES, RM_CTX_DOWN_STAGES, RM_CTX_DOWN_TARGET) for tuning sweeps.
#ifndef RM_CTX_GLU_STAGES
#define RM_CTX_GLU_STAGES 2
#endif
#ifndef RM_CTX_DOWN_STAGES
#define RM_CTX_DOWN_STAGES 3
#endif
#ifndef RM_CTX_DOWN_TARGET
#define RM_CTX_DOWN_TARGET 256
#endif
constexpr int kCtxBM = 256;                         // rows per tile; the padded row count is a multiple
constexpr int kCtxGluBN = 128;                      // gate/up: neurons per tile
constexpr int kCtxDownTarget = RM_CTX_DOWN_TARGET;  // down: workgroups the K split aims for
inline int ctx_down_bn(int d) { return d % 128 == 0 ? 128 : 64; }
struct ContextPlan {
    int d = 0, d_ff = 0, act = 0, n_tok = 0, max_rows = 0, m_pad = 0;
    int down_bn = 128;    // output columns per down tile
    int down_splits = 1;  // K slices of the down GEMM (float32 partials [splits][m_pad][d] when > 1)
    size_t off_a = 0, off_h = 0, off_part = 0, total = 0;
};
hipError_t launch_context_select(const float *x, const float *x_ref, int n_tok, int d, int v0, int P, int k,
                                 float *drift, int32_t *rows, int32_t *count, hipStream_t st);
// blocked: the three weight matrices come in the blocked layout written by launch_pack_blocked.
hipError_t launch_context_ffn(const ContextPlan &p, const void *w_gate, const void *w_up, const void *w_down_t,
                              bool blocked, const float *x, const int32_t *rows, const int32_t *count, float *y,
                              void *ws, hipStream_t st);
// A row-major bf16 [R][K] matrix (R, K multiples of 64) into the blocked layout of the context GEMMs.
hipError_t launch_pack_blocked(const void *src, int R, int K, void *dst, hipStream_t st);

// Group neuron masks (group_mask.hip): the down rows' norms, and Eq. 1 scores + per-step top-K + union + rerank.
constexpr int kGroupMaxDff = 16384;
hipError_t launch_neuron_norms(const void *w_down, int d_ff, int d, int wdtype, float *norms, hipStream_t st);
hipError_t launch_group_masks(const float *h, int S, int L, int d_ff, int T, const float *norms, int k,
                              float *scores, uint8_t *mask, hipStream_t st);

// Index lists 0 .. d_ff-1 and counts d_ff for every sample in the workspace (the dense reference runs the
// sparse kernels on them).
hipError_t launch_identity_lists(const Plan &p, void *ws, hipStream_t st);

// First layer's FFN input: xn = x * g (or x) in the FFN input dtype, and (norm only) its per-token sums of
// squares.
hipError_t launch_prologue(const Plan &p, const float *x, const float *norm_g, void *ws, hipStream_t st);

// rm_mask_compact of n_masks masks and launch_prologue in one launch.
hipError_t launch_compact_prologue(const Plan &p, const uint8_t *mask, int n_masks, int32_t *idx, int32_t *count,
                                   const float *x, const float *norm_g, void *ws, hipStream_t st);

// Gate/up projection of the listed neurons + SiLU * up -> H in the workspace.  norm: scale by the per-token
// RMSNorm factor formed from the workspace's sums of squares.
// Eq. 4 (both optional, [B][max_count][T] float32): h_anchor is subtracted from h before it goes into H (a
// delta step); with h_out, h of the listed slots is written there instead of H (capturing an anchor's h^M).
hipError_t launch_gateup_bf16(const Plan &p, const void *w_gate, const void *w_up, const int32_t *idx,
                              const int32_t *count, bool norm, const float *h_anchor, float *h_out, void *ws,
                              hipStream_t st);
hipError_t launch_gateup_f32(const Plan &p, const void *w_gate, const void *w_up, const int32_t *idx,
                             const int32_t *count, bool norm, const float *h_anchor, float *h_out, void *ws,
                             hipStream_t st);

// Down projection of the listed neurons: per-K-slice float32 partials of H W_down[idx] in the workspace.  The
// bf16 form needs no count: H is zero in every slot past the list.
hipError_t launch_down_bf16(const Plan &p, const void *w_down, const int32_t *idx, void *ws, hipStream_t st);
// With p.fused_down: the down projection and the epilogue's work in one launch (same results as
// launch_down_bf16 + launch_epilogue up to the order of the K sum).
hipError_t launch_down_fused(const Plan &p, const void *w_down, const int32_t *idx, const int32_t *count,
                             const float *x, float *y, const float *g_next, bool emit_xn, const float *ya_in,
                             float *ya_out, const float *out_gate, void *ws, hipStream_t st);
// With p.xcd_layer: the gate/up and the down projection in one launch that reads the float32 FFN input xin
// [T][d] and the norm gain (null: no norm) itself, so no prologue precedes it; it leaves per-slice partials, as
// launch_down_bf16 writes them, for launch_epilogue (which need not emit the next layer's xn).
hipError_t launch_layer_xcd(const Plan &p, const void *w_gate, const void *w_up, const void *w_down,
                            const int32_t *idx, const int32_t *count, const float *xin, const float *norm_g,
                            const float *h_anchor, void *ws, hipStream_t st);
hipError_t launch_down_f32(const Plan &p, const void *w_down, const int32_t *idx, const int32_t *count, void *ws,
                           hipStream_t st);

// y = x + the slices' partials in slice order; if emit_xn, also the next layer's FFN input (y * g_next, or y)
// and, with g_next, its per-token sums of squares.  Eq. 4 (optional, [B][T][d] float32): y = x + (ya_in +
// partials) on a delta step; ya_out receives the partials' sum (the FFN output) on an anchor step.  out_gate
// (optional, [B][d]) multiplies the FFN part before the residual.
hipError_t launch_epilogue(const Plan &p, const int32_t *count, const float *x, float *y, const float *g_next,
                           bool emit_xn, const float *ya_in, float *ya_out, const float *out_gate, void *ws,
                           hipStream_t st);

// Streaming read of bytes (a multiple of 16) of buf by `workgroups` workgroups of 512 threads (measure.hip).
hipError_t launch_stream_read(const void *buf, size_t bytes, int workgroups, uint32_t *sink, hipStream_t st);

// Profiling hook: the events armed by rm_profile_kernel_events for the next launch of `kernel` by this thread
// (null when disarmed), which are disarmed by taking them.
void profile_take(int kernel, hipEvent_t *begin, hipEvent_t *end);

// Launch of a gate/up or down kernel: with armed events through hipExtLaunchKernel, which records the kernel's
// own start and end time (the interval a kernel trace reports), else a plain launch.
template <typename... Params, typename... Args>
inline hipError_t launch_timed(int kernel, void (*fn)(Params...), dim3 grid, dim3 block, hipStream_t st,
                               Args... args) {
    static_assert(sizeof...(Params) == sizeof...(Args), "kernel argument count");
    hipEvent_t b = nullptr, e = nullptr;
    profile_take(kernel, &b, &e);
    std::tuple<Params...> conv{args...};  // the kernel's own parameter types
    return std::apply(
        [&](auto &...v) {
            void *argv[] = {static_cast<void *>(&v)...};
            if (b != nullptr || e != nullptr)
                return hipExtLaunchKernel(reinterpret_cast<const void *>(fn), grid, block, argv, 0, st, b, e, 0);
            return hipLaunchKernel(reinterpret_cast<const void *>(fn), grid, block, argv, 0, st);
        },
        conv);
}

}  // namespace rm

// ---------------------------------------------------------------------------------------------------------
// Device helpers
// ---------------------------------------------------------------------------------------------------------

typedef __bf16 rm_bf16x8 __attribute__((ext_vector_type(8)));
typedef float rm_f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t rm_u32x4 __attribute__((ext_vector_type(4)));

// float -> bfloat16 bits, round to nearest even (NaN stays a quiet NaN).
__device__ __forceinline__ uint32_t rm_f32_to_bf16_bits(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0u;
    return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ float rm_bf16_bits_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

// 1 / sqrt(mean of squares + eps) from a row's summed squares.
__device__ __forceinline__ float rm_rnorm_from_ssq(float s, int d, float eps) {
    return 1.0f / sqrtf(s / static_cast<float>(d) + eps);
}

// A row's partial sums of squares are added in two levels: the 8 partials of each 256-column span in order (the
// span's sum), then the spans' sums in order; a row whose d is not a multiple of 256 ends with a shorter span.
// Kernels whose waves each hold one span add the spans in parallel and only the spans' sums in sequence.
constexpr int kSsqSpan = 8;  // partials per span

// The sum of one whole span's 8 partials, lo = partials 0-3, hi = 4-7.
__device__ __forceinline__ float rm_ssq_span(float4 lo, float4 hi) {
    float s = lo.x;
    s += lo.y;
    s += lo.z;
    s += lo.w;
    s += hi.x;
    s += hi.y;
    s += hi.z;
    s += hi.w;
    return s;
}

// RMSNorm factor of token row `row` (= b * T + t): 1 / sqrt(mean of squares + eps), from the row's partial sums
// of squares by 32-column block, added in the two-level order above.
__device__ __forceinline__ float rm_token_rnorm(const float *ssq, int row, int d, float eps) {
    const int n = rm::ssq_parts(d);
    const int stride4 = rm::ssq_stride(d) / 4;
    const float4 *p = reinterpret_cast<const float4 *>(ssq + static_cast<size_t>(row) * rm::ssq_stride(d));
    float s = 0.0f;  // + the first span's sum: exact
    for (int k0 = 0; k0 < n; k0 += 4 * kSsqSpan) {  // four spans: eight float4 loads in flight, then the sums
        float4 v[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = p[min(k0 / 4 + i, stride4 - 1)];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int k = k0 + j * kSsqSpan;
            if (k >= n) break;
            if (k + kSsqSpan <= n) {
                s += rm_ssq_span(v[2 * j], v[2 * j + 1]);
            } else {  // the row's last, shorter span
                const float part[8] = {v[2 * j].x,     v[2 * j].y,     v[2 * j].z,     v[2 * j].w,
                                       v[2 * j + 1].x, v[2 * j + 1].y, v[2 * j + 1].z, v[2 * j + 1].w};
                float b = part[0];
                for (int i = 1; i < n - k; ++i) b += part[i];
                s += b;
            }
        }
    }
    return rm_rnorm_from_ssq(s, d, eps);
}

// Sum of squares of a 32-column block, in one fixed order shared by every kernel that writes the partials, so
// that a layer's norm factors do not depend on which kernel produced its input: per pair of columns
// fma(c1, c1, fma(c0, c0, 0)), per group of 4 columns the sum of its two pairs, then the 8 groups of the block
// added by a lane butterfly (xor 1, 2, 4 over the groups).  rm_ssq32: lanes 8 k .. 8 k + 7 hold the block's 32
// columns, 4 per lane (ok: the lane's columns lie inside the row).
__device__ __forceinline__ float rm_ssq32(float4 v, bool ok) {
    float ss = 0.0f;
    if (ok) ss = fmaf(v.y, v.y, fmaf(v.x, v.x, 0.0f)) + fmaf(v.w, v.w, fmaf(v.z, v.z, 0.0f));
    for (int off = 1; off < 8; off <<= 1) ss += __shfl_xor(ss, off);
    return ss;
}
// The same block with 2 columns per lane, lanes 16 k .. 16 k + 15: lanes 2 g and 2 g + 1 hold group g's two pairs
// (their sum is the group's, the same bits in both lanes), then the butterfly over the groups (xor 2, 4, 8).
__device__ __forceinline__ float rm_ssq32_pairs(float x, float y, bool ok) {
    const float p = ok ? fmaf(y, y, fmaf(x, x, 0.0f)) : 0.0f;
    float ss = p + __shfl_xor(p, 1);
    for (int off = 2; off < 16; off <<= 1) ss += __shfl_xor(ss, off);
    return ss;
}

// SiLU(z) = z / (1 + e^-z); e^-z overflows to +inf for very negative z, giving -0, never NaN.
__device__ __forceinline__ float rm_silu(float z) { return z / (1.0f + expf(-z)); }

// GELU, tanh form: 0.5 z (1 + tanh(sqrt(2/pi) (z + 0.044715 z^3))); tanh saturates, so large |z| gives z or -0.
__device__ __forceinline__ float rm_gelu_tanh(float z) {
    return 0.5f * z * (1.0f + tanhf(0.7978845608028654f * (z + 0.044715f * z * z * z)));
}

// The gated linear unit's activation (act: an rm_act).
__device__ __forceinline__ float rm_glu_act(int act, float z) {
    return act == RM_ACT_GELU_TANH ? rm_gelu_tanh(z) : rm_silu(z);
}
