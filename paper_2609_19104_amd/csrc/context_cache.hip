// Context Cache: visual-token recomputation of a VLM FFN layer (paper section 4.1, "Visual-Token Recomputation",
// Eq. 2 and Eq. 3).
//
// The token rows of a layer's FFN input x (after RMSNorm, float32 [N][d]) whose visual tokens are rows
// [v0, v0 + P):
//   drift_kernel:          Eq. 2 for each visual row, d_p = RMS(x_p - xbar_p) / max(RMS(x_p), 1e-6), one wave
//                          per row.  The top-k decision below depends on it, so it has a fixed float32 order: lane j
//                          adds the squares of columns j, j + 64, ... one rounding per operation, the 64 lane sums
//                          are folded 32, 16, ..., 1 apart, then rounded division and correctly rounded roots.
//   select_rows_kernel:    one 1024-thread workgroup: the k visual rows with the largest drift (radix select, ties
//                          to the lower token) plus every non-visual row, as an ascending row list and its count.
//   gather_rows_kernel:    the listed rows of x as bf16 into the workspace, zero rows up to the padded count.
//   gemm_nt_kernel<GLU>:   H = act(A W_gate^T) * (A W_up^T), bf16 [rows][d_ff].
//   gemm_nt_kernel<SCAT>:  y[row_i] = H_i W_down^T (W_down as nn.Linear's [d][d_ff]): Eq. 3's recomputed rows
//                          written into the caller's buffer, which holds the reference outputs everywhere else.
//                          With K = d_ff long and few output tiles, the down product is split over K instead
//                          (<PART>: float32 partials per K slice) and reduce_scatter_kernel adds the slices in
//                          order into the listed rows of y (no atomics).
//
// The two projections are dense contractions with enough reuse for the matrix cores (about 400 rows against
// 2048 x 16384 weights: 390 FLOP per weight byte, above the bf16 ridge of MI355X), so both run on
// v_mfma_f32_16x16x32_bf16 with both operands contiguous along K: a workgroup of 4 waves owns a BM x BN tile,
// stages 64-wide K slices of A and B through double-buffered LDS (16-byte loads, padded rows), and each wave
// accumulates a (BM/2) x (BN/2) quarter (for the gate/up product, one accumulator set per matrix).  Workgroups
// that share a weight tile are numbered onto one XCD so that its L2 serves the re-reads.
#include "rm_select.h"

namespace {

using rm_sel::kSelPerThread;
using rm_sel::kSelThreads;
using rm_sel::mul_rounded;
using rm_sel::select_top_k;
using rm_sel::SelLds;

typedef __bf16 ctx_bf16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ rm_f32x4 mfma16(rm_u32x4 a, rm_u32x4 b, rm_f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(ctx_bf16x8, a),
                                                   __builtin_bit_cast(ctx_bf16x8, b), c, 0, 0, 0);
}

// Workgroup numbering so that consecutive logical ids share an XCD (workgroup i runs on XCD i mod 8).
__device__ __forceinline__ int xcd_order(int id, int n) {
    const int a = n >> 3, r = n & 7, x = id & 7;
    return x * a + min(x, r) + (id >> 3);
}

// ------------------------------------------------------------------------------------------ Eq. 2

__global__ __launch_bounds__(64) void drift_kernel(const float *__restrict__ x, const float *__restrict__ xr, int d,
                                                   int v0, float *__restrict__ drift) {
    const int p = blockIdx.x;
    const int lane = threadIdx.x;
    const float *xa = x + static_cast<size_t>(v0 + p) * d;
    const float *xb = xr + static_cast<size_t>(v0 + p) * d;
    float sd = 0.0f, sx = 0.0f;
    // Eight columns of each input in flight per lane before the in-order sums (columns past d are not added).
    for (int c0 = lane; c0 < d; c0 += 8 * 64) {
        float va[8], vb[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int c = min(c0 + u * 64, d - 1);
            va[u] = xa[c];
            vb[u] = xb[c];
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            if (c0 + u * 64 >= d) break;
            const float diff = __fsub_rn(va[u], vb[u]);
            sd = __fadd_rn(sd, mul_rounded(diff, diff));
            sx = __fadd_rn(sx, mul_rounded(va[u], va[u]));
        }
    }
    for (int off = 32; off >= 1; off >>= 1) {
        sd = __fadd_rn(sd, __shfl_xor(sd, off));
        sx = __fadd_rn(sx, __shfl_xor(sx, off));
    }
    if (lane == 0) {
        const float fd = static_cast<float>(d);
        const float rd = __builtin_sqrtf(__fdiv_rn(sd, fd));
        const float rx = __builtin_sqrtf(__fdiv_rn(sx, fd));
        drift[p] = __fdiv_rn(rd, fmaxf(rx, 1e-6f));
    }
}

// ------------------------------------------------------------------------------------------ row selection

__global__ __launch_bounds__(kSelThreads) void select_rows_kernel(const float *__restrict__ drift, int n_tok, int v0,
                                                                  int P, int k, int32_t *__restrict__ rows,
                                                                  int32_t *__restrict__ count) {
    __shared__ SelLds l;
    __shared__ uint8_t chosen[kSelThreads * kSelPerThread];
    const int tid = threadIdx.x;
    const int p0 = tid * kSelPerThread;
    uint32_t valid = 0, key[kSelPerThread];
#pragma unroll
    for (int i = 0; i < kSelPerThread; ++i) {
        const bool ok = p0 + i < P;
        if (ok) valid |= 1u << i;
        key[i] = ok ? __float_as_uint(drift[p0 + i]) : 0u;  // drift >= 0: its bits order like its value
    }
    const uint32_t sel = select_top_k(key, valid, k, P, l);
#pragma unroll
    for (int i = 0; i < kSelPerThread; ++i) chosen[p0 + i] = static_cast<uint8_t>((sel >> i) & 1u);
    __syncthreads();
    // Rows tid * 16 .. tid * 16 + 15 of the sequence, in order.
    const int r0 = tid * kSelPerThread;
    uint32_t take = 0;
#pragma unroll
    for (int i = 0; i < kSelPerThread; ++i) {
        const int r = r0 + i;
        const bool visual = r >= v0 && r < v0 + P;
        if (r < n_tok && (!visual || chosen[r - v0])) take |= 1u << i;
    }
    int pos = rm_sel::block_excl_scan(__popc(take), l);
#pragma unroll
    for (int i = 0; i < kSelPerThread; ++i)
        if ((take >> i) & 1u) rows[pos++] = r0 + i;
    if (tid == kSelThreads - 1) count[0] = pos;  // the last thread's end is the total
}

// ------------------------------------------------------------------------------------------ gather

__global__ __launch_bounds__(256) void gather_rows_kernel(const float *__restrict__ x, int d,
                                                          const int32_t *__restrict__ rows,
                                                          const int32_t *__restrict__ count, int max_rows, int m_pad,
                                                          int n_tok, uint16_t *__restrict__ A) {
    const int i = blockIdx.x * 4 + (threadIdx.x >> 6);  // one wave per row
    const int lane = threadIdx.x & 63;
    if (i >= m_pad) return;
    const int cnt = min(max(count[0], 0), max_rows);
    uint16_t *dst = A + static_cast<size_t>(i) * d;
    if (i >= cnt) {
        for (int c = lane * 4; c < d; c += 256) *reinterpret_cast<uint2 *>(dst + c) = make_uint2(0u, 0u);
        return;
    }
    const int r = min(max(rows[i], 0), n_tok - 1);
    const float *src = x + static_cast<size_t>(r) * d;
    for (int c = lane * 4; c < d; c += 256) {
        const float4 v = *reinterpret_cast<const float4 *>(src + c);
        uint2 packed;
        packed.x = rm_f32_to_bf16_bits(v.x) | (rm_f32_to_bf16_bits(v.y) << 16);
        packed.y = rm_f32_to_bf16_bits(v.z) | (rm_f32_to_bf16_bits(v.w) << 16);
        *reinterpret_cast<uint2 *>(dst + c) = packed;
    }
}

// ------------------------------------------------------------------------------------------ GEMM

enum { kEpiGlu = 0, kEpiScatter = 1, kEpiPartial = 2 };

struct GemmArgs {
    const uint16_t *A;       // bf16 [m_pad][K]
    const uint16_t *B0, *B1; // bf16 [N][K] (B1: the up matrix of the gate/up product)
    int K, N, m_pad;
    const int32_t *count;    // rows of A in use (device), clamped to [0, max_rows]
    int max_rows, act;
    uint16_t *H;             // kEpiGlu: bf16 [m_pad][N]
    float *y;                // kEpiScatter: float32 [n_tok][N], row rows[i] receives output row i
    const int32_t *rows;
    int n_tok;
    int splits;              // K slices (workgroups per output tile); kEpiPartial: slice s writes part[s]
    float *part;             // kEpiPartial: float32 [splits][m_pad][N]
};

constexpr int kKt = 64;          // K per LDS stage (two matrix-core steps)
constexpr int kPitch = kKt + 8;  // bf16 per LDS row: 16 bytes of padding against bank conflicts

template <int BM, int BN, int NB, int EPI>
__global__ __launch_bounds__(256) void gemm_nt_kernel(GemmArgs a) {
    constexpr int WM = BM / 2, WN = BN / 2, TM = WM / 16, TN = WN / 16;
    constexpr int A_PIECES = BM * kKt / 8 / 256;       // 16-byte pieces per thread and stage
    constexpr int B_PIECES = NB * BN * kKt / 8 / 256;
    static_assert(A_PIECES >= 1 && B_PIECES >= 1, "tile too small for 256 threads");
    __shared__ __attribute__((aligned(16))) uint16_t As[2][BM * kPitch];
    __shared__ __attribute__((aligned(16))) uint16_t Bs[2][NB * BN * kPitch];

    const int mt = a.m_pad / BM;
    const int q = xcd_order(blockIdx.x, gridDim.x);  // = (n tile * splits + K slice) * mt + m tile
    const int m0 = (q % mt) * BM;
    const int ks_id = (q / mt) % a.splits;
    const int n0 = (q / mt / a.splits) * BN;
    const int k_len = a.K / a.splits;  // a multiple of kKt
    const int k_base = ks_id * k_len;
    const int cnt = min(max(a.count[0], 0), a.max_rows);
    if (m0 >= cnt) return;  // the whole tile is past the rows in use

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave & 1, wn = wave >> 1;
    const int r = lane & 15, grp = lane >> 4;

    rm_u32x4 ra[A_PIECES], rb[B_PIECES];
    auto load_stage = [&](int k0) {
#pragma unroll
        for (int p = 0; p < A_PIECES; ++p) {
            const int e = tid + p * 256;
            ra[p] = *reinterpret_cast<const rm_u32x4 *>(a.A + static_cast<size_t>(m0 + (e >> 3)) * a.K + k_base + k0 +
                                                       (e & 7) * 8);
        }
#pragma unroll
        for (int p = 0; p < B_PIECES; ++p) {
            const int e = tid + p * 256;
            const int nb = e / (BN * 8);
            const int rem = e - nb * BN * 8;
            const uint16_t *B = nb ? a.B1 : a.B0;
            rb[p] = *reinterpret_cast<const rm_u32x4 *>(B + static_cast<size_t>(n0 + (rem >> 3)) * a.K + k_base + k0 +
                                                       (rem & 7) * 8);
        }
    };
    auto store_stage = [&](int buf) {
#pragma unroll
        for (int p = 0; p < A_PIECES; ++p) {
            const int e = tid + p * 256;
            *reinterpret_cast<rm_u32x4 *>(&As[buf][(e >> 3) * kPitch + (e & 7) * 8]) = ra[p];
        }
#pragma unroll
        for (int p = 0; p < B_PIECES; ++p) {
            const int e = tid + p * 256;
            *reinterpret_cast<rm_u32x4 *>(&Bs[buf][(e >> 3) * kPitch + (e & 7) * 8]) = rb[p];
        }
    };

    rm_f32x4 acc[NB][TM][TN];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int tm = 0; tm < TM; ++tm)
#pragma unroll
            for (int tn = 0; tn < TN; ++tn) acc[nb][tm][tn] = rm_f32x4{0.f, 0.f, 0.f, 0.f};

    const int nk = k_len / kKt;
    load_stage(0);
    store_stage(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        const bool more = kt + 1 < nk;
        if (more) load_stage((kt + 1) * kKt);  // in flight while this stage's products run
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            rm_u32x4 af[TM], bf[NB][TN];
#pragma unroll
            for (int tm = 0; tm < TM; ++tm)
                af[tm] = *reinterpret_cast<const rm_u32x4 *>(
                    &As[buf][(wm * WM + tm * 16 + r) * kPitch + ks * 32 + grp * 8]);
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                for (int tn = 0; tn < TN; ++tn)
                    bf[nb][tn] = *reinterpret_cast<const rm_u32x4 *>(
                        &Bs[buf][(nb * BN + wn * WN + tn * 16 + r) * kPitch + ks * 32 + grp * 8]);
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                for (int tm = 0; tm < TM; ++tm)
#pragma unroll
                    for (int tn = 0; tn < TN; ++tn) acc[nb][tm][tn] = mfma16(af[tm], bf[nb][tn], acc[nb][tm][tn]);
        }
        if (more) store_stage(buf ^ 1);  // buf ^ 1 was last read before the previous barrier
        __syncthreads();
    }

    // Lane (grp, r), register i of a tile: row 4 grp + i, column r.
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int m = m0 + wm * WM + tm * 16 + grp * 4 + i;
            if (m >= cnt) continue;
#pragma unroll
            for (int tn = 0; tn < TN; ++tn) {
                const int n = n0 + wn * WN + tn * 16 + r;
                if constexpr (EPI == kEpiGlu) {
                    const float h = rm_glu_act(a.act, acc[0][tm][tn][i]) * acc[NB - 1][tm][tn][i];
                    a.H[static_cast<size_t>(m) * a.N + n] = static_cast<uint16_t>(rm_f32_to_bf16_bits(h));
                } else if constexpr (EPI == kEpiPartial) {
                    a.part[(static_cast<size_t>(ks_id) * a.m_pad + m) * a.N + n] = acc[0][tm][tn][i];
                } else {
                    const int row = min(max(a.rows[m], 0), a.n_tok - 1);
                    a.y[static_cast<size_t>(row) * a.N + n] = acc[0][tm][tn][i];
                }
            }
        }
    }
}

// y[rows[i]] = the K slices' partials of output row i, added in slice order (one thread per 4 columns).
__global__ __launch_bounds__(256) void reduce_scatter_kernel(const float *__restrict__ part, int splits, int m_pad,
                                                             int N, const int32_t *__restrict__ rows,
                                                             const int32_t *__restrict__ count, int max_rows,
                                                             int n_tok, float *__restrict__ y) {
    const int cnt = min(max(count[0], 0), max_rows);
    const int per_row = N / 4;
    const long long e = static_cast<long long>(blockIdx.x) * 256 + threadIdx.x;
    const int i = static_cast<int>(e / per_row);
    if (i >= cnt) return;
    const int c = static_cast<int>(e - static_cast<long long>(i) * per_row) * 4;
    float4 s = *reinterpret_cast<const float4 *>(part + static_cast<size_t>(i) * N + c);
    for (int k = 1; k < splits; ++k) {
        const float4 v = *reinterpret_cast<const float4 *>(part + (static_cast<size_t>(k) * m_pad + i) * N + c);
        s = make_float4(s.x + v.x, s.y + v.y, s.z + v.z, s.w + v.w);
    }
    const int row = min(max(rows[i], 0), n_tok - 1);
    *reinterpret_cast<float4 *>(y + static_cast<size_t>(row) * N + c) = s;
}

}  // namespace

namespace rm {

hipError_t launch_context_select(const float *x, const float *x_ref, int n_tok, int d, int v0, int P, int k,
                                 float *drift, int32_t *rows, int32_t *count, hipStream_t st) {
    if (P > 0) {
        hipLaunchKernelGGL(drift_kernel, dim3(P), dim3(64), 0, st, x, x_ref, d, v0, drift);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(select_rows_kernel, dim3(1), dim3(kSelThreads), 0, st, static_cast<const float *>(drift),
                       n_tok, v0, P, k, rows, count);
    return hipGetLastError();
}

hipError_t launch_context_ffn(const ContextPlan &p, const void *w_gate, const void *w_up, const void *w_down_t,
                              const float *x, const int32_t *rows, const int32_t *count, float *y, void *ws,
                              hipStream_t st) {
    char *base = static_cast<char *>(ws);
    uint16_t *A = reinterpret_cast<uint16_t *>(base + p.off_a);
    uint16_t *H = reinterpret_cast<uint16_t *>(base + p.off_h);
    hipLaunchKernelGGL(gather_rows_kernel, dim3((p.m_pad + 3) / 4), dim3(256), 0, st, x, p.d, rows, count,
                       p.max_rows, p.m_pad, p.n_tok, A);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;

    GemmArgs g{};
    g.A = A;
    g.B0 = static_cast<const uint16_t *>(w_gate);
    g.B1 = static_cast<const uint16_t *>(w_up);
    g.K = p.d;
    g.N = p.d_ff;
    g.m_pad = p.m_pad;
    g.count = count;
    g.max_rows = p.max_rows;
    g.act = p.act;
    g.H = H;
    g.splits = 1;
    launch_timed(RM_KERNEL_GATEUP, gemm_nt_kernel<kCtxGluBM, kCtxGluBN, 2, kEpiGlu>,
                 dim3((p.m_pad / kCtxGluBM) * (p.d_ff / kCtxGluBN)), dim3(256), st, g);
    e = hipGetLastError();
    if (e != hipSuccess) return e;

    GemmArgs o{};
    o.A = H;
    o.B0 = static_cast<const uint16_t *>(w_down_t);
    o.B1 = o.B0;
    o.K = p.d_ff;
    o.N = p.d;
    o.m_pad = p.m_pad;
    o.count = count;
    o.max_rows = p.max_rows;
    o.y = y;
    o.rows = rows;
    o.n_tok = p.n_tok;
    o.splits = p.down_splits;
    const dim3 grid((p.m_pad / kCtxDownBM) * (p.d / kCtxDownBN) * p.down_splits);
    if (p.down_splits == 1) {
        launch_timed(RM_KERNEL_DOWN, gemm_nt_kernel<kCtxDownBM, kCtxDownBN, 1, kEpiScatter>, grid, dim3(256), st, o);
        return hipGetLastError();
    }
    // Split over K: the slices' float32 partials, then their ordered sum scattered into y.
    o.part = reinterpret_cast<float *>(base + p.off_part);
    launch_timed(RM_KERNEL_DOWN, gemm_nt_kernel<kCtxDownBM, kCtxDownBN, 1, kEpiPartial>, grid, dim3(256), st, o);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const long long n4 = static_cast<long long>(p.max_rows) * (p.d / 4);
    hipLaunchKernelGGL(reduce_scatter_kernel, dim3(static_cast<unsigned>((n4 + 255) / 256)), dim3(256), 0, st,
                       static_cast<const float *>(o.part), p.down_splits, p.m_pad, p.d, rows, count, p.max_rows,
                       p.n_tok, y);
    return hipGetLastError();
}

}  // namespace rm
