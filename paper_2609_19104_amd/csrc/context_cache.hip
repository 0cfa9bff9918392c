// Context Cache: visual-token recomputation of a VLM FFN layer (paper section 4.1, "Visual-Token Recomputation",
// Eq. 2 and Eq. 3).
//
// The token rows of a layer's FFN input x (after RMSNorm, float32 [N][d]) whose visual tokens are rows
// [v0, v0 + P):
//   drift_kernel:          Eq. 2 for each visual row, d_p = RMS(x_p - xbar_p) / max(RMS(x_p), 1e-6), one wave
//                          per row.  The top-k decision below depends on it, so it has a fixed float32 order: lane j
//                          adds the squares of columns j, j + 64, ... one rounding per operation, the 64 lane sums
//                          are folded 32, 16, ..., 1 apart, then rounded division and correctly rounded roots.
//   select_rows_kernel:    one workgroup (256 threads up to 4096 rows, else 1024): the k visual rows with the
//                          largest drift (radix select, ties to the lower token) plus every non-visual row, as an
//                          ascending row list and its count.
//   gather_rows_kernel:    the listed rows of x as bf16 into the workspace, zero rows up to the padded count.
//   gemm_dma_kernel<GLU>:  H = act(A W_gate^T) * (A W_up^T), bf16 [rows][d_ff].
//   gemm_dma_kernel<SCAT>: y[row_i] = H_i W_down^T (W_down as nn.Linear's [d][d_ff]): Eq. 3's recomputed rows
//                          written into the caller's buffer, which holds the reference outputs everywhere else.
//                          With K = d_ff long and few output tiles, the down product is split over K instead
//                          (<PART>: float32 partials per K slice) and reduce_scatter_kernel adds the slices in
//                          order into the listed rows of y (no atomics).
//
// The two projections are dense contractions with enough reuse for the matrix cores (about 400 rows against
// 2048 x 16384 weights: 390 FLOP per weight byte, above the bf16 ridge of MI355X), so both run on
// v_mfma_f32_16x16x32_bf16 with both operands contiguous along K.  On this shape the limit is how fast a compute
// unit pulls tiles out of L2, not the matrix cores, so the tiles are as large as one workgroup per compute unit
// allows: 256 rows by 128 columns of each weight matrix (2 MB read per gate/up workgroup over K = 2048), 8 waves
// each accumulating 64 x 64 per matrix, K staged 64 wide (one cache line per row) straight from memory into LDS.
// Workgroups that share a weight tile are numbered onto one XCD so that its L2 serves the re-reads.
#include "rm_select.h"

namespace {

using rm_sel::kSelPerThread;
using rm_sel::kSelThreads;
using rm_sel::kSelThreadsSmall;
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
    // kDriftCols columns of each input in flight per lane (all of a 2048-wide row in one round trip) before the
    // in-order sums; columns past d are not added.
    constexpr int kDriftCols = 32;
    for (int c0 = lane; c0 < d; c0 += kDriftCols * 64) {
        float va[kDriftCols], vb[kDriftCols];
#pragma unroll
        for (int u = 0; u < kDriftCols; ++u) {
            const int c = min(c0 + u * 64, d - 1);
            va[u] = xa[c];
            vb[u] = xb[c];
        }
        // No branch between the loads and the sums (a branch lets the compiler sink each load to its use, one
        // round trip per column): a column past d adds +0, which leaves the non-negative sums unchanged.
#pragma unroll
        for (int u = 0; u < kDriftCols; ++u) {
            const bool in = c0 + u * 64 < d;
            const float diff = __fsub_rn(va[u], vb[u]);
            sd = __fadd_rn(sd, in ? mul_rounded(diff, diff) : 0.0f);
            sx = __fadd_rn(sx, in ? mul_rounded(va[u], va[u]) : 0.0f);
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

template <int kThreads>
__global__ __launch_bounds__(kThreads) void select_rows_kernel(const float *__restrict__ drift, int n_tok, int v0,
                                                               int P, int k, int32_t *__restrict__ rows,
                                                               int32_t *__restrict__ count) {
    __shared__ SelLds<kThreads> l;
    __shared__ uint8_t chosen[kThreads * kSelPerThread];
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
    if (tid == kThreads - 1) count[0] = pos;  // the last thread's end is the total
}

// ------------------------------------------------------------------------------------------ blocked layout

// The GEMM operands live in a blocked layout: a bf16 matrix [R][K] (R and K multiples of 64) as 64-row x 64-column
// blocks of 8 KB, the blocks of one 64-row tile consecutive along K.  Inside a block, row r holds its 64 columns
// (128 bytes) as eight 16-byte pieces, piece p at position p ^ swz(r): a block is the exact image of its rows in
// the GEMM's LDS stage, so one K stage of a tile is one contiguous read.  swz permutes the pieces so that the
// matrix-core fragment reads (16 rows at one piece) hit distinct LDS banks, both with 32 banks served 8 lanes a
// cycle and with 64 banks served 16 lanes a cycle (the counters show no conflicts).
constexpr int kStageK = 64;                       // K per GEMM stage and per block column
constexpr int kRowBytes = kStageK * 2;
constexpr int kBlockElems = 64 * kStageK;

__device__ __forceinline__ int ctx_swz(int r) { return (r ^ (r >> 3)) & 7; }  // r: row mod 16

__device__ __forceinline__ size_t blocked_offset(int row, int col, int K) {  // element offset of (row, col)
    const int r = row & 63, piece = (col % kStageK) >> 3;
    return (static_cast<size_t>(row >> 6) * (K / kStageK) + col / kStageK) * kBlockElems + r * kStageK +
           ((piece ^ ctx_swz(r & 15)) << 3) + (col & 7);
}

// Weight packing: one thread per 16-byte piece of a row-major [R][K] matrix.
__global__ __launch_bounds__(256) void pack_blocked_kernel(const uint16_t *__restrict__ src, int R, int K,
                                                           uint16_t *__restrict__ dst) {
    const long long e = static_cast<long long>(blockIdx.x) * 256 + threadIdx.x;
    const int per_row = K >> 3;
    if (e >= static_cast<long long>(R) * per_row) return;
    const int row = static_cast<int>(e / per_row);
    const int col = static_cast<int>(e - static_cast<long long>(row) * per_row) * 8;
    *reinterpret_cast<rm_u32x4 *>(dst + blocked_offset(row, col, K)) =
        *reinterpret_cast<const rm_u32x4 *>(src + static_cast<size_t>(row) * K + col);
}

// ------------------------------------------------------------------------------------------ gather

// The listed rows of x as bf16 in the blocked layout [m_pad][d]; rows from the count up to m_pad are zero.
__global__ __launch_bounds__(256) void gather_rows_kernel(const float *__restrict__ x, int d,
                                                          const int32_t *__restrict__ rows,
                                                          const int32_t *__restrict__ count, int max_rows, int m_pad,
                                                          int n_tok, uint16_t *__restrict__ A) {
    const int i = blockIdx.x * 4 + (threadIdx.x >> 6);  // one wave per row
    const int lane = threadIdx.x & 63;
    if (i >= m_pad) return;
    const int cnt = min(max(count[0], 0), max_rows);
    if (i >= cnt) {
        for (int c = lane * 4; c < d; c += 256)
            *reinterpret_cast<uint2 *>(A + blocked_offset(i, c, d)) = make_uint2(0u, 0u);
        return;
    }
    const int r = min(max(rows[i], 0), n_tok - 1);
    const float *src = x + static_cast<size_t>(r) * d;
    for (int c = lane * 4; c < d; c += 256) {
        const float4 v = *reinterpret_cast<const float4 *>(src + c);
        uint2 packed;
        packed.x = rm_f32_to_bf16_bits(v.x) | (rm_f32_to_bf16_bits(v.y) << 16);
        packed.y = rm_f32_to_bf16_bits(v.z) | (rm_f32_to_bf16_bits(v.w) << 16);
        *reinterpret_cast<uint2 *>(A + blocked_offset(i, c, d)) = packed;
    }
}

// ------------------------------------------------------------------------------------------ GEMM

enum { kEpiGlu = 0, kEpiScatter = 1, kEpiPartial = 2 };

struct GemmArgs {
    const uint16_t *A;       // bf16 [m_pad][K], blocked
    const uint16_t *B0, *B1; // bf16 [N][K], row-major or blocked (B1: the up matrix of the gate/up product)
    int K, N, m_pad;
    const int32_t *count;    // rows of A in use (device), clamped to [0, max_rows]
    int max_rows, act;
    uint16_t *H;             // kEpiGlu: bf16 [m_pad][N], blocked
    float *y;                // kEpiScatter: float32 [n_tok][N], row rows[i] receives output row i
    const int32_t *rows;
    int n_tok;
    int splits;              // K slices (workgroups per output tile); kEpiPartial: slice s writes part[s]
    float *part;             // kEpiPartial: float32 [splits][m_pad][N]
};

// ------------------------------------------------------------------------------------------ DMA-staged GEMM

// The tiles are moved by the load unit straight into LDS (global_load_lds_dwordx4), with no register staging:
// STAGES buffers, all but one in flight.  A stage is 64 wide along K (two matrix-core steps, 128 bytes per row) and
// holds the tile's BM rows of A, then BN rows of each B matrix, in the blocked layout's row image; a load
// instruction fills 1 KB = 8 rows, lane l writing bytes [16 l, 16 l + 16).  A (and B when B_BLOCKED) come blocked,
// so each load reads 1 KB of consecutive memory; a row-major B is read 128 bytes per row, each lane taking the
// piece that belongs at its position.

// One load of 16 bytes per lane into LDS at lds + 16 lane (M0 holds the wave's LDS base while it issues; M0 is
// the compiler's register, so its value is kept and put back).  Issued as inline assembly so that the compiler,
// which cannot tell the stage buffers apart, adds no wait of its own for it before the LDS reads: the waits are
// the explicit ones below.
__device__ __forceinline__ void dma16(const void *g, uint32_t lds) {
    uint32_t keep;
    asm volatile(
        "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off\n\ts_mov_b32 m0, %0"
        : "=&s"(keep)
        : "v"(g), "s"(lds)
        : "memory");
}

// Wait until at most N of this wave's vector-memory operations are in flight and all its LDS operations are
// done, then the workgroup barrier.  The compiler may not move memory accesses across it.
template <int N>
__device__ __forceinline__ void dma_wait_barrier() {
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}

__device__ __forceinline__ uint32_t lds_addr(const uint8_t *p) {
    return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) uint8_t *)p));
}

// Waves per SIMD that the stage buffers allow (160 KB of LDS per compute unit), at most 2: the register budget
// follows from it.
constexpr int dma_waves_per_simd(int lds_bytes, int waves) {
    return (163840 / lds_bytes) * waves / 4 >= 2 ? 2 : 1;
}

template <int TM, int TN, int NB, int STAGES, int WAVES_M, bool B_BLOCKED, int EPI>
__global__ __launch_bounds__(128 * WAVES_M,
                             dma_waves_per_simd(STAGES * (16 * WAVES_M * TM + NB * 32 * TN) * kRowBytes, 2 * WAVES_M))
void gemm_dma_kernel(GemmArgs a) {
    constexpr int WAVES = 2 * WAVES_M;             // WAVES_M x 2 waves, each (16 TM) x (16 TN) per matrix
    constexpr int BM = 16 * WAVES_M * TM, BN = 32 * TN;
    constexpr int ROWS = BM + NB * BN;             // a stage: BM rows of A, then BN rows of each B matrix
    constexpr int RPB = 1024 / kRowBytes;          // rows per 1 KB load block
    static_assert(ROWS % (WAVES * RPB) == 0 && BM % (WAVES * RPB) == 0, "load blocks must split evenly");
    static_assert(BM % 64 == 0 && BN % 64 == 0, "tiles of whole 64-row blocks");
    constexpr int BPW = ROWS / RPB / WAVES;        // load blocks per wave and stage
    constexpr int JA = BM / RPB / WAVES;           // the wave's first JA load blocks are rows of A
    static_assert(STAGES >= 2 && STAGES <= 4 && BPW * (STAGES - 2) <= 63, "vmcnt range");
    constexpr int STAGE = ROWS * kRowBytes;
    __shared__ __attribute__((aligned(1024))) uint8_t lds[STAGES][STAGE];

    const int mt = a.m_pad / BM;
    const int ntl = a.N / BN;
    // q = (K slice * ntl + n tile) * mt + m tile: the tiles of one K slice share an XCD (so its L2 holds the slice
    // of A that they all read), and the m tiles of one n tile are neighbours (sharing the weight rows).
    const int q = xcd_order(blockIdx.x, gridDim.x);
    const int m0 = (q % mt) * BM;
    const int n0 = ((q / mt) % ntl) * BN;
    const int ks_id = q / mt / ntl;
    const int k_len = a.K / a.splits;  // a multiple of kStageK
    const int k_base = ks_id * k_len;
    const int cnt = min(max(a.count[0], 0), a.max_rows);
    if (m0 >= cnt) return;  // the whole tile is past the rows in use

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave % WAVES_M, wn = wave / WAVES_M;
    const int r = lane & 15, grp = lane >> 4;

    // Source of this lane's 16 bytes in each of the wave's load blocks (block wave + WAVES j) at stage 0; a
    // blocked operand advances one 8 KB block per stage, a row-major one 128 bytes.
    const size_t kblocks = static_cast<size_t>(a.K / kStageK), kb0 = static_cast<size_t>(k_base / kStageK);
    const uint16_t *src[BPW];
#pragma unroll
    for (int j = 0; j < BPW; ++j) {
        const int row = (wave + WAVES * j) * RPB;  // first stage row of the block
        const uint16_t *base;
        int mrow;
        if (j < JA) {
            base = a.A;
            mrow = m0 + row;
        } else {
            const int rb = row - BM;
            const int nb = rb / BN;
            base = nb ? a.B1 : a.B0;
            mrow = n0 + rb - nb * BN;
        }
        if (j < JA || B_BLOCKED) {
            src[j] = base + ((mrow >> 6) * kblocks + kb0) * kBlockElems + (mrow & 63) * kStageK + lane * 8;
        } else {
            constexpr int kPieces = kStageK / 8;
            const int rr = mrow + lane / kPieces;  // row of this lane's piece
            const int piece = (lane % kPieces) ^ ctx_swz(rr & 15);
            src[j] = base + static_cast<size_t>(rr) * a.K + k_base + piece * 8;
        }
    }
    const uint32_t lds0 = lds_addr(&lds[0][0]);
    auto issue = [&](int kt) {
        const uint32_t buf = lds0 + (kt % STAGES) * STAGE;
#pragma unroll
        for (int j = 0; j < BPW; ++j) {
            const size_t step = (j < JA || B_BLOCKED) ? kBlockElems : kStageK;
            dma16(src[j] + static_cast<size_t>(kt) * step,
                  __builtin_amdgcn_readfirstlane(buf + (wave + WAVES * j) * 1024));
        }
    };

    rm_f32x4 acc[NB][TM][TN];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int tm = 0; tm < TM; ++tm)
#pragma unroll
            for (int tn = 0; tn < TN; ++tn) acc[nb][tm][tn] = rm_f32x4{0.f, 0.f, 0.f, 0.f};

    // Fragment reads: row r of a 16-row tile, piece 4 ks + grp (K elements 32 ks + 8 grp ..) at its permuted place.
    auto compute = [&](const uint8_t *buf) {
#pragma unroll
        for (int ks = 0; ks < kStageK / 32; ++ks) {
            const int frag = r * kRowBytes + (((ks * 4 + grp) ^ ctx_swz(r)) << 4);
            rm_u32x4 af[TM], bf[NB][TN];
#pragma unroll
            for (int tm = 0; tm < TM; ++tm)
                af[tm] = *reinterpret_cast<const rm_u32x4 *>(buf + (wm * TM * 16 + tm * 16) * kRowBytes + frag);
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                for (int tn = 0; tn < TN; ++tn)
                    bf[nb][tn] = *reinterpret_cast<const rm_u32x4 *>(
                        buf + (BM + nb * BN + wn * TN * 16 + tn * 16) * kRowBytes + frag);
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                for (int tm = 0; tm < TM; ++tm)
#pragma unroll
                    for (int tn = 0; tn < TN; ++tn)
                        acc[nb][tm][tn] = mfma16(af[tm], bf[nb][tn], acc[nb][tm][tn]);
        }
    };
    // Stage kt: wait for its loads (the later stages' may stay in flight), barrier (every wave is also done with
    // the buffer read at stage kt - 1), refill that buffer with stage kt + STAGES - 1, compute stage kt.
    const int nk = k_len / kStageK;
#pragma unroll
    for (int s = 0; s < STAGES - 1; ++s)
        if (s < nk) issue(s);
    for (int kt = 0; kt < nk; ++kt) {
        const int later = min(nk - 1 - kt, STAGES - 2);  // stages issued after kt
        if (STAGES >= 4 && later >= 2)
            dma_wait_barrier<(STAGES >= 4 ? 2 : 0) * BPW>();
        else if (STAGES >= 3 && later == 1)
            dma_wait_barrier<BPW>();
        else
            dma_wait_barrier<0>();
        if (kt + STAGES - 1 < nk) issue(kt + STAGES - 1);
        compute(&lds[kt % STAGES][0]);
    }

    // Lane (grp, r), register i of a tile: row 4 grp + i, column r.  The scatter's destination rows are all read
    // before any store (a read behind the row test would wait for each one in turn).
    int dst[TM][4];
    if constexpr (EPI == kEpiScatter) {
#pragma unroll
        for (int tm = 0; tm < TM; ++tm)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int m = min(m0 + wm * TM * 16 + tm * 16 + grp * 4 + i, cnt - 1);
                dst[tm][i] = min(max(a.rows[m], 0), a.n_tok - 1);
            }
    }
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int m = m0 + wm * TM * 16 + tm * 16 + grp * 4 + i;
            if (m >= cnt) continue;
#pragma unroll
            for (int tn = 0; tn < TN; ++tn) {
                const int n = n0 + wn * TN * 16 + tn * 16 + r;
                if constexpr (EPI == kEpiGlu) {
                    const float h = rm_glu_act(a.act, acc[0][tm][tn][i]) * acc[NB - 1][tm][tn][i];
                    a.H[blocked_offset(m, n, a.N)] = static_cast<uint16_t>(rm_f32_to_bf16_bits(h));
                } else if constexpr (EPI == kEpiPartial) {
                    a.part[(static_cast<size_t>(ks_id) * a.m_pad + m) * a.N + n] = acc[0][tm][tn][i];
                } else {
                    a.y[static_cast<size_t>(dst[tm][i]) * a.N + n] = acc[0][tm][tn][i];
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
    // Each thread covers 16 rows of the sequence: 256 threads while they fit (fewer waves at each barrier).
    if (n_tok <= kSelThreadsSmall * kSelPerThread)
        hipLaunchKernelGGL(select_rows_kernel<kSelThreadsSmall>, dim3(1), dim3(kSelThreadsSmall), 0, st,
                           static_cast<const float *>(drift), n_tok, v0, P, k, rows, count);
    else
        hipLaunchKernelGGL(select_rows_kernel<kSelThreads>, dim3(1), dim3(kSelThreads), 0, st,
                           static_cast<const float *>(drift), n_tok, v0, P, k, rows, count);
    return hipGetLastError();
}

template <bool B_BLOCKED>
static hipError_t context_gemms(const ContextPlan &p, const uint16_t *w_gate, const uint16_t *w_up,
                                const uint16_t *w_down_t, const int32_t *rows, const int32_t *count, float *y,
                                char *base, hipStream_t st) {
    constexpr int kWavesM = kCtxBM / 64;
    static_assert(kCtxGluBN == 128, "gate/up tiles of 4 x 16 neurons per wave");
    uint16_t *H = reinterpret_cast<uint16_t *>(base + p.off_h);
    GemmArgs g{};
    g.A = reinterpret_cast<const uint16_t *>(base + p.off_a);
    g.B0 = w_gate;
    g.B1 = w_up;
    g.K = p.d;
    g.N = p.d_ff;
    g.m_pad = p.m_pad;
    g.count = count;
    g.max_rows = p.max_rows;
    g.act = p.act;
    g.H = H;
    g.splits = 1;
    hipError_t e =
        launch_timed(RM_KERNEL_GATEUP, gemm_dma_kernel<4, 4, 2, RM_CTX_GLU_STAGES, kWavesM, B_BLOCKED, kEpiGlu>,
                     dim3((p.m_pad / kCtxBM) * (p.d_ff / kCtxGluBN)), dim3(128 * kWavesM), st, g);
    if (e == hipSuccess) e = hipGetLastError();
    if (e != hipSuccess) return e;

    GemmArgs o{};
    o.A = H;
    o.B0 = w_down_t;
    o.B1 = w_down_t;
    o.K = p.d_ff;
    o.N = p.d;
    o.m_pad = p.m_pad;
    o.count = count;
    o.max_rows = p.max_rows;
    o.y = y;
    o.rows = rows;
    o.n_tok = p.n_tok;
    o.splits = p.down_splits;
    o.part = reinterpret_cast<float *>(base + p.off_part);  // used when split
    const dim3 grid((p.m_pad / kCtxBM) * (p.d / p.down_bn) * p.down_splits), block(128 * kWavesM);
    constexpr int S = RM_CTX_DOWN_STAGES;
    const bool wide = p.down_bn == 128;
    if (p.down_splits == 1) {
        e = wide ? launch_timed(RM_KERNEL_DOWN, gemm_dma_kernel<4, 4, 1, S, kWavesM, B_BLOCKED, kEpiScatter>, grid,
                                block, st, o)
                 : launch_timed(RM_KERNEL_DOWN, gemm_dma_kernel<4, 2, 1, S, kWavesM, B_BLOCKED, kEpiScatter>, grid,
                                block, st, o);
        return e != hipSuccess ? e : hipGetLastError();
    }
    // Split over K: the slices' float32 partials, then their ordered sum scattered into y.
    e = wide ? launch_timed(RM_KERNEL_DOWN, gemm_dma_kernel<4, 4, 1, S, kWavesM, B_BLOCKED, kEpiPartial>, grid, block,
                            st, o)
             : launch_timed(RM_KERNEL_DOWN, gemm_dma_kernel<4, 2, 1, S, kWavesM, B_BLOCKED, kEpiPartial>, grid, block,
                            st, o);
    if (e == hipSuccess) e = hipGetLastError();
    if (e != hipSuccess) return e;
    const long long n4 = static_cast<long long>(p.max_rows) * (p.d / 4);
    hipLaunchKernelGGL(reduce_scatter_kernel, dim3(static_cast<unsigned>((n4 + 255) / 256)), dim3(256), 0, st,
                       static_cast<const float *>(o.part), p.down_splits, p.m_pad, p.d, rows, count, p.max_rows,
                       p.n_tok, y);
    return hipGetLastError();
}

hipError_t launch_context_ffn(const ContextPlan &p, const void *w_gate, const void *w_up, const void *w_down_t,
                              bool blocked, const float *x, const int32_t *rows, const int32_t *count, float *y,
                              void *ws, hipStream_t st) {
    char *base = static_cast<char *>(ws);
    hipLaunchKernelGGL(gather_rows_kernel, dim3((p.m_pad + 3) / 4), dim3(256), 0, st, x, p.d, rows, count,
                       p.max_rows, p.m_pad, p.n_tok, reinterpret_cast<uint16_t *>(base + p.off_a));
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const auto *wg = static_cast<const uint16_t *>(w_gate);
    const auto *wu = static_cast<const uint16_t *>(w_up);
    const auto *wd = static_cast<const uint16_t *>(w_down_t);
    return blocked ? context_gemms<true>(p, wg, wu, wd, rows, count, y, base, st)
                   : context_gemms<false>(p, wg, wu, wd, rows, count, y, base, st);
}

hipError_t launch_pack_blocked(const void *src, int R, int K, void *dst, hipStream_t st) {
    const long long pieces = static_cast<long long>(R) * (K / 8);
    hipLaunchKernelGGL(pack_blocked_kernel, dim3(static_cast<unsigned>((pieces + 255) / 256)), dim3(256), 0, st,
                       static_cast<const uint16_t *>(src), R, K, static_cast<uint16_t *>(dst));
    return hipGetLastError();
}

}  // namespace rm
