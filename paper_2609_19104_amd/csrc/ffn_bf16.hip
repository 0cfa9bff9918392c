// bf16 masked SwiGLU FFN on CDNA4 matrix cores (v_mfma_f32_16x16x32_bf16), float32 accumulation.
//
// Eq. 4 of the paper, with a zero anchor: only the listed neurons' rows of W_gate / W_up and their rows of the
// neuron-major W_down are read from HBM; the weights are gathered in place, row by row, with no compact copy.
// Each wave issues all of its HBM weight loads before its first matrix-core instruction and keeps its
// L2-resident operand loads one batch ahead of the matrix cores, so a wave waits for HBM about once rather
// than once per step.
//
// gate/up (gateup_bf16_kernel), 512 threads
//   One workgroup per 8 listed neurons.  The 16-row A tile holds those neurons' 8 gate rows and 8 up rows,
//   loaded straight from HBM (a lane reads 16 contiguous bytes; 4 lanes cover a row's 64-byte step).  The B
//   tile is the bf16 FFN input xn^T, 16 tokens per tile, read from L2 (every workgroup needs all of it).  The
//   eight waves split the model width d into contiguous eighths; their float32 tiles are summed in LDS in a
//   fixed order, then h = SiLU(g) * u is written to H[t][slot] in bf16.  Slots past the list get h = 0.
//
// down (down_bf16_kernel), 256 threads
//   Workgroup = (64-column tile, K-slice of 32-neuron chunks, sample).  A = H (tokens x slots), 16 bytes per
//   lane.  B = the listed W_down rows.  The matrix core wants 8 consecutive K values (neurons) per lane, but a
//   neuron's row is contiguous along the columns, so each lane loads an 8 x 4 block (8 rows x 8 bytes) and
//   feeds 4 matrix-core calls, call q taking column q of the block: call q's 16 output columns are physical
//   columns 4 n + q.  No LDS transpose is needed, and 16 lanes read one full 128-byte line of a row.  The four
//   waves take interleaved chunks of the slice; their tiles are summed in LDS in a fixed order and the slice's
//   float32 partial [T][64] is stored.  The epilogue kernel adds the slices in order to the residual.
#include "rm_internal.h"

namespace {

constexpr int kGuThreads = 512;
constexpr int kGuWaves = kGuThreads / 64;
constexpr int kDnThreads = 256;
constexpr int kDnWaves = kDnThreads / 64;
constexpr int kMaxSteps = 8;  // gate/up K steps (of 32) whose weight loads are issued together

__device__ __forceinline__ rm_f32x4 mfma_bf16(rm_u32x4 a, rm_u32x4 b, rm_f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(rm_bf16x8, a),
                                                   __builtin_bit_cast(rm_bf16x8, b), c, 0, 0, 0);
}

__device__ __forceinline__ rm_u32x4 load16(const uint16_t *p) { return *reinterpret_cast<const rm_u32x4 *>(p); }
__device__ __forceinline__ uint2 load8(const uint16_t *p) { return *reinterpret_cast<const uint2 *>(p); }

__device__ __forceinline__ int clamp_neuron(int n, int d_ff) { return n < 0 ? 0 : (n >= d_ff ? d_ff - 1 : n); }
__device__ __forceinline__ int clamp_count(int c, int max_count) { return c < 0 ? 0 : (c > max_count ? max_count : c); }

// ------------------------------------------------------------------------------------------ gate / up

// x fragments of two K steps for NT token tiles.
template <int NT>
struct GuX {
    rm_u32x4 x[2][NT];
};

template <int NT>
__device__ __forceinline__ void gu_load_x(GuX<NT> &c, const uint16_t *const *xr, const bool *xv, int s, int s_end) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const bool ok = s + i < s_end;
#pragma unroll
        for (int tt = 0; tt < NT; ++tt)
            c.x[i][tt] = (ok && xv[tt]) ? load16(xr[tt] + (s + i) * 32) : rm_u32x4{0, 0, 0, 0};
    }
}

template <int NT>
__device__ __forceinline__ void gu_mma2(rm_u32x4 a0, rm_u32x4 a1, const GuX<NT> &c, int s, int s_end,
                                        rm_f32x4 *acc) {
    if (s < s_end) {
#pragma unroll
        for (int tt = 0; tt < NT; ++tt) acc[tt] = mfma_bf16(a0, c.x[0][tt], acc[tt]);
    }
    if (s + 1 < s_end) {
#pragma unroll
        for (int tt = 0; tt < NT; ++tt) acc[tt] = mfma_bf16(a1, c.x[1][tt], acc[tt]);
    }
}

template <int NT>
__global__ __launch_bounds__(kGuThreads) void gateup_bf16_kernel(
    const uint16_t *__restrict__ wg, const uint16_t *__restrict__ wu, const uint16_t *__restrict__ xn,
    const int32_t *__restrict__ idx, const int32_t *__restrict__ count, int max_count, int d_ff, int d, int T,
    int tpad, uint16_t *__restrict__ H, int kcap) {
    const int b = blockIdx.y;
    const int slot0 = blockIdx.x * rm::kBfNeurPerBlk;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int cnt = idx ? clamp_count(count[b], max_count) : d_ff;
    uint16_t *Hb = H + static_cast<size_t>(b) * tpad * kcap;

    if (slot0 >= cnt) {
        for (int t = tid; t < tpad; t += kGuThreads)
            *reinterpret_cast<rm_u32x4 *>(Hb + static_cast<size_t>(t) * kcap + slot0) = rm_u32x4{0, 0, 0, 0};
        return;
    }

    const int r = lane & 15;    // A row (0-7 gate, 8-15 up) and B column (token within the tile)
    const int grp = lane >> 4;  // which 8 of the 32 K values of a step this lane carries
    const int slot = slot0 + (r & 7);
    const bool valid = slot < cnt;
    const int n = valid ? (idx ? clamp_neuron(idx[static_cast<size_t>(b) * d_ff + slot], d_ff) : slot) : 0;
    const uint16_t *wrow = ((r < 8) ? wg : wu) + static_cast<size_t>(n) * d + grp * 8;

    const int nsteps = d / 32;
    const int s_begin = (nsteps * wave) / kGuWaves;
    const int s_end = (nsteps * (wave + 1)) / kGuWaves;

    __shared__ rm_f32x4 red[kGuWaves][NT][64];

    for (int t0 = 0; t0 < T; t0 += rm::kBfTokBlock) {
        rm_f32x4 acc[NT];
        const uint16_t *xr[NT];
        bool xv[NT];
#pragma unroll
        for (int tt = 0; tt < NT; ++tt) {
            acc[tt] = rm_f32x4{0.f, 0.f, 0.f, 0.f};
            const int t = t0 + tt * 16 + r;
            xv[tt] = t < T;
            xr[tt] = xn + (static_cast<size_t>(b) * T + (xv[tt] ? t : 0)) * d + grp * 8;
        }
        // All of the wave's weight loads (HBM) go out first, up to kMaxSteps K steps at a time; the x loads
        // (L2) follow two steps at a time, one pair ahead of the matrix-core work.
        for (int sb = s_begin; sb < s_end; sb += kMaxSteps) {
            rm_u32x4 a[kMaxSteps];
#pragma unroll
            for (int i = 0; i < kMaxSteps; ++i)
                a[i] = (valid && sb + i < s_end) ? load16(wrow + (sb + i) * 32) : rm_u32x4{0, 0, 0, 0};
            GuX<NT> x0, x1;
            gu_load_x(x0, xr, xv, sb, s_end);
#pragma unroll
            for (int i = 0; i < kMaxSteps; i += 4) {
                if (sb + i + 2 < s_end) gu_load_x(x1, xr, xv, sb + i + 2, s_end);
                gu_mma2(a[i], a[i + 1], x0, sb + i, s_end, acc);
                if (sb + i + 4 < s_end && i + 4 < kMaxSteps) gu_load_x(x0, xr, xv, sb + i + 4, s_end);
                gu_mma2(a[i + 2], a[i + 3], x1, sb + i + 2, s_end, acc);
            }
        }
#pragma unroll
        for (int tt = 0; tt < NT; ++tt) red[wave][tt][lane] = acc[tt];
        __syncthreads();

        // Output tile: lane L, register i holds row 4*(L/16)+i (gate rows 0-7, up rows 8-15) and token L%16.
        const int j = tid & 7;     // neuron of the block
        const int tok = tid >> 3;  // token of the 64-token block
        const int tt = tok >> 4;
        float h = 0.0f;
        if (tt < NT) {
            const int tc = tok & 15;
            const int lg = (j >> 2) * 16 + tc;
            const int lu = ((j + 8) >> 2) * 16 + tc;
            const int reg = j & 3;
            float gsum = red[0][tt][lg][reg];
            float usum = red[0][tt][lu][reg];
#pragma unroll
            for (int w = 1; w < kGuWaves; ++w) {
                gsum += red[w][tt][lg][reg];
                usum += red[w][tt][lu][reg];
            }
            h = rm_silu(gsum) * usum;
        }
        Hb[static_cast<size_t>(t0 + tok) * kcap + slot0 + j] = static_cast<uint16_t>(rm_f32_to_bf16_bits(h));
        __syncthreads();
    }
}

// ------------------------------------------------------------------------------------------ down

template <int NT>
struct DnChunk {
    uint2 w[8];
    rm_u32x4 a[NT];
};

template <int NT>
__device__ __forceinline__ void dn_load(DnChunk<NT> &c, const uint16_t *__restrict__ wd, const int32_t *idxb,
                                        const uint16_t *Hrow, int kcap, int kb, int cnt, int d_ff, int d, int col,
                                        bool colok) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const int slot = kb + j;
        c.w[j] = make_uint2(0u, 0u);
        if (slot < cnt && colok) {
            const int n = idxb ? clamp_neuron(idxb[slot], d_ff) : slot;
            c.w[j] = load8(wd + static_cast<size_t>(n) * d + col);
        }
    }
#pragma unroll
    for (int tt = 0; tt < NT; ++tt) c.a[tt] = load16(Hrow + static_cast<size_t>(tt * 16) * kcap + kb);
}

template <int NT>
__device__ __forceinline__ void dn_mma(const DnChunk<NT> &c, rm_f32x4 (*acc)[4]) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        // B fragment of call q: column q of the 8 x 4 block, rows 0..7 in K order, two bf16 per dword.
        const int dw = q >> 1;
        const int sh = (q & 1) * 16;
        uint32_t v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = dw ? c.w[j].y : c.w[j].x;
        rm_u32x4 bq;
        bq.x = ((v[0] >> sh) & 0xffffu) | (((v[1] >> sh) & 0xffffu) << 16);
        bq.y = ((v[2] >> sh) & 0xffffu) | (((v[3] >> sh) & 0xffffu) << 16);
        bq.z = ((v[4] >> sh) & 0xffffu) | (((v[5] >> sh) & 0xffffu) << 16);
        bq.w = ((v[6] >> sh) & 0xffffu) | (((v[7] >> sh) & 0xffffu) << 16);
#pragma unroll
        for (int tt = 0; tt < NT; ++tt) acc[tt][q] = mfma_bf16(c.a[tt], bq, acc[tt][q]);
    }
}

template <int NT>
__global__ __launch_bounds__(kDnThreads) void down_bf16_kernel(
    const uint16_t *__restrict__ H, const uint16_t *__restrict__ wd, const int32_t *__restrict__ idx,
    const int32_t *__restrict__ count, int max_count, int d_ff, int d, int T, int tpad, int kcap, int slices,
    int chunks_per_slice, float *__restrict__ part) {
    const int ct = blockIdx.x;
    const int s = blockIdx.y;
    const int b = blockIdx.z;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int cnt = idx ? clamp_count(count[b], max_count) : d_ff;
    const int nchunks = (cnt + rm::kBfChunk - 1) / rm::kBfChunk;
    const int c_begin = s * chunks_per_slice;
    const int c_end = min(c_begin + chunks_per_slice, nchunks);
    if (c_begin >= c_end) return;  // no neuron of this sample falls in the slice; the epilogue skips it

    const int grp = lane >> 4;  // K group: slots 8*grp .. 8*grp+7 of a chunk
    const int nn = lane & 15;   // A row (token in tile) and B column group (physical columns 4*nn + q)
    const int col = ct * rm::kBfColTile + nn * 4;
    const bool colok = col < d;
    const int32_t *idxb = idx ? idx + static_cast<size_t>(b) * d_ff : nullptr;
    float *P = part + (static_cast<size_t>(b) * slices + s) * static_cast<size_t>(T) * d;

    __shared__ rm_f32x4 red[kDnWaves][NT][4][64];

    for (int t0 = 0; t0 < T; t0 += rm::kBfTokBlock) {
        rm_f32x4 acc[NT][4];
#pragma unroll
        for (int tt = 0; tt < NT; ++tt)
#pragma unroll
            for (int q = 0; q < 4; ++q) acc[tt][q] = rm_f32x4{0.f, 0.f, 0.f, 0.f};

        const uint16_t *Hrow = H + (static_cast<size_t>(b) * tpad + t0 + nn) * kcap;
        DnChunk<NT> c0, c1;
        int c = c_begin + wave;
        if (c < c_end) dn_load(c0, wd, idxb, Hrow, kcap, c * rm::kBfChunk + grp * 8, cnt, d_ff, d, col, colok);
        for (; c < c_end; c += 2 * kDnWaves) {
            const int cn = c + kDnWaves;
            const bool more = cn < c_end;
            if (more) dn_load(c1, wd, idxb, Hrow, kcap, cn * rm::kBfChunk + grp * 8, cnt, d_ff, d, col, colok);
            dn_mma(c0, acc);
            if (!more) break;
            const int cnn = cn + kDnWaves;
            if (cnn < c_end) dn_load(c0, wd, idxb, Hrow, kcap, cnn * rm::kBfChunk + grp * 8, cnt, d_ff, d, col, colok);
            dn_mma(c1, acc);
        }

#pragma unroll
        for (int tt = 0; tt < NT; ++tt)
#pragma unroll
            for (int q = 0; q < 4; ++q) red[wave][tt][q][lane] = acc[tt][q];
        __syncthreads();
        // Wave w sums token tile w over the four waves (order 0, 1, 2, 3) and stores it.
        if (wave < NT) {
            const int tt = wave;
            rm_f32x4 v[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                v[q] = red[0][tt][q][lane];
#pragma unroll
                for (int w = 1; w < kDnWaves; ++w) v[q] += red[w][tt][q][lane];
            }
            // lane L, register i: token 4*(L/16)+i of the tile, physical column 4*(L%16) + q.
            if (colok) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int t = t0 + tt * 16 + grp * 4 + i;
                    if (t < T) {
                        float4 o;
                        o.x = v[0][i];
                        o.y = v[1][i];
                        o.z = v[2][i];
                        o.w = v[3][i];
                        *reinterpret_cast<float4 *>(P + static_cast<size_t>(t) * d + col) = o;
                    }
                }
            }
        }
        __syncthreads();
    }
}

int token_tiles(int T) {
    const int tiles = (T + 15) / 16;
    return tiles >= 4 ? 4 : tiles;
}

}  // namespace

namespace rm {

hipError_t launch_gateup_bf16(const Plan &p, const void *w_gate, const void *w_up, const int32_t *idx,
                              const int32_t *count, void *ws, hipStream_t st) {
    char *base = static_cast<char *>(ws);
    const uint16_t *xn = reinterpret_cast<const uint16_t *>(base + p.off_xn);
    uint16_t *H = reinterpret_cast<uint16_t *>(base + p.off_h);
    const auto *wg = static_cast<const uint16_t *>(w_gate);
    const auto *wu = static_cast<const uint16_t *>(w_up);
    const dim3 grid(p.gate_blocks, p.B), block(kGuThreads);
    profile_before(RM_KERNEL_GATEUP, st);
    switch (token_tiles(p.T)) {
        case 1: hipLaunchKernelGGL(gateup_bf16_kernel<1>, grid, block, 0, st, wg, wu, xn, idx, count, p.max_count, p.d_ff, p.d, p.T, p.tpad, H, p.kcap); break;
        case 2: hipLaunchKernelGGL(gateup_bf16_kernel<2>, grid, block, 0, st, wg, wu, xn, idx, count, p.max_count, p.d_ff, p.d, p.T, p.tpad, H, p.kcap); break;
        case 3: hipLaunchKernelGGL(gateup_bf16_kernel<3>, grid, block, 0, st, wg, wu, xn, idx, count, p.max_count, p.d_ff, p.d, p.T, p.tpad, H, p.kcap); break;
        default: hipLaunchKernelGGL(gateup_bf16_kernel<4>, grid, block, 0, st, wg, wu, xn, idx, count, p.max_count, p.d_ff, p.d, p.T, p.tpad, H, p.kcap); break;
    }
    hipError_t e = hipGetLastError();
    profile_after(RM_KERNEL_GATEUP, st);
    return e;
}

hipError_t launch_down_bf16(const Plan &p, const void *w_down, const int32_t *idx, const int32_t *count, void *ws,
                            hipStream_t st) {
    char *base = static_cast<char *>(ws);
    const uint16_t *H = reinterpret_cast<const uint16_t *>(base + p.off_h);
    float *part = reinterpret_cast<float *>(base + p.off_part);
    const auto *wd = static_cast<const uint16_t *>(w_down);
    const dim3 grid(p.ncol, p.slices, p.B), block(kDnThreads);
    profile_before(RM_KERNEL_DOWN, st);
    switch (token_tiles(p.T)) {
        case 1: hipLaunchKernelGGL(down_bf16_kernel<1>, grid, block, 0, st, H, wd, idx, count, p.max_count, p.d_ff, p.d, p.T, p.tpad, p.kcap, p.slices, p.slice_units, part); break;
        case 2: hipLaunchKernelGGL(down_bf16_kernel<2>, grid, block, 0, st, H, wd, idx, count, p.max_count, p.d_ff, p.d, p.T, p.tpad, p.kcap, p.slices, p.slice_units, part); break;
        case 3: hipLaunchKernelGGL(down_bf16_kernel<3>, grid, block, 0, st, H, wd, idx, count, p.max_count, p.d_ff, p.d, p.T, p.tpad, p.kcap, p.slices, p.slice_units, part); break;
        default: hipLaunchKernelGGL(down_bf16_kernel<4>, grid, block, 0, st, H, wd, idx, count, p.max_count, p.d_ff, p.d, p.T, p.tpad, p.kcap, p.slices, p.slice_units, part); break;
    }
    hipError_t e = hipGetLastError();
    profile_after(RM_KERNEL_DOWN, st);
    return e;
}

}  // namespace rm
