// bf16 masked SwiGLU FFN on CDNA4 matrix cores (v_mfma_f32_16x16x32_bf16), float32 accumulation.
//
// Eq. 4 of the paper, with a zero anchor: only the listed neurons' rows of W_gate / W_up and their rows of the
// neuron-major W_down are read from HBM; the weights are gathered in place, row by row, with no compact copy.
// Each wave issues its HBM weight loads before its first matrix-core instruction; the count and the index
// list are loaded together, so a wave waits for two memory round trips (index, then weights) before it can
// compute.
//
// FFN input.  xn holds bf16(x * g) (or bf16(x) without a norm); the per-token RMSNorm factor
// r_t = 1 / sqrt(mean(x_t^2) + eps) multiplies each gate and up sum after the matrix cores, which is exact in
// real arithmetic because r_t is constant along the reduction.  The per-token sums of squares (ssq) come from
// the prologue or from the previous layer's epilogue.
//
// gate/up, 512 threads = 8 waves, one 16-row A tile per wave = 8 gate rows + 8 up rows of 8 listed neurons,
// loaded straight from HBM (16 contiguous bytes per lane).  B = xn^T, 16 tokens per tile.
//   gateup_direct:  1 group of 8 neurons per workgroup; the 8 waves split d; B is read from L2.  Used when the
//                   list is short, so that there are enough workgroups for the 256 compute units.
//   gateup_staged:  NG groups (16..64 neurons) per workgroup, 8 / NG waves per group splitting d; B is
//                   staged in LDS in 256-column chunks (double-buffered) and shared by all NG groups, so each
//                   byte of xn read from L2 serves NG times more neurons.
//   Both sum the d-split waves in LDS in a fixed order, then write h = SiLU(r g) * (r u) to H[t][slot] in
//   bf16.  Slots past the list get h = 0 so that the down projection can read whole 32-neuron chunks.
//
// down, 256 threads.  Workgroup = (64-column tile, K-slice of 32-neuron chunks, sample).  A = H (tokens x
//   slots), 16 bytes per lane.  B = the listed W_down rows.  The matrix core wants 8 consecutive K values
//   (neurons) per lane, but a neuron's row is contiguous along the columns, so each lane loads an 8 x 4 block
//   (8 rows x 8 bytes) and feeds 4 matrix-core calls, call q taking column q of the block: call q's 16 output
//   columns are physical columns 4 n + q.  No LDS transpose is needed, and 16 lanes read a full 128-byte line
//   of a row.  The four waves take interleaved chunks; their tiles are summed in LDS in a fixed order and the
//   slice's float32 partial is stored.  The epilogue kernel adds the slices in order to the residual.
#include "rm_internal.h"

namespace {

constexpr int kGuThreads = 512;
constexpr int kGuWaves = kGuThreads / 64;
constexpr int kDnThreads = 256;
constexpr int kDnWaves = kDnThreads / 64;
constexpr int kMaxSteps = 8;      // direct gate/up: K steps (of 32) whose weight loads are issued together
constexpr int kChunkCols = 256;   // staged gate/up: xn columns per LDS chunk (8 K steps)
constexpr int kChunkSteps = kChunkCols / 32;
constexpr int kRowPitch = kChunkCols + 8;  // bf16 elements per LDS row (16 bytes of padding against conflicts)

__device__ __forceinline__ rm_f32x4 mfma_bf16(rm_u32x4 a, rm_u32x4 b, rm_f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(rm_bf16x8, a),
                                                   __builtin_bit_cast(rm_bf16x8, b), c, 0, 0, 0);
}

__device__ __forceinline__ rm_u32x4 load16(const uint16_t *p) { return *reinterpret_cast<const rm_u32x4 *>(p); }
__device__ __forceinline__ uint2 load8(const uint16_t *p) { return *reinterpret_cast<const uint2 *>(p); }
__device__ __forceinline__ rm_u32x4 zero16() { return rm_u32x4{0u, 0u, 0u, 0u}; }

__device__ __forceinline__ int clamp_neuron(int n, int d_ff) { return n < 0 ? 0 : (n >= d_ff ? d_ff - 1 : n); }
__device__ __forceinline__ int clamp_count(int c, int max_count) { return c < 0 ? 0 : (c > max_count ? max_count : c); }

struct GuArgs {
    const uint16_t *wg, *wu, *xn;
    const int32_t *idx, *count;
    const float *ssq;  // [B][T] per-token sums of squares, or null (no norm)
    float eps;
    int max_count, d_ff, d, T, tpad, kcap;
    uint16_t *H;
};

// Per-token RMSNorm factors of tokens t0 .. t0+63 into LDS (1 without a norm).
__device__ __forceinline__ void load_rnorm(const GuArgs &a, int b, int t0, float *rn) {
    const int t = t0 + static_cast<int>(threadIdx.x);
    if (threadIdx.x < 64) {
        float r = 1.0f;
        if (a.ssq != nullptr && t < a.T)
            r = 1.0f / sqrtf(a.ssq[static_cast<size_t>(b) * a.T + t] / static_cast<float>(a.d) + a.eps);
        rn[threadIdx.x] = r;
    }
}

// The neuron index of this lane's row, loaded without waiting for the count (slots beyond the list are
// masked once the count is known; their index entries are only clamped into range).
__device__ __forceinline__ int lane_neuron(const GuArgs &a, int b, int slot) {
    if (a.idx == nullptr) return slot < a.d_ff ? slot : 0;
    return slot < a.d_ff ? clamp_neuron(a.idx[static_cast<size_t>(b) * a.d_ff + slot], a.d_ff) : 0;
}

// h for 8 neurons x 64 tokens from the summed gate/up tile in LDS; one value per thread of a 512-thread group.
// red: [ds][NT][64 lanes] f32x4 tiles of one neuron group (lane L, register i = row 4*(L/16)+i, token L%16).
template <int NT>
__device__ __forceinline__ float group_h(const rm_f32x4 (*red)[NT][64], int ds, int j, int tok, const float *rn) {
    const int tt = tok >> 4;
    if (tt >= NT) return 0.0f;
    const int tc = tok & 15;
    const int lg = (j >> 2) * 16 + tc;
    const int lu = ((j + 8) >> 2) * 16 + tc;
    const int reg = j & 3;
    float gsum = red[0][tt][lg][reg];
    float usum = red[0][tt][lu][reg];
    for (int w = 1; w < ds; ++w) {
        gsum += red[w][tt][lg][reg];
        usum += red[w][tt][lu][reg];
    }
    const float r = rn[tok];
    return rm_silu(gsum * r) * (usum * r);
}

// ------------------------------------------------------------------------------------------ gate / up, direct

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
        for (int tt = 0; tt < NT; ++tt) c.x[i][tt] = (ok && xv[tt]) ? load16(xr[tt] + (s + i) * 32) : zero16();
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
__global__ __launch_bounds__(kGuThreads) void gateup_direct_kernel(GuArgs a) {
    const int b = blockIdx.y;
    const int slot0 = blockIdx.x * 8;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int r = lane & 15;    // A row (0-7 gate, 8-15 up) and B column (token within the tile)
    const int grp = lane >> 4;  // which 8 of the 32 K values of a step this lane carries
    const int slot = slot0 + (r & 7);
    const int n = lane_neuron(a, b, slot);
    const int cnt = a.idx ? clamp_count(a.count[b], a.max_count) : a.d_ff;
    uint16_t *Hb = a.H + static_cast<size_t>(b) * a.tpad * a.kcap;

    if (slot0 >= cnt) {
        for (int t = tid; t < a.tpad; t += kGuThreads)
            *reinterpret_cast<rm_u32x4 *>(Hb + static_cast<size_t>(t) * a.kcap + slot0) = zero16();
        return;
    }
    const bool valid = slot < cnt;
    const uint16_t *wrow = ((r < 8) ? a.wg : a.wu) + static_cast<size_t>(n) * a.d + grp * 8;
    const int nsteps = a.d / 32;
    const int s_begin = (nsteps * wave) / kGuWaves;
    const int s_end = (nsteps * (wave + 1)) / kGuWaves;

    __shared__ rm_f32x4 red[kGuWaves][NT][64];
    __shared__ float rn[64];

    for (int t0 = 0; t0 < a.T; t0 += rm::kBfTokBlock) {
        load_rnorm(a, b, t0, rn);
        rm_f32x4 acc[NT];
        const uint16_t *xr[NT];
        bool xv[NT];
#pragma unroll
        for (int tt = 0; tt < NT; ++tt) {
            acc[tt] = rm_f32x4{0.f, 0.f, 0.f, 0.f};
            const int t = t0 + tt * 16 + r;
            xv[tt] = t < a.T;
            xr[tt] = a.xn + (static_cast<size_t>(b) * a.T + (xv[tt] ? t : 0)) * a.d + grp * 8;
        }
        for (int sb = s_begin; sb < s_end; sb += kMaxSteps) {
            rm_u32x4 w[kMaxSteps];
#pragma unroll
            for (int i = 0; i < kMaxSteps; ++i) w[i] = (sb + i < s_end) ? load16(wrow + (sb + i) * 32) : zero16();
            GuX<NT> x0, x1;
            gu_load_x(x0, xr, xv, sb, s_end);
            if (!valid) {
#pragma unroll
                for (int i = 0; i < kMaxSteps; ++i) w[i] = zero16();
            }
#pragma unroll
            for (int i = 0; i < kMaxSteps; i += 4) {
                if (sb + i + 2 < s_end) gu_load_x(x1, xr, xv, sb + i + 2, s_end);
                gu_mma2(w[i], w[i + 1], x0, sb + i, s_end, acc);
                if (sb + i + 4 < s_end && i + 4 < kMaxSteps) gu_load_x(x0, xr, xv, sb + i + 4, s_end);
                gu_mma2(w[i + 2], w[i + 3], x1, sb + i + 2, s_end, acc);
            }
        }
#pragma unroll
        for (int tt = 0; tt < NT; ++tt) red[wave][tt][lane] = acc[tt];
        __syncthreads();
        const float h = group_h<NT>(red, kGuWaves, tid & 7, tid >> 3, rn);
        Hb[static_cast<size_t>(t0 + (tid >> 3)) * a.kcap + slot0 + (tid & 7)] =
            static_cast<uint16_t>(rm_f32_to_bf16_bits(h));
        __syncthreads();
    }
}

// ------------------------------------------------------------------------------------------ gate / up, staged

template <int NT, int NG>
__global__ __launch_bounds__(kGuThreads) void gateup_staged_kernel(GuArgs a) {
    constexpr int DS = kGuWaves / NG;            // waves per neuron group (d split)
    constexpr int SPW = kChunkSteps / DS;        // K steps per wave and chunk
    const int b = blockIdx.y;
    const int blk0 = blockIdx.x * 8 * NG;        // first slot of the workgroup
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int g = wave / DS;                     // neuron group of this wave
    const int part = wave % DS;                  // d-split part of this wave
    const int r = lane & 15;
    const int grp = lane >> 4;
    const int slot0 = blk0 + g * 8;
    const int slot = slot0 + (r & 7);
    const int n = lane_neuron(a, b, slot);
    const int cnt = a.idx ? clamp_count(a.count[b], a.max_count) : a.d_ff;
    uint16_t *Hb = a.H + static_cast<size_t>(b) * a.tpad * a.kcap;

    if (blk0 >= cnt) {
        for (int e = tid; e < a.tpad * NG; e += kGuThreads) {
            const int t = e / NG, gg = e % NG;
            *reinterpret_cast<rm_u32x4 *>(Hb + static_cast<size_t>(t) * a.kcap + blk0 + gg * 8) = zero16();
        }
        return;
    }
    const bool valid = slot < cnt;
    const uint16_t *wrow = ((r < 8) ? a.wg : a.wu) + static_cast<size_t>(n) * a.d + grp * 8;
    const int nchunks = (a.d + kChunkCols - 1) / kChunkCols;

    __shared__ __attribute__((aligned(16))) uint16_t xs[2][64 * kRowPitch];
    __shared__ rm_f32x4 red[NG][DS][NT][64];
    __shared__ float rn[64];

    // Cooperative staging of one xn chunk: 64 rows x 256 columns, 16 bytes per thread and pass.
    auto stage_load = [&](int t0, int c, rm_u32x4 *v) {
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            const int e = tid + p * kGuThreads;  // 0 .. 2047
            const int row = e >> 5;              // 32 x 16 bytes per row
            const int col = c * kChunkCols + (e & 31) * 8;
            const int t = t0 + row;
            v[p] = (row < NT * 16 && t < a.T && col < a.d) ? load16(a.xn + (static_cast<size_t>(b) * a.T + t) * a.d + col)
                                                            : zero16();
        }
    };
    auto stage_store = [&](int buf, const rm_u32x4 *v) {
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            const int e = tid + p * kGuThreads;
            const int row = e >> 5;
            *reinterpret_cast<rm_u32x4 *>(&xs[buf][row * kRowPitch + (e & 31) * 8]) = v[p];
        }
    };

    for (int t0 = 0; t0 < a.T; t0 += rm::kBfTokBlock) {
        load_rnorm(a, b, t0, rn);
        rm_f32x4 acc[NT];
#pragma unroll
        for (int tt = 0; tt < NT; ++tt) acc[tt] = rm_f32x4{0.f, 0.f, 0.f, 0.f};

        rm_u32x4 xv[4], w0[SPW], w1[SPW];
        stage_load(t0, 0, xv);
#pragma unroll
        for (int i = 0; i < SPW; ++i) {
            const int s = part * SPW + i;
            w0[i] = (s * 32 < a.d) ? load16(wrow + s * 32) : zero16();
        }
        stage_store(0, xv);
        __syncthreads();
        for (int c = 0; c < nchunks; ++c) {
            const int buf = c & 1;
            const bool more = c + 1 < nchunks;
            if (more) {
                stage_load(t0, c + 1, xv);
#pragma unroll
                for (int i = 0; i < SPW; ++i) {
                    const int col = (c + 1) * kChunkCols + (part * SPW + i) * 32;
                    w1[i] = (col < a.d) ? load16(wrow + col) : zero16();
                }
            }
#pragma unroll
            for (int i = 0; i < SPW; ++i) {
                const int lc = (part * SPW + i) * 32;  // column within the chunk
                if (c * kChunkCols + lc < a.d) {
                    const rm_u32x4 aw = valid ? w0[i] : zero16();
#pragma unroll
                    for (int tt = 0; tt < NT; ++tt) {
                        const rm_u32x4 bx =
                            *reinterpret_cast<const rm_u32x4 *>(&xs[buf][(tt * 16 + r) * kRowPitch + lc + grp * 8]);
                        acc[tt] = mfma_bf16(aw, bx, acc[tt]);
                    }
                }
            }
            if (more) {
                stage_store(buf ^ 1, xv);
#pragma unroll
                for (int i = 0; i < SPW; ++i) w0[i] = w1[i];
            }
            __syncthreads();
        }
#pragma unroll
        for (int tt = 0; tt < NT; ++tt) red[g][part][tt][lane] = acc[tt];
        __syncthreads();
#pragma unroll
        for (int gg = 0; gg < NG; ++gg) {
            // Thread tid forms h for neuron (tid & 7) of group gg and token tid >> 3.
            const float h = group_h<NT>(red[gg], DS, tid & 7, tid >> 3, rn);
            Hb[static_cast<size_t>(t0 + (tid >> 3)) * a.kcap + blk0 + gg * 8 + (tid & 7)] =
                static_cast<uint16_t>(rm_f32_to_bf16_bits(h));
        }
        __syncthreads();
    }
}

// ------------------------------------------------------------------------------------------ down

template <int NT>
struct DnChunk {
    uint2 w[8];
    rm_u32x4 a[NT];
};

struct DnArgs {
    const uint16_t *H, *wd;
    const int32_t *idx, *count;
    int max_count, d_ff, d, T, tpad, kcap, slices, chunks_per_slice;
    float *part;
};

template <int NT>
__device__ __forceinline__ void dn_load(DnChunk<NT> &c, const DnArgs &a, const int32_t *idxb, const uint16_t *Hrow,
                                        int kb, int col, bool colok) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const int slot = kb + j;
        int n = slot < a.d_ff ? slot : 0;
        if (idxb != nullptr) n = slot < a.d_ff ? clamp_neuron(idxb[slot], a.d_ff) : 0;
        c.w[j] = colok ? load8(a.wd + static_cast<size_t>(n) * a.d + col) : make_uint2(0u, 0u);
    }
#pragma unroll
    for (int tt = 0; tt < NT; ++tt) c.a[tt] = load16(Hrow + static_cast<size_t>(tt * 16) * a.kcap + kb);
}

// Slots at or past the count hold h = 0 in H, so their (clamped, loaded) weights contribute nothing.
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
__global__ __launch_bounds__(kDnThreads) void down_bf16_kernel(DnArgs a) {
    const int ct = blockIdx.x;
    const int s = blockIdx.y;
    const int b = blockIdx.z;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int grp = lane >> 4;  // K group: slots 8*grp .. 8*grp+7 of a chunk
    const int nn = lane & 15;   // A row (token in tile) and B column group (physical columns 4*nn + q)
    const int col0 = ct * rm::kBfColTile;
    const int col = col0 + nn * 4;
    const bool colok = col < a.d;
    const int32_t *idxb = a.idx ? a.idx + static_cast<size_t>(b) * a.d_ff : nullptr;
    const size_t stride = static_cast<size_t>(a.T) * a.d;
    float *part_b = a.part + static_cast<size_t>(b) * a.slices * stride;
    float *P = part_b + static_cast<size_t>(s) * stride;
    const int c_begin = s * a.chunks_per_slice;

    // The first chunk of the first token block is loaded before the count is known (its slots are below
    // kcap and its indices are clamped, so the loads stay in bounds); the count then trims the work.
    DnChunk<NT> c0, c1;
    const int c_first = c_begin + wave;
    const bool first_loaded = c_first < min(c_begin + a.chunks_per_slice, a.kcap / rm::kBfChunk);
    if (first_loaded)
        dn_load(c0, a, idxb, a.H + (static_cast<size_t>(b) * a.tpad + nn) * a.kcap, c_first * rm::kBfChunk + grp * 8,
                col, colok);

    const int cnt = a.idx ? clamp_count(a.count[b], a.max_count) : a.d_ff;
    const int nchunks = (cnt + rm::kBfChunk - 1) / rm::kBfChunk;
    const int c_end = min(c_begin + a.chunks_per_slice, nchunks);

    __shared__ rm_f32x4 red[kDnWaves][NT][4][64];

    if (c_begin < c_end) {
        for (int t0 = 0; t0 < a.T; t0 += rm::kBfTokBlock) {
            rm_f32x4 acc[NT][4];
#pragma unroll
            for (int tt = 0; tt < NT; ++tt)
#pragma unroll
                for (int q = 0; q < 4; ++q) acc[tt][q] = rm_f32x4{0.f, 0.f, 0.f, 0.f};

            const uint16_t *Hrow = a.H + (static_cast<size_t>(b) * a.tpad + t0 + nn) * a.kcap;
            int c = c_first;
            if (c < c_end && !(t0 == 0 && first_loaded))
                dn_load(c0, a, idxb, Hrow, c * rm::kBfChunk + grp * 8, col, colok);
            for (; c < c_end; c += 2 * kDnWaves) {
                const int cn = c + kDnWaves;
                const bool more = cn < c_end;
                if (more) dn_load(c1, a, idxb, Hrow, cn * rm::kBfChunk + grp * 8, col, colok);
                dn_mma(c0, acc);
                if (!more) break;
                const int cnn = cn + kDnWaves;
                if (cnn < c_end) dn_load(c0, a, idxb, Hrow, cnn * rm::kBfChunk + grp * 8, col, colok);
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
                        if (t < a.T) {
                            float4 o;
                            o.x = v[0][i];
                            o.y = v[1][i];
                            o.z = v[2][i];
                            o.w = v[3][i];
                            *reinterpret_cast<float4 *>(P + static_cast<size_t>(t) * a.d + col) = o;
                        }
                    }
                }
            }
            __syncthreads();
        }
    }

}

int token_tiles(int T) {
    const int tiles = (T + 15) / 16;
    return tiles >= 4 ? 4 : tiles;
}

template <int NT>
void launch_gateup_nt(const rm::Plan &p, const GuArgs &a, hipStream_t st) {
    const dim3 block(kGuThreads);
    const dim3 grid(p.gate_blocks, p.B);
    switch (p.gate_groups) {
        case 1: hipLaunchKernelGGL(gateup_direct_kernel<NT>, grid, block, 0, st, a); break;
        case 2: hipLaunchKernelGGL((gateup_staged_kernel<NT, 2>), grid, block, 0, st, a); break;
        case 4: hipLaunchKernelGGL((gateup_staged_kernel<NT, 4>), grid, block, 0, st, a); break;
        default: hipLaunchKernelGGL((gateup_staged_kernel<NT, 8>), grid, block, 0, st, a); break;
    }
}

}  // namespace

namespace rm {

hipError_t launch_gateup_bf16(const Plan &p, const void *w_gate, const void *w_up, const int32_t *idx,
                              const int32_t *count, bool norm, void *ws, hipStream_t st) {
    char *base = static_cast<char *>(ws);
    GuArgs a;
    a.wg = static_cast<const uint16_t *>(w_gate);
    a.wu = static_cast<const uint16_t *>(w_up);
    a.xn = reinterpret_cast<const uint16_t *>(base + p.off_xn);
    a.idx = idx;
    a.count = count;
    a.ssq = norm ? reinterpret_cast<const float *>(base + p.off_ssq) : nullptr;
    a.eps = p.eps;
    a.max_count = p.max_count;
    a.d_ff = p.d_ff;
    a.d = p.d;
    a.T = p.T;
    a.tpad = p.tpad;
    a.kcap = p.kcap;
    a.H = reinterpret_cast<uint16_t *>(base + p.off_h);
    profile_before(RM_KERNEL_GATEUP, st);
    switch (token_tiles(p.T)) {
        case 1: launch_gateup_nt<1>(p, a, st); break;
        case 2: launch_gateup_nt<2>(p, a, st); break;
        case 3: launch_gateup_nt<3>(p, a, st); break;
        default: launch_gateup_nt<4>(p, a, st); break;
    }
    hipError_t e = hipGetLastError();
    profile_after(RM_KERNEL_GATEUP, st);
    return e;
}

hipError_t launch_down_bf16(const Plan &p, const void *w_down, const int32_t *idx, const int32_t *count, void *ws,
                            hipStream_t st) {
    char *base = static_cast<char *>(ws);
    DnArgs a;
    a.H = reinterpret_cast<const uint16_t *>(base + p.off_h);
    a.wd = static_cast<const uint16_t *>(w_down);
    a.idx = idx;
    a.count = count;
    a.max_count = p.max_count;
    a.d_ff = p.d_ff;
    a.d = p.d;
    a.T = p.T;
    a.tpad = p.tpad;
    a.kcap = p.kcap;
    a.slices = p.slices;
    a.chunks_per_slice = p.slice_units;
    a.part = reinterpret_cast<float *>(base + p.off_part);
    const dim3 grid(p.ncol, p.slices, p.B), block(kDnThreads);
    profile_before(RM_KERNEL_DOWN, st);
    switch (token_tiles(p.T)) {
        case 1: hipLaunchKernelGGL(down_bf16_kernel<1>, grid, block, 0, st, a); break;
        case 2: hipLaunchKernelGGL(down_bf16_kernel<2>, grid, block, 0, st, a); break;
        case 3: hipLaunchKernelGGL(down_bf16_kernel<3>, grid, block, 0, st, a); break;
        default: hipLaunchKernelGGL(down_bf16_kernel<4>, grid, block, 0, st, a); break;
    }
    hipError_t e = hipGetLastError();
    profile_after(RM_KERNEL_DOWN, st);
    return e;
}

}  // namespace rm
