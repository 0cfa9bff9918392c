// bf16 masked SwiGLU FFN on CDNA4 matrix cores (v_mfma_f32_16x16x32_bf16), float32 accumulation.
//
// Eq. 4 of the paper, with a zero anchor: only the listed neurons' rows of W_gate / W_up and their rows of the
// neuron-major W_down are read from HBM; the weights are gathered in place, row by row, with no compact copy.
//
// gate/up (gateup_bf16_kernel)
//   One workgroup per 8 listed neurons.  The 16-row A tile of the matrix core holds those neurons' 8 gate rows
//   and 8 up rows, loaded straight from HBM (each lane reads 16 contiguous bytes of a row; a row segment of
//   64 bytes per step is read by 4 lanes).  The B tile is the bf16 FFN input xn^T, 16 tokens per tile, read
//   from L2 (every workgroup needs all of it).  The four waves split the model width d into contiguous
//   quarters and their float32 tiles are summed in LDS in a fixed order; then h = SiLU(g) * u is formed and
//   written to H[t][slot] in bf16.  Slots past the list get h = 0 so that the down projection can always read
//   whole 32-neuron chunks.
//
// down + residual (down_bf16_kernel)
//   Workgroup = (128-column tile, K-slice of 32-neuron chunks, sample).  A = H (tokens x slots), read 16 bytes
//   per lane.  B = the listed W_down rows.  The matrix core wants 8 consecutive K values (neurons) per lane,
//   but a neuron's row is contiguous along the columns, so each lane loads an 8 x 8 block (8 rows x 16 bytes)
//   and feeds 8 matrix-core calls, call q taking column q of the block: call q's 16 output columns are
//   physical columns 8 n + q.  No LDS transpose is needed and every row segment read is 256 contiguous bytes
//   per 16 lanes.  The four waves take interleaved chunks of the slice and are summed in LDS in a fixed order;
//   the slice's partial goes to the workspace and the column tile is finished by the ticket scheme of
//   rm_finish.h (fixed-order sum over slices, + x, no float atomics).
#include "rm_finish.h"
#include "rm_internal.h"

namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ rm_f32x4 mfma_bf16(rm_u32x4 a, rm_u32x4 b, rm_f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(rm_bf16x8, a),
                                                   __builtin_bit_cast(rm_bf16x8, b), c, 0, 0, 0);
}

__device__ __forceinline__ rm_u32x4 load16(const uint16_t *p) { return *reinterpret_cast<const rm_u32x4 *>(p); }

__device__ __forceinline__ int clamp_neuron(int n, int d_ff) { return n < 0 ? 0 : (n >= d_ff ? d_ff - 1 : n); }

__global__ __launch_bounds__(kThreads) void gateup_bf16_kernel(
    const uint16_t *__restrict__ wg, const uint16_t *__restrict__ wu, const uint16_t *__restrict__ xn,
    const int32_t *__restrict__ idx, const int32_t *__restrict__ count, int max_count, int d_ff, int d, int T,
    int tpad, uint16_t *__restrict__ H, int kcap) {
    const int b = blockIdx.y;
    const int slot0 = blockIdx.x * rm::kBfNeurPerBlk;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    int cnt = idx ? count[b] : d_ff;
    cnt = cnt < 0 ? 0 : (cnt > max_count ? max_count : cnt);
    uint16_t *Hb = H + static_cast<size_t>(b) * tpad * kcap;

    if (slot0 >= cnt) {
        for (int t = tid; t < tpad; t += kThreads)
            *reinterpret_cast<rm_u32x4 *>(Hb + static_cast<size_t>(t) * kcap + slot0) = rm_u32x4{0, 0, 0, 0};
        return;
    }

    const int r = lane & 15;   // A row (0-7 gate, 8-15 up) and B column (token within the tile)
    const int grp = lane >> 4; // which 8 of the 32 K values of a step this lane carries
    const int slot = slot0 + (r & 7);
    const bool valid = slot < cnt;
    const int n = valid ? (idx ? clamp_neuron(idx[static_cast<size_t>(b) * d_ff + slot], d_ff) : slot) : 0;
    const uint16_t *wrow = ((r < 8) ? wg : wu) + static_cast<size_t>(n) * d + grp * 8;

    const int nsteps = d / 32;
    const int s_begin = (nsteps * wave) / rm::kBfWaves;
    const int s_end = (nsteps * (wave + 1)) / rm::kBfWaves;

    __shared__ rm_f32x4 red[rm::kBfWaves][4][64];

    for (int t0 = 0; t0 < T; t0 += rm::kBfTokBlock) {
        rm_f32x4 acc[4];
        const uint16_t *xr[4];
        bool xv[4];
#pragma unroll
        for (int tt = 0; tt < 4; ++tt) {
            acc[tt] = rm_f32x4{0.f, 0.f, 0.f, 0.f};
            const int t = t0 + tt * 16 + r;
            xv[tt] = t < T;
            xr[tt] = xn + (static_cast<size_t>(b) * T + (xv[tt] ? t : 0)) * d + grp * 8;
        }
        for (int s = s_begin; s < s_end; ++s) {
            const int col = s * 32;
            const rm_u32x4 a = valid ? load16(wrow + col) : rm_u32x4{0, 0, 0, 0};
#pragma unroll
            for (int tt = 0; tt < 4; ++tt) {
                const rm_u32x4 bx = xv[tt] ? load16(xr[tt] + col) : rm_u32x4{0, 0, 0, 0};
                acc[tt] = mfma_bf16(a, bx, acc[tt]);
            }
        }
#pragma unroll
        for (int tt = 0; tt < 4; ++tt) red[wave][tt][lane] = acc[tt];
        __syncthreads();

        // Output tile: lane L, register i holds row 4*(L/16)+i (gate rows 0-7, up rows 8-15) and token L%16.
        const int j = tid & 7;  // neuron of the block
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            const int tok = (tid >> 3) + 32 * half;
            const int tt = tok >> 4;
            const int tc = tok & 15;
            const int lg = (j >> 2) * 16 + tc;
            const int lu = ((j + 8) >> 2) * 16 + tc;
            const int reg = j & 3;
            const float gsum = ((red[0][tt][lg][reg] + red[1][tt][lg][reg]) + red[2][tt][lg][reg]) +
                               red[3][tt][lg][reg];
            const float usum = ((red[0][tt][lu][reg] + red[1][tt][lu][reg]) + red[2][tt][lu][reg]) +
                               red[3][tt][lu][reg];
            const float h = rm_silu(gsum) * usum;
            Hb[static_cast<size_t>(t0 + tok) * kcap + slot0 + j] = static_cast<uint16_t>(rm_f32_to_bf16_bits(h));
        }
        __syncthreads();
    }
}

__global__ __launch_bounds__(kThreads) void down_bf16_kernel(
    const uint16_t *__restrict__ H, const uint16_t *__restrict__ wd, const int32_t *__restrict__ idx,
    const int32_t *__restrict__ count, int max_count, int d_ff, int d, int T, int tpad, int kcap, int slices,
    int chunks_per_slice, const float *x, float *y, float *__restrict__ part, int *__restrict__ tickets) {
    const int ct = blockIdx.x;
    const int s = blockIdx.y;
    const int b = blockIdx.z;
    const int ncol = gridDim.x;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    int cnt = idx ? count[b] : d_ff;
    cnt = cnt < 0 ? 0 : (cnt > max_count ? max_count : cnt);
    const int nchunks = (cnt + rm::kBfChunk - 1) / rm::kBfChunk;
    const int used_slices = (nchunks + chunks_per_slice - 1) / chunks_per_slice;
    const int c_begin = s * chunks_per_slice;
    const int c_end = min(c_begin + chunks_per_slice, nchunks);

    const int grp = lane >> 4;  // K group: slots 8*grp .. 8*grp+7 of a chunk
    const int nn = lane & 15;   // A row (token in tile) and B column group (physical columns 8*nn + q)
    const int col0 = ct * rm::kBfColTile;
    const bool colok = col0 + nn * 8 < d;
    const uint16_t *Hb = H + static_cast<size_t>(b) * tpad * kcap;
    const int32_t *idxb = idx ? idx + static_cast<size_t>(b) * d_ff : nullptr;
    float *part_tile = part + (static_cast<size_t>(b) * ncol + ct) * slices * static_cast<size_t>(T) * rm::kBfColTile;
    float *P = part_tile + static_cast<size_t>(s) * T * rm::kBfColTile;

    __shared__ rm_f32x4 red[rm::kBfWaves - 1][8][64];

    if (c_begin < c_end) {
        for (int t0 = 0; t0 < T; t0 += rm::kBfTokBlock) {
            rm_f32x4 acc[4][8];
#pragma unroll
            for (int tt = 0; tt < 4; ++tt)
#pragma unroll
                for (int q = 0; q < 8; ++q) acc[tt][q] = rm_f32x4{0.f, 0.f, 0.f, 0.f};

            for (int c = c_begin + wave; c < c_end; c += rm::kBfWaves) {
                const int kb = c * rm::kBfChunk + grp * 8;
                rm_u32x4 w[8];
#pragma unroll
                for (int jj = 0; jj < 8; ++jj) {
                    const int slot = kb + jj;
                    w[jj] = rm_u32x4{0, 0, 0, 0};
                    if (slot < cnt && colok) {
                        const int n = idxb ? clamp_neuron(idxb[slot], d_ff) : slot;
                        w[jj] = load16(wd + static_cast<size_t>(n) * d + col0 + nn * 8);
                    }
                }
                rm_u32x4 a[4];
#pragma unroll
                for (int tt = 0; tt < 4; ++tt)
                    a[tt] = load16(Hb + static_cast<size_t>(t0 + tt * 16 + nn) * kcap + kb);
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    // B fragment of call q: column q of the 8 x 8 block, rows 0..7 (K order), 2 per dword.
                    const int dw = q >> 1;
                    const int sh = (q & 1) * 16;
                    rm_u32x4 bq;
                    bq.x = ((w[0][dw] >> sh) & 0xffffu) | (((w[1][dw] >> sh) & 0xffffu) << 16);
                    bq.y = ((w[2][dw] >> sh) & 0xffffu) | (((w[3][dw] >> sh) & 0xffffu) << 16);
                    bq.z = ((w[4][dw] >> sh) & 0xffffu) | (((w[5][dw] >> sh) & 0xffffu) << 16);
                    bq.w = ((w[6][dw] >> sh) & 0xffffu) | (((w[7][dw] >> sh) & 0xffffu) << 16);
#pragma unroll
                    for (int tt = 0; tt < 4; ++tt) acc[tt][q] = mfma_bf16(a[tt], bq, acc[tt][q]);
                }
            }

            // Sum the four waves: ((w0 + w1) + w2) + w3, one token tile at a time.
#pragma unroll
            for (int tt = 0; tt < 4; ++tt) {
                if (wave > 0) {
#pragma unroll
                    for (int q = 0; q < 8; ++q) red[wave - 1][q][lane] = acc[tt][q];
                }
                __syncthreads();
                if (wave == 0) {
#pragma unroll
                    for (int q = 0; q < 8; ++q) {
                        rm_f32x4 v = acc[tt][q];
                        v += red[0][q][lane];
                        v += red[1][q][lane];
                        v += red[2][q][lane];
                        // lane L, register i: token 4*(L/16)+i of the tile, physical column 8*(L%16) + q
                        acc[tt][q] = v;
                    }
                    if (colok) {
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            const int t = t0 + tt * 16 + grp * 4 + i;
                            if (t < T) {
                                float *dst = P + static_cast<size_t>(t) * rm::kBfColTile + nn * 8;
                                float4 lo, hi;
                                lo.x = acc[tt][0][i];
                                lo.y = acc[tt][1][i];
                                lo.z = acc[tt][2][i];
                                lo.w = acc[tt][3][i];
                                hi.x = acc[tt][4][i];
                                hi.y = acc[tt][5][i];
                                hi.z = acc[tt][6][i];
                                hi.w = acc[tt][7][i];
                                reinterpret_cast<float4 *>(dst)[0] = lo;
                                reinterpret_cast<float4 *>(dst)[1] = hi;
                            }
                        }
                    }
                }
                __syncthreads();
            }
        }
    }

    rm_finish_column_tile<rm::kBfColTile>(part_tile, slices, used_slices, tickets + static_cast<size_t>(b) * ncol + ct,
                                          x + static_cast<size_t>(b) * T * d, y + static_cast<size_t>(b) * T * d,
                                          T, d, col0);
}

}  // namespace

namespace rm {

hipError_t launch_gateup_bf16(const Plan &p, const void *w_gate, const void *w_up, const int32_t *idx,
                              const int32_t *count, void *ws, hipStream_t st) {
    char *base = static_cast<char *>(ws);
    const uint16_t *xn = reinterpret_cast<const uint16_t *>(base + p.off_xn);
    uint16_t *H = reinterpret_cast<uint16_t *>(base + p.off_h);
    profile_before(RM_KERNEL_GATEUP, st);
    hipLaunchKernelGGL(gateup_bf16_kernel, dim3(p.gate_blocks, p.B), dim3(kThreads), 0, st,
                       static_cast<const uint16_t *>(w_gate), static_cast<const uint16_t *>(w_up), xn, idx, count,
                       p.max_count, p.d_ff, p.d, p.T, p.tpad, H, p.kcap);
    hipError_t e = hipGetLastError();
    profile_after(RM_KERNEL_GATEUP, st);
    return e;
}

hipError_t launch_down_bf16(const Plan &p, const void *w_down, const int32_t *idx, const int32_t *count,
                            const float *x, float *y, void *ws, hipStream_t st) {
    char *base = static_cast<char *>(ws);
    const uint16_t *H = reinterpret_cast<const uint16_t *>(base + p.off_h);
    float *part = reinterpret_cast<float *>(base + p.off_part);
    int *tickets = reinterpret_cast<int *>(base + p.off_ticket);
    profile_before(RM_KERNEL_DOWN, st);
    hipLaunchKernelGGL(down_bf16_kernel, dim3(p.ncol, p.slices, p.B), dim3(kThreads), 0, st, H,
                       static_cast<const uint16_t *>(w_down), idx, count, p.max_count, p.d_ff, p.d, p.T, p.tpad,
                       p.kcap, p.slices, p.slice_units, x, y, part, tickets);
    hipError_t e = hipGetLastError();
    profile_after(RM_KERNEL_DOWN, st);
    return e;
}

}  // namespace rm
