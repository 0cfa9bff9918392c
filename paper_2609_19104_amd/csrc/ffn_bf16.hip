// bf16 masked SwiGLU FFN on CDNA4 matrix cores (v_mfma_f32_16x16x32_bf16), float32 accumulation.
//
// Eq. 4 of the paper, with a zero anchor: only the listed neurons' rows of W_gate / W_up and their rows of the
// neuron-major W_down are read from HBM; the weights are gathered in place, row by row, with no compact copy.
// Every load is unconditional, from an address clamped into its buffer, and results that must not count are
// masked where they are consumed: a load under a branch makes the compiler wait for all earlier loads before
// the branch joins, which would serialize a wave's memory round trips.  A wave therefore issues all of a
// chunk's loads back to back and waits once.
//
// FFN input.  xn holds bf16(x * g) (or bf16(x) without a norm); the per-token RMSNorm factor
// r_t = 1 / sqrt(mean(x_t^2) + eps) multiplies each gate and up sum after the matrix cores, which is exact in
// real arithmetic because r_t is constant along the reduction.  The per-token sums of squares (ssq) come from
// the prologue or from the previous layer's epilogue.
//
// gate/up, 512 threads = 8 waves, one 16-row A tile per wave = 8 gate rows + 8 up rows of 8 listed neurons,
// loaded straight from HBM (16 contiguous bytes per lane).  B = xn^T, 16 tokens per tile.
//   gateup_direct:  1 group of 8 neurons per workgroup; the 8 waves split d; B is read from L2.  Used when the
//                   list is short, so that there are enough workgroups for the 256 compute units (and d is
//                   256, 512, 1024 or 2048).
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
//   down_fused: for lists of at most 64 chunks, one workgroup sums the whole list for its tile and does the
//   epilogue's work: one sample, 32 columns (2 per lane, 2 calls per chunk) and 16 tokens; several samples, 64
//   columns and the whole 64-token block, the chunks in stages.
#include "rm_internal.h"

namespace {

using rm::launch_timed;

constexpr int kGuThreads = 512;
constexpr int kGuWaves = kGuThreads / 64;
constexpr int kDnThreads = 256;
constexpr int kDnWaves = kDnThreads / 64;
constexpr int kDfThreads = rm::kDfWaves * 64;
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

// Workgroups are dispatched to the 8 XCDs in turn (workgroup i to XCD i mod 8), each XCD with its own L2.  The
// logical index of workgroup `id` of `n` numbers the workgroups so that logical indices [k a, (k + 1) a) (about
// n / 8 of them) run on XCD k: consecutive logical indices share an L2.  The kernels put the samples of one
// neuron block (gate/up) or of one column tile and K-slice (down) at consecutive logical indices: the lists of
// different samples overlap, and their common rows are then fetched once per L2 instead of once per sample.
__device__ __forceinline__ int xcd_logical(int id, int n) {
    const int a = n >> 3, r = n & 7, x = id & 7;
    return x * a + min(x, r) + (id >> 3);
}

struct GuArgs {
    const uint16_t *wg, *wu, *xn;
    const int32_t *idx, *count;
    const float *ssq;  // [B][T][d / 256] per-token partial sums of squares, or null (no norm)
    float eps;
    int max_count, d_ff, d, T, tpad, kcap, B, act;
    uint16_t *H;
    // Eq. 4 (optional, [B][max_count][T] float32): h_anchor is subtracted from h before it is rounded into H
    // (the delta step); with h_out the kernel writes h there in float32 instead of writing H (the anchor step).
    const float *h_anchor;
    float *h_out;
};

// Per-token RMSNorm factors of tokens t0 .. t0+63 into LDS (1 without a norm).
__device__ __forceinline__ void load_rnorm(const GuArgs &a, int b, int t0, float *rn) {
    const int t = t0 + static_cast<int>(threadIdx.x);
    if (threadIdx.x < 64) {
        float r = 1.0f;
        if (a.ssq != nullptr && t < a.T) r = rm_token_rnorm(a.ssq, b * a.T + t, a.d, a.eps);
        rn[threadIdx.x] = r;
    }
}

// The Eq. 4 anchor value h_a of (slot, token t) for gu_store_h, loaded ahead of the products so that the store
// of h waits for no memory: an unconditional load of a clamped in-bounds address (without an anchor it reads the
// list's first entry and the value is not used).
__device__ __forceinline__ float anchor_h(const GuArgs &a, int b, int slot, int t) {
    const size_t ai = (static_cast<size_t>(b) * a.max_count + min(slot, a.max_count - 1)) * a.T + min(t, a.T - 1);
    const float *p = a.h_anchor != nullptr ? a.h_anchor + ai : reinterpret_cast<const float *>(a.idx);
    return *p;
}

// The partial sums of squares of one token block (tokens 0..63 of sample b; rows past T repeat the last token),
// NS spans of 8 partials (256 columns) per token, loaded by the workgroup's 512 threads in memory order: thread e
// takes span e % NS of token e / NS (32 contiguous bytes; threads past 64 NS repeat the last), so that a wave
// reads whole lines.  The load is unconditional, so that it never sits under a branch (where the compiler would
// wait for every load in flight): without a norm it reads the FFN input instead, whose rows are longer, and the
// value is not used.
template <int NS>
__device__ __forceinline__ void load_spans(const GuArgs &a, int b, float4 &lo, float4 &hi) {
    const int e = min(static_cast<int>(threadIdx.x), 64 * NS - 1);
    const int t = min(e / NS, a.T - 1);
    const float *src = a.ssq != nullptr ? a.ssq : reinterpret_cast<const float *>(a.xn);
    const float4 *p =
        reinterpret_cast<const float4 *>(src + static_cast<size_t>(b * a.T + t) * rm::ssq_stride(a.d)) + 2 * (e % NS);
    lo = p[0];
    hi = p[1];
}

// The thread's span sum into LDS: token t's spans at spans[t (NS + 1) + k] (rows padded against bank conflicts).
template <int NS>
__device__ __forceinline__ void store_span(float *spans, float4 lo, float4 hi) {
    const int e = threadIdx.x;
    if (e < 64 * NS) spans[(e / NS) * (NS + 1) + e % NS] = rm_ssq_span(lo, hi);
}

// RMSNorm factor of token t (< 64) from its spans' sums in LDS, added in span order; 1 without a norm and for
// tokens past T.
template <int NS>
__device__ __forceinline__ float span_rnorm(const GuArgs &a, const float *spans, int t) {
    if (a.ssq == nullptr || t >= a.T) return 1.0f;
    const float *p = spans + t * (NS + 1);
    float s = p[0];
#pragma unroll
    for (int k = 1; k < NS; ++k) s += p[k];
    return rm_rnorm_from_ssq(s, a.d, a.eps);
}

// The neuron index of this lane's row (slot clamped into the list; entries past the count are only clamped
// into range, their h is masked when stored).
__device__ __forceinline__ int lane_neuron(const GuArgs &a, int b, int slot) {
    return clamp_neuron(a.idx[static_cast<size_t>(b) * a.d_ff + min(slot, a.d_ff - 1)], a.d_ff);
}

// ------------------------------------------------------------------------------------------ gate / up, direct

// Writes h for 8 neurons x 64 tokens of token block t0 from the summed tile; slots at or past the count and
// tokens at or past T get h = 0 (their rows and columns were computed from clamped loads).  H is chunk-major
// (32-slot chunks, then tokens).  Thread tid finishes tile row tid & 7 (its gate row; the up row is 8 further) for
// token tid >> 3, whose list slot is `slot` (< 0: a duplicate row, nothing stored) and RMSNorm factor r.
// ha_pre: the Eq. 4 anchor value was loaded ahead (ha, from anchor_h), else it is loaded here.
// red(w, tt, lane) is d-part w's tile tt (lane L, register i = row 4 (L / 16) + i, token L % 16).
template <int NT, typename RedAt>
__device__ __forceinline__ void gu_store_h(const GuArgs &a, uint16_t *Hb, int b, RedAt red, int ds, int t0,
                                           int slot, int cnt, float r, bool ha_pre = false, float ha = 0.0f) {
    const int j = threadIdx.x & 7;
    const int tok = threadIdx.x >> 3;
    const int tt = tok >> 4, tc = tok & 15;
    float h = 0.0f;
    if (tt < NT) {
        const int lg = (j >> 2) * 16 + tc;        // gate row j of the tile: lane 16 (j / 4) + token, register j % 4
        const int lu = ((j + 8) >> 2) * 16 + tc;  // up row j + 8
        const int reg = j & 3;
        float gsum = red(0, tt, lg)[reg];
        float usum = red(0, tt, lu)[reg];
        for (int w = 1; w < ds; ++w) {
            gsum += red(w, tt, lg)[reg];
            usum += red(w, tt, lu)[reg];
        }
        h = rm_glu_act(a.act, gsum * r) * (usum * r);
    }
    if (slot < 0) return;
    const int t = t0 + tok;
    const bool live = slot < cnt && t < a.T;
    const size_t ai = (static_cast<size_t>(b) * a.max_count + slot) * a.T + t;  // [b][slot][t] when live
    if (a.h_out != nullptr) {  // anchor capture: float32 h of the listed slots, H untouched
        if (live) a.h_out[ai] = h;
        return;
    }
    if (a.h_anchor != nullptr && live) h -= ha_pre ? ha : a.h_anchor[ai];  // Eq. 4: h_t - h_a, rounded once
    if (!live) h = 0.0f;
    Hb[(static_cast<size_t>(slot >> 5) * a.tpad + t) * rm::kBfChunk + (slot & 31)] =
        static_cast<uint16_t>(rm_f32_to_bf16_bits(h));
}

// Geometry of the direct kernel's per-wave column slice: SPW K steps of 32 columns, staged in sub-slices of at
// most 4 steps (256 bytes per token row) through the wave's own LDS region.
template <int SPW>
struct DirGeom {
    static constexpr int kSubSteps = SPW < 4 ? SPW : 4;
    static constexpr int kSubs = SPW / kSubSteps;
    static constexpr int kRowBytes = kSubSteps * 64;
    static constexpr int kPieces = kRowBytes / 16;   // 16-byte pieces per token row = loads per lane per sub-slice
    static constexpr int kPitch = kRowBytes + 16;    // LDS row pitch: 16 bytes of padding against bank conflicts
    static constexpr int kRegion = 64 * kPitch;      // bytes per wave: 64 token rows
};

// One group of 8 listed neurons per workgroup; wave w takes columns [w * 32 SPW, (w + 1) * 32 SPW) of d = 256 SPW.
// The wave copies its slice of the FFN input (64 token rows) into its own LDS region with whole-line loads
// (each instruction covers 4 rows x 256 bytes), then reads it back in matrix-core fragment order.  Loading the
// fragments straight from memory would touch sixteen half-used lines per instruction, which moves the same
// bytes about three times slower.  Every load of a wave is issued before its first wait: the neuron index, the
// input slice, then the weights (which need the index); the scheduling barrier keeps the compiler from
// interleaving loads with the matrix-core work, so the wave waits for memory once.  No early exit on the count:
// the count only masks the stored h, and its load is not waited for until then.
// kOneBlock: T <= 64, the token-block loop runs once (and compiles away, with its conservative waits).
template <int NT, int SPW, bool kOneBlock>
__global__ __launch_bounds__(kGuThreads) void gateup_direct_kernel(GuArgs a) {
    using G = DirGeom<SPW>;
    const int q = xcd_logical(blockIdx.x, gridDim.x);  // = block * B + sample
    const int b = q % a.B;
    const int slot0 = (q / a.B) * 8;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int r = lane & 15;    // A row (0-7 gate, 8-15 up) and B column (token within the tile)
    const int grp = lane >> 4;  // which 8 of the 32 K values of a step this lane carries
    const int cnt = clamp_count(a.count[b], a.max_count);  // used only when h is stored
    const int raw_n = a.idx[static_cast<size_t>(b) * a.d_ff + min(slot0 + (r & 7), a.d_ff - 1)];
    float ha = anchor_h(a, b, slot0 + (tid & 7), tid >> 3);  // token block 0's anchor value (Eq. 4)
    uint16_t *Hb = a.H + static_cast<size_t>(b) * a.tpad * a.kcap;
    const int col0 = wave * SPW * 32;

    __shared__ __attribute__((aligned(16))) unsigned char lds[kGuWaves * G::kRegion];
    __shared__ float rn[kOneBlock ? (SPW + 1) * 64 : 64];  // kOneBlock: the spans' sums, else the factors
    unsigned char *region = lds + wave * G::kRegion;
    auto red = [&](int w, int tt, int l) -> const rm_f32x4 & {
        return *reinterpret_cast<const rm_f32x4 *>(lds + w * G::kRegion + (tt * 64 + l) * 16);
    };

    // Input slice of token block t0: piece e = j * 64 + lane is row e / kPieces, 16-byte piece e % kPieces.
    auto load_x = [&](int t0, rm_u32x4 (&xv)[G::kSubs][G::kPieces]) {
#pragma unroll
        for (int s = 0; s < G::kSubs; ++s)
#pragma unroll
            for (int j = 0; j < G::kPieces; ++j) {
                const int e = j * 64 + lane;
                const int t = min(t0 + e / G::kPieces, a.T - 1);  // rows past T repeat the last token
                xv[s][j] = load16(a.xn + (static_cast<size_t>(b) * a.T + t) * a.d + col0 + s * G::kSubSteps * 32 +
                                  (e % G::kPieces) * 8);
            }
    };
    rm_u32x4 xv[G::kSubs][G::kPieces];
    load_x(0, xv);
    __builtin_amdgcn_sched_barrier(0);  // the input loads go out before the wait for the index
    rm_u32x4 w[SPW];
    {
        const int n = clamp_neuron(raw_n, a.d_ff);
        const uint16_t *wrow = ((r < 8) ? a.wg : a.wu) + static_cast<size_t>(n) * a.d + col0 + grp * 8;
#pragma unroll
        for (int i = 0; i < SPW; ++i) w[i] = load16(wrow + i * 32);
    }
    // One token block (kOneBlock): behind the weights, the token block's partial sums of squares (SPW spans per
    // token, d = 256 SPW); their span sums go to LDS after the products, so that the norm factors need no memory
    // round trip after them.
    float4 sp_lo = make_float4(0.f, 0.f, 0.f, 0.f), sp_hi = sp_lo;
    if constexpr (kOneBlock) load_spans<SPW>(a, b, sp_lo, sp_hi);
    for (int t0 = 0;;) {
        __builtin_amdgcn_sched_barrier(0);
        rm_f32x4 acc[NT];
#pragma unroll
        for (int tt = 0; tt < NT; ++tt) acc[tt] = rm_f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < G::kSubs; ++s) {
            // The wave's own region: its LDS operations run in order, so no barrier is needed between the
            // previous sub-slice's fragment reads and these writes.
#pragma unroll
            for (int j = 0; j < G::kPieces; ++j) {
                const int e = j * 64 + lane;
                *reinterpret_cast<rm_u32x4 *>(region + (e / G::kPieces) * G::kPitch + (e % G::kPieces) * 16) = xv[s][j];
            }
#pragma unroll
            for (int i = 0; i < G::kSubSteps; ++i)
#pragma unroll
                for (int tt = 0; tt < NT; ++tt) {
                    const rm_u32x4 bx =
                        *reinterpret_cast<const rm_u32x4 *>(region + (tt * 16 + r) * G::kPitch + i * 64 + grp * 16);
                    acc[tt] = mfma_bf16(w[s * G::kSubSteps + i], bx, acc[tt]);
                }
        }
        // The summed tile goes into the wave's region (its fragment reads precede these writes).
#pragma unroll
        for (int tt = 0; tt < NT; ++tt) *reinterpret_cast<rm_f32x4 *>(region + (tt * 64 + lane) * 16) = acc[tt];
        if constexpr (kOneBlock) {
            store_span<SPW>(rn, sp_lo, sp_hi);
        } else {
            load_rnorm(a, b, t0, rn);
        }
        __syncthreads();
        const float rt = kOneBlock ? span_rnorm<SPW>(a, rn, tid >> 3) : rn[tid >> 3];
        gu_store_h<NT>(a, Hb, b, red, kGuWaves, t0, slot0 + (tid & 7), cnt, rt, true, ha);
        t0 += rm::kBfTokBlock;
        if (kOneBlock || t0 >= a.T) break;
        __syncthreads();  // every wave has read the tiles before the regions are refilled
        load_x(t0, xv);
        ha = anchor_h(a, b, slot0 + (tid & 7), t0 + (tid >> 3));
    }
}

// ------------------------------------------------------------------------------------------ gate / up, staged

template <int NT, int NG>
__global__ __launch_bounds__(kGuThreads) void gateup_staged_kernel(GuArgs a) {
    constexpr int DS = kGuWaves / NG;            // waves per neuron group (d split)
    constexpr int SPW = kChunkSteps / DS;        // K steps per wave and chunk
    const int q = xcd_logical(blockIdx.x, gridDim.x);  // = block * B + sample
    const int b = q % a.B;
    const int blk0 = (q / a.B) * 8 * NG;         // first slot of the workgroup
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int g = wave / DS;                     // neuron group of this wave
    const int part = wave % DS;                  // d-split part of this wave
    const int r = lane & 15;
    const int grp = lane >> 4;
    const int slot0 = blk0 + g * 8;
    const int n = lane_neuron(a, b, slot0 + (r & 7));
    const int cnt = clamp_count(a.count[b], a.max_count);
    uint16_t *Hb = a.H + static_cast<size_t>(b) * a.tpad * a.kcap;

    if (blk0 >= cnt) {  // the whole group is past the list: h = 0 (nothing to capture for an anchor)
        if (a.h_out != nullptr) return;
        for (int e = tid; e < a.tpad * NG; e += kGuThreads) {
            const int t = e / NG, slot = blk0 + (e % NG) * 8;
            *reinterpret_cast<rm_u32x4 *>(Hb + (static_cast<size_t>(slot >> 5) * a.tpad + t) * rm::kBfChunk +
                                          (slot & 31)) = zero16();
        }
        return;
    }
    const uint16_t *wrow = ((r < 8) ? a.wg : a.wu) + static_cast<size_t>(n) * a.d + grp * 8;
    const int nchunks = (a.d + kChunkCols - 1) / kChunkCols;
    const int last_col = a.d - 32;  // clamp target of out-of-range K steps (their products are skipped)

    __shared__ __attribute__((aligned(16))) uint16_t xs[2][64 * kRowPitch];
    __shared__ rm_f32x4 red[NG][DS][NT][64];
    __shared__ float rn[64];

    // Cooperative staging of one xn chunk: 64 rows x 256 columns, 16 bytes per thread and pass.  Rows past T
    // and columns past d re-read clamped positions; they only feed outputs that are discarded.
    auto stage_load = [&](int t0, int c, rm_u32x4 *v) {
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            const int e = tid + p * kGuThreads;  // 0 .. 2047
            const int row = e >> 5;              // 32 x 16 bytes per row
            const int col = min(c * kChunkCols + (e & 31) * 8, a.d - 8);
            const int t = min(t0 + row, a.T - 1);
            v[p] = load16(a.xn + (static_cast<size_t>(b) * a.T + t) * a.d + col);
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
        rm_f32x4 acc[NT];
#pragma unroll
        for (int tt = 0; tt < NT; ++tt) acc[tt] = rm_f32x4{0.f, 0.f, 0.f, 0.f};

        rm_u32x4 xv[4], w0[SPW], w1[SPW];
#pragma unroll
        for (int i = 0; i < SPW; ++i) w0[i] = load16(wrow + min((part * SPW + i) * 32, last_col));
        stage_load(t0, 0, xv);
        stage_store(0, xv);
        __syncthreads();
        for (int c = 0; c < nchunks; ++c) {
            const int buf = c & 1;
            const bool more = c + 1 < nchunks;
            if (more) {
#pragma unroll
                for (int i = 0; i < SPW; ++i)
                    w1[i] = load16(wrow + min((c + 1) * kChunkCols + (part * SPW + i) * 32, last_col));
                stage_load(t0, c + 1, xv);
            }
#pragma unroll
            for (int i = 0; i < SPW; ++i) {
                const int lc = (part * SPW + i) * 32;  // column within the chunk
                if (c * kChunkCols + lc < a.d) {
#pragma unroll
                    for (int tt = 0; tt < NT; ++tt) {
                        const rm_u32x4 bx =
                            *reinterpret_cast<const rm_u32x4 *>(&xs[buf][(tt * 16 + r) * kRowPitch + lc + grp * 8]);
                        acc[tt] = mfma_bf16(w0[i], bx, acc[tt]);
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
        load_rnorm(a, b, t0, rn);
#pragma unroll
        for (int tt = 0; tt < NT; ++tt) red[g][part][tt][lane] = acc[tt];
        __syncthreads();
        // Thread tid forms h for neuron (tid & 7) of each group and token tid >> 3.
#pragma unroll
        for (int gg = 0; gg < NG; ++gg) {
            auto red_g = [&](int w, int tt, int l) -> const rm_f32x4 & { return red[gg][w][tt][l]; };
            gu_store_h<NT>(a, Hb, b, red_g, DS, t0, blk0 + gg * 8 + (tid & 7), cnt, rn[tid >> 3]);
        }
        __syncthreads();
    }
}

// The same with NCH = ceil(d / 256) known at compile time (d <= 2048): fully unrolled, so the double buffer
// (weights in registers, xn in LDS) is indexed at compile time and every wait count is exact.
template <int NT, int NG, int NCH>
__global__ __launch_bounds__(kGuThreads) void gateup_staged_unrolled_kernel(GuArgs a) {
    constexpr int DS = kGuWaves / NG;
    constexpr int SPW = kChunkSteps / DS;
    const int q = xcd_logical(blockIdx.x, gridDim.x);  // = block * B + sample
    const int b = q % a.B;
    const int blk0 = (q / a.B) * 8 * NG;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int g = wave / DS;
    const int part = wave % DS;
    const int r = lane & 15;
    const int grp = lane >> 4;
    const int slot0 = blk0 + g * 8;
    const int n = lane_neuron(a, b, slot0 + (r & 7));
    const int cnt = clamp_count(a.count[b], a.max_count);
    uint16_t *Hb = a.H + static_cast<size_t>(b) * a.tpad * a.kcap;

    if (blk0 >= cnt) {  // the whole group is past the list: h = 0 (nothing to capture for an anchor)
        if (a.h_out != nullptr) return;
        for (int e = tid; e < a.tpad * NG; e += kGuThreads) {
            const int t = e / NG, slot = blk0 + (e % NG) * 8;
            *reinterpret_cast<rm_u32x4 *>(Hb + (static_cast<size_t>(slot >> 5) * a.tpad + t) * rm::kBfChunk +
                                          (slot & 31)) = zero16();
        }
        return;
    }
    const uint16_t *wrow = ((r < 8) ? a.wg : a.wu) + static_cast<size_t>(n) * a.d + grp * 8;
    const int last_col = a.d - 32;

    __shared__ __attribute__((aligned(16))) uint16_t xs[2][64 * kRowPitch];
    __shared__ rm_f32x4 red[NG][DS][NT][64];
    __shared__ float rn[64];

    for (int t0 = 0; t0 < a.T; t0 += rm::kBfTokBlock) {
        auto stage_load = [&](int c, rm_u32x4 *v) {
#pragma unroll
            for (int p = 0; p < 4; ++p) {
                const int e = tid + p * kGuThreads;
                const int row = e >> 5;
                const int col = min(c * kChunkCols + (e & 31) * 8, a.d - 8);
                const int t = min(t0 + row, a.T - 1);
                v[p] = load16(a.xn + (static_cast<size_t>(b) * a.T + t) * a.d + col);
            }
        };
        auto stage_store = [&](int buf, const rm_u32x4 *v) {
#pragma unroll
            for (int p = 0; p < 4; ++p) {
                const int e = tid + p * kGuThreads;
                *reinterpret_cast<rm_u32x4 *>(&xs[buf][(e >> 5) * kRowPitch + (e & 31) * 8]) = v[p];
            }
        };
        rm_f32x4 acc[NT];
#pragma unroll
        for (int tt = 0; tt < NT; ++tt) acc[tt] = rm_f32x4{0.f, 0.f, 0.f, 0.f};
        rm_u32x4 w[2][SPW], xv[4];
#pragma unroll
        for (int i = 0; i < SPW; ++i) w[0][i] = load16(wrow + min((part * SPW + i) * 32, last_col));
        stage_load(0, xv);
        stage_store(0, xv);
        __syncthreads();
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            if (c + 1 < NCH) {
#pragma unroll
                for (int i = 0; i < SPW; ++i)
                    w[(c + 1) & 1][i] = load16(wrow + min((c + 1) * kChunkCols + (part * SPW + i) * 32, last_col));
                stage_load(c + 1, xv);
            }
#pragma unroll
            for (int i = 0; i < SPW; ++i) {
                const int lc = (part * SPW + i) * 32;
                if (c * kChunkCols + lc < a.d) {
#pragma unroll
                    for (int tt = 0; tt < NT; ++tt) {
                        const rm_u32x4 bx =
                            *reinterpret_cast<const rm_u32x4 *>(&xs[c & 1][(tt * 16 + r) * kRowPitch + lc + grp * 8]);
                        acc[tt] = mfma_bf16(w[c & 1][i], bx, acc[tt]);
                    }
                }
            }
            if (c + 1 < NCH) stage_store((c + 1) & 1, xv);
            __syncthreads();
        }
        load_rnorm(a, b, t0, rn);
#pragma unroll
        for (int tt = 0; tt < NT; ++tt) red[g][part][tt][lane] = acc[tt];
        __syncthreads();
#pragma unroll
        for (int gg = 0; gg < NG; ++gg) {
            auto red_g = [&](int w, int tt, int l) -> const rm_f32x4 & { return red[gg][w][tt][l]; };
            gu_store_h<NT>(a, Hb, b, red_g, DS, t0, blk0 + gg * 8 + (tid & 7), cnt, rn[tid >> 3]);
        }
        __syncthreads();
    }
}

// ------------------------------------------------------------------------------------------ gate / up, pipelined

// For long lists (T <= 64, d = 256 NCH with NCH in {1, 2, 4, 8}).  NG groups of 8 neurons per workgroup as
// in the staged kernel; column chunk c of the FFN input (64 token rows x 256 columns) is shared by the groups
// through LDS.  Every wave loads its share of chunk c's input (whole 512-byte rows) together with its weights
// for chunk c, P chunks ahead, input first.  A wave's memory counter completes in issue order, so waiting for
// chunk c leaves chunks c+1 .. c+P-1 in flight; and the input of a chunk never waits behind weights of later
// chunks, whose deep queue would otherwise delay it by their whole transfer time.  The input goes through
// registers into a double-buffered LDS tile, with one barrier per chunk.
// kTwoPerCU: for grids larger than the compute unit count, a register budget for two workgroups per compute
// unit (two chunks in flight), so that the whole grid is resident at once instead of running in two rounds.
template <int NG, int NCH, bool kTwoPerCU>
__global__ __launch_bounds__(kGuThreads, (NG == 2 || kTwoPerCU) ? 4 : 2) void gateup_pipe_kernel(GuArgs a) {
    constexpr int NT = 4;
    constexpr int DS = kGuWaves / NG;  // waves per neuron group (d split within a chunk)
    constexpr int SPW = kChunkSteps / DS;  // K steps per wave and chunk
    constexpr int P0 = kTwoPerCU ? (NG == 2 ? 3 : 2) : (NG == 8 ? 3 : (NG == 4 ? 4 : 3));  // chunks in flight
    constexpr int P = P0 < NCH ? P0 : NCH;
    const int q = xcd_logical(blockIdx.x, gridDim.x);  // = block * B + sample
    const int b = q % a.B;
    const int blk0 = (q / a.B) * 8 * NG;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int g = wave / DS;
    const int part = wave % DS;
    const int r = lane & 15;
    const int grp = lane >> 4;
    const int n = lane_neuron(a, b, blk0 + g * 8 + (r & 7));
    const int cnt = clamp_count(a.count[b], a.max_count);
    uint16_t *Hb = a.H + static_cast<size_t>(b) * a.tpad * a.kcap;
    const uint16_t *wrow = ((r < 8) ? a.wg : a.wu) + static_cast<size_t>(n) * a.d + part * SPW * 32 + grp * 8;

    __shared__ __attribute__((aligned(16))) uint16_t xs[2][64 * kRowPitch];
    static_assert(sizeof(rm_f32x4) * NG * DS * NT * 64 <= sizeof(xs), "reduction tiles must fit the input tile");
    auto red = [&](int gg, int w2, int tt, int l) -> rm_f32x4 & {
        return reinterpret_cast<rm_f32x4 *>(&xs[0][0])[((gg * DS + w2) * NT + tt) * 64 + l];
    };

    // Step c processes column chunk (c + block) mod NCH: if every workgroup swept the chunks in the same
    // order, all of them would read the same 512-byte window of their rows at once and load a few memory
    // channels only (measured: about a quarter less bandwidth than with rotated orders).
    const int rot = (q / a.B) & (NCH - 1);
    // Step c into register slot c % P: the input pieces e = tid + 512 q (row e / 32, 16-byte piece e % 32),
    // then the weights.
    rm_u32x4 xv[P][4], w[P][SPW];
    auto load_chunk = [&](int c) {
        const int col = ((c + rot) & (NCH - 1)) * kChunkCols;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = tid + q * kGuThreads;
            const int t = min(e >> 5, a.T - 1);  // rows past T repeat the last token
            xv[c % P][q] = load16(a.xn + (static_cast<size_t>(b) * a.T + t) * a.d + col + (e & 31) * 8);
        }
#pragma unroll
        for (int i = 0; i < SPW; ++i) w[c % P][i] = load16(wrow + col + i * 32);
    };
#pragma unroll
    for (int c = 0; c < P; ++c) load_chunk(c);
    // Behind the first chunks, the partial sums of squares of tokens 0..63 (NCH spans per token); their span sums
    // go to LDS after the products, so that forming the norm factors needs no memory round trip after them.
    // With 8 groups two to a compute unit at d = 2048 those registers would spill: there the factors are loaded
    // after the products instead.
    constexpr bool kSpans = !(NCH == 8 && NG == 8 && kTwoPerCU);
    __shared__ float spans[(NCH + 1) * 64];
    float4 sp_lo = make_float4(0.f, 0.f, 0.f, 0.f), sp_hi = sp_lo;
    if constexpr (kSpans) load_spans<NCH>(a, b, sp_lo, sp_hi);

    rm_f32x4 acc[NT];
#pragma unroll
    for (int tt = 0; tt < NT; ++tt) acc[tt] = rm_f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        // Buffer c & 1 was last read in chunk c - 2, before every wave passed chunk c - 1's barrier.
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = tid + q * kGuThreads;
            *reinterpret_cast<rm_u32x4 *>(&xs[c & 1][(e >> 5) * kRowPitch + (e & 31) * 8]) = xv[c % P][q];
        }
        __syncthreads();
#pragma unroll
        for (int i = 0; i < SPW; ++i)
#pragma unroll
            for (int tt = 0; tt < NT; ++tt) {
                const rm_u32x4 bx = *reinterpret_cast<const rm_u32x4 *>(
                    &xs[c & 1][(tt * 16 + r) * kRowPitch + (part * SPW + i) * 32 + grp * 8]);
                acc[tt] = mfma_bf16(w[c % P][i], bx, acc[tt]);
            }
        if (c + P < NCH) load_chunk(c + P);
    }
    if constexpr (kSpans) {
        store_span<NCH>(spans, sp_lo, sp_hi);
    } else {
        load_rnorm(a, b, 0, spans);
    }
    __syncthreads();  // every wave is done with the input tiles before they hold the reduction
#pragma unroll
    for (int tt = 0; tt < NT; ++tt) red(g, part, tt, lane) = acc[tt];
    __syncthreads();
    const float rt = kSpans ? span_rnorm<NCH>(a, spans, tid >> 3) : spans[tid >> 3];
#pragma unroll
    for (int gg = 0; gg < NG; ++gg)
        gu_store_h<NT>(a, Hb, b, [&](int w2, int tt, int l) -> const rm_f32x4 & { return red(gg, w2, tt, l); }, DS, 0,
                       blk0 + gg * 8 + (tid & 7), cnt, rt);
}

// ------------------------------------------------------------------------------------------ gate / up, spread

// For one sample's lists of more than 256 groups of 8 listed slots (T <= 64, d = 256 NCH with NCH in {1, 2, 4,
// 8}): G workgroups (one per compute unit).  The list is cut into quads of 4 consecutive slots, dealt round-robin:
// workgroup q takes quads q, q + G, q + 2G, ... (m or m + 1 of them), so the weight bytes per compute unit differ
// by at most one quad.  Two quads fill one 16-row weight tile (tile rows 0-3 and 8-11: the first quad's gate and
// up rows, rows 4-7 and 12-15 the second's); an odd last quad is paired with itself, its duplicate rows coalescing
// with the originals in the same load instruction, and only one copy of h is stored.  Every compute unit streams
// weights, and all the workgroup's tiles share each staged chunk of the FFN input.  Wave w takes columns
// [32 w, 32 w + 32) of every 256-column chunk for all the tiles.  The chunk pipeline is the pipelined kernel's
// (weights and input of a chunk issued ahead, rotated chunk order); each tile's 8 wave partials are added in wave
// order through LDS.
// pre(): extra loads of the caller, issued right behind the first weight chunks (PRE_AT = 0) or behind the loads
// of chunk PRE_AT - 1 inside the chunk loop (the one-launch layer form fetches its down-projection rows there);
// PXM: input chunks in flight.
#ifndef RM_SPREAD_WTILES
#define RM_SPREAD_WTILES 9
#endif
#ifndef RM_SPREAD_PX
#define RM_SPREAD_PX 6
#endif
struct NoPre {
    __device__ void operator()() const {}
};
// kLate (the one-launch layer form, whose workgroups write the input first): early() runs behind the index
// loads, and the first input chunks are loaded after it instead of ahead of the indices.  With a meet() (the
// layer form at d = 2048) the first weight chunks go out after early(), then meet() waits for the other
// workgroups, then the input chunks go out.
template <int NG, int NCH, int PXM = RM_SPREAD_PX, int PRE_AT = 0, bool kLate = false, typename Pre = NoPre,
          typename Early = NoPre, typename Meet = NoPre>
__device__ __forceinline__ void gateup_spread_body(const GuArgs &a, int q, int G, int nquads,
                                                   uint16_t (*xs)[64 * kRowPitch], rm_f32x4 *red2, float *spans,
                                                   Pre pre = Pre{}, Early early = Early{}, Meet meet = Meet{}) {
    constexpr int NT = 4;
    constexpr int PW0 = RM_SPREAD_WTILES / (NG > 0 ? NG : 1);  // weight chunks in flight
    constexpr int PW = PW0 < 1 ? 1 : (PW0 < NCH ? PW0 : NCH);
    constexpr int PX = PXM < NCH ? PXM : NCH;  // input chunks in flight
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int r = lane & 15;
    const int grp = lane >> 4;
    const int cnt = clamp_count(a.count[0], a.max_count);
    // Tile j: quads 2j and 2j + 1 of this workgroup (the second is the first again when it does not exist).
    auto quad_of = [&](int j, int half) {
        const int k = min(2 * j + half, nquads - 1);
        return q + k * G;
    };
    int raw_n[NG];
#pragma unroll
    for (int j = 0; j < NG; ++j) {
        const int k = min(2 * j + ((r >> 2) & 1), nquads - 1);  // local quad of this lane's row
        raw_n[j] = a.idx[min((q + k * G) * 4 + (r & 3), a.d_ff - 1)];
    }
    __builtin_amdgcn_sched_barrier(0);  // the index loads go out first
    const int rot = q & (NCH - 1);
    rm_u32x4 xv[PX][4], w[PW][NG];
    const uint16_t *wrow[NG];
    // Chunk c of the input: 64 token rows (rows past T repeat the last token) x 256 columns in 16-byte pieces.
    auto load_x = [&](int c) {
        const int col = ((c + rot) & (NCH - 1)) * kChunkCols;
#pragma unroll
        for (int qq = 0; qq < 4; ++qq) {
            const int e = tid + qq * kGuThreads;
            const int t = min(e >> 5, a.T - 1);
            xv[c % PX][qq] = load16(a.xn + static_cast<size_t>(t) * a.d + col + (e & 31) * 8);
        }
    };
    auto store_x = [&](int c) {  // into LDS buffer c & 1
#pragma unroll
        for (int qq = 0; qq < 4; ++qq) {
            const int e = tid + qq * kGuThreads;
            *reinterpret_cast<rm_u32x4 *>(&xs[c & 1][(e >> 5) * kRowPitch + (e & 31) * 8]) = xv[c % PX][qq];
        }
    };
    auto load_w = [&](int c) {
        const int col = ((c + rot) & (NCH - 1)) * kChunkCols;
#pragma unroll
        for (int j = 0; j < NG; ++j) w[c % PW][j] = load16(wrow[j] + col);
    };
    // The input of the first chunks goes out before the wait for the indices, then the weights.
    if constexpr (!kLate) {
#pragma unroll
        for (int c = 0; c < PX; ++c) load_x(c);
    }
    __builtin_amdgcn_sched_barrier(0);
    early();
    constexpr bool kMeet = !__is_same(Meet, NoPre);
    if constexpr (kLate && !kMeet) {
#pragma unroll
        for (int c = 0; c < PX; ++c) load_x(c);
        __builtin_amdgcn_sched_barrier(0);
    }
    // Rows 8-15 of a tile read W_up: an offset added to W_gate's address.  (Selecting between the two pointers
    // lets the compiler fetch the chosen one from the kernel arguments with a vector load, issued behind the
    // input chunks, which would hold every weight load until all of them have arrived.)
    const ptrdiff_t up_off = r < 8 ? 0 : a.wu - a.wg;
#pragma unroll
    for (int j = 0; j < NG; ++j)
        wrow[j] = a.wg + up_off + static_cast<size_t>(clamp_neuron(raw_n[j], a.d_ff)) * a.d + wave * 32 + grp * 8;
#pragma unroll
    for (int c = 0; c < PW; ++c) load_w(c);
    if constexpr (kMeet) {  // the first weights go out before the caller's meeting, the input after it
        __builtin_amdgcn_sched_barrier(0);
        meet();
#pragma unroll
        for (int c = 0; c < PX; ++c) load_x(c);
        __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (PRE_AT == 0) pre();
    // Behind the first weights, the partial sums of squares of tokens 0..63 (NCH spans per token); their span
    // sums go to LDS after the products, so that forming the norm factors needs no memory round trip after them.
    float4 sp_lo, sp_hi;
    load_spans<NCH>(a, 0, sp_lo, sp_hi);

    rm_f32x4 acc[NG][NT];
#pragma unroll
    for (int j = 0; j < NG; ++j)
#pragma unroll
        for (int tt = 0; tt < NT; ++tt) acc[j][tt] = rm_f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        // Buffer c & 1 was last read in chunk c - 2, before every wave passed chunk c - 1's barrier.
        store_x(c);
        __syncthreads();
        if (c + PX < NCH) load_x(c + PX);
#pragma unroll
        for (int tt = 0; tt < NT; ++tt) {
            const rm_u32x4 bx =
                *reinterpret_cast<const rm_u32x4 *>(&xs[c & 1][(tt * 16 + r) * kRowPitch + wave * 32 + grp * 8]);
#pragma unroll
            for (int j = 0; j < NG; ++j) acc[j][tt] = mfma_bf16(w[c % PW][j], bx, acc[j][tt]);
        }
        if (c + PW < NCH) load_w(c + PW);
        if (PRE_AT > 0 && c + 1 == (PRE_AT < NCH ? PRE_AT : NCH)) pre();
    }
    store_span<NCH>(spans, sp_lo, sp_hi);
    // The waves' partial tiles of every tile go through LDS at once (tiles 0 and 1 in the input buffers, free once
    // every wave has passed the barrier below, tile 2 in red2) and are added in wave order: one barrier for all.
    __syncthreads();  // every wave is done with the input tiles
    auto red_at = [&](int j) -> rm_f32x4 * {
        return j < 2 ? reinterpret_cast<rm_f32x4 *>(&xs[0][0]) + j * kGuWaves * NT * 64 : red2;
    };
#pragma unroll
    for (int j = 0; j < NG; ++j)
#pragma unroll
        for (int tt = 0; tt < NT; ++tt) red_at(j)[(wave * NT + tt) * 64 + lane] = acc[j][tt];
    __syncthreads();
    const float rt = span_rnorm<NCH>(a, spans, tid >> 3);
    const int jj = tid & 7;  // the tile row (neuron) this thread stores
#pragma unroll
    for (int j = 0; j < NG; ++j) {
        const bool dup = jj >= 4 && 2 * j + 1 >= nquads;  // the second half repeats the first quad
        const int slot = dup ? -1 : quad_of(j, jj >> 2) * 4 + (jj & 3);
        const rm_f32x4 *red = red_at(j);
        gu_store_h<NT>(a, a.H, 0,
                       [&](int w2, int tt, int l) -> const rm_f32x4 & { return red[(w2 * NT + tt) * 64 + l]; },
                       kGuWaves, 0, slot, cnt, rt);
    }
}

// NG: tiles of the workgroups with the most quads (ceil(max quads / 2)).  A workgroup's own quad count m or m + 1
// decides its tile count, uniformly over the workgroup.
template <int NG, int NCH>
__global__ __launch_bounds__(kGuThreads) void gateup_spread_kernel(GuArgs a) {
    static_assert(NG <= 3, "two reduction tiles in the input buffers, a third in red2");
    __shared__ __attribute__((aligned(16))) uint16_t xs[2][64 * kRowPitch];
    __shared__ rm_f32x4 red2[NG > 2 ? kGuWaves * 4 * 64 : 1];
    __shared__ float spans[(NCH + 1) * 64];
    static_assert(2 * sizeof(rm_f32x4) * kGuWaves * 4 * 64 <= sizeof(xs), "two reduction tiles fit the input tile");
    const int G = gridDim.x;
    const int q = blockIdx.x;
    const int nq = a.kcap / 4;
    const int mine = (nq - q + G - 1) / G;  // quads of this workgroup (none when the list has fewer quads than G)
    if (mine < 1) return;
    if ((mine + 1) / 2 == NG)
        gateup_spread_body<NG, NCH>(a, q, G, mine, xs, red2, spans);
    else if constexpr (NG > 1)
        gateup_spread_body<NG - 1, NCH>(a, q, G, mine, xs, red2, spans);
}

// ------------------------------------------------------------------------------------------ down

template <int NT>
struct DnChunk {
    uint2 w[8];
    rm_u32x4 a[NT];
};

struct DnArgs {
    const uint16_t *H, *wd;
    const int32_t *idx;
    int d_ff, d, T, tpad, kcap, slices, chunks_per_slice, B, ncol;
    float *part;
};

// Slots at or past the count hold h = 0 in H (the gate/up kernels write every slot below kcap), so the products
// of their chunks are exact zeros and the kernel does not read the count; the epilogue skips whole slices past
// it, so an empty list still gives y = x bit for bit.
// CW calls, one per column of the lane's CW columns (CW = 2 reads only the low dword of each weight row).
template <int NT, int CW = 4>
__device__ __forceinline__ void dn_mma(const DnChunk<NT> &c, rm_f32x4 (*acc)[4]) {
#pragma unroll
    for (int q = 0; q < CW; ++q) {
        // B fragment of call q: column q of the 8 x CW block, rows 0..7 in K order, two bf16 per dword.
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

// CPW: chunks per wave (a slice has 4 * CPW chunks); the chunk pipeline below is unrolled straight-line code.
// Load order: the slice's neuron indices, then the first chunks' H tiles (which do not depend on the indices),
// then, once the indices are in LDS, the weights; the wave waits for memory once per pipeline stage.
template <int NT, int CPW, bool kOneBlock>
__global__ __launch_bounds__(kDnThreads) void down_bf16_kernel(DnArgs a) {
    const int q = xcd_logical(blockIdx.x, gridDim.x);  // = (slice * ncol + column tile) * B + sample
    const int b = q % a.B;
    const int ct = (q / a.B) % a.ncol;
    const int s = (q / a.B) / a.ncol;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int grp = lane >> 4;  // K group: slots 8*grp .. 8*grp+7 of a chunk
    const int nn = lane & 15;   // A row (token in tile) and B column group (physical columns 4*nn + q)
    const int colw = ct * rm::kBfColTile + nn * 4;
    const bool colok = colw < a.d;
    const int col = min(colw, a.d - 4);  // columns past d re-read column d-4; those outputs are not stored
    const size_t stride = static_cast<size_t>(a.T) * a.d;
    float *P = a.part + (static_cast<size_t>(b) * a.slices + s) * stride;
    const int cps = a.chunks_per_slice;
    const int c_begin = s * cps;
    const int c_last = min(c_begin + cps, a.kcap / rm::kBfChunk) - 1;  // last chunk of the slice below kcap
    const uint16_t *Hb = a.H + static_cast<size_t>(b) * a.tpad * a.kcap;

    // The slice's neuron indices, clamped into [0, d_ff), are staged once in LDS: the waves read them with LDS
    // loads, which do not wait behind the weight loads in flight.
    constexpr int kIdxPerThread = rm::kBfMaxChunksPerSlice * rm::kBfChunk / kDnThreads;
    __shared__ __attribute__((aligned(16))) int sidx[rm::kBfMaxChunksPerSlice * rm::kBfChunk];
    int iv[kIdxPerThread];
#pragma unroll
    for (int q = 0; q < kIdxPerThread; ++q) {
        const int i = min(tid + q * kDnThreads, cps * rm::kBfChunk - 1);
        iv[q] = a.idx[static_cast<size_t>(b) * a.d_ff + min(c_begin * rm::kBfChunk + i, a.d_ff - 1)];
    }
    __builtin_amdgcn_sched_barrier(0);  // the index loads go out first

    // Chunk k of this wave is chunk c_begin + wave + 4 k of the slice, clamped to the slice (unconditional
    // loads; the matrix-core step of a chunk past the list is skipped).
    auto chunk_of = [&](int k) { return min(c_begin + wave + k * kDnWaves, c_last); };
    auto load_h = [&](DnChunk<NT> &cc, int k, int t0) {
        const int ce = chunk_of(k);
#pragma unroll
        for (int tt = 0; tt < NT; ++tt)  // chunk-major H: 16 tokens x 64 bytes, one contiguous kilobyte
            cc.a[tt] = load16(Hb + (static_cast<size_t>(ce) * a.tpad + t0 + tt * 16 + nn) * rm::kBfChunk + grp * 8);
    };
    auto load_w = [&](DnChunk<NT> &cc, int k) {
        const int kb = (chunk_of(k) - c_begin) * rm::kBfChunk + grp * 8;
        const int4 i0 = *reinterpret_cast<const int4 *>(sidx + kb);
        const int4 i1 = *reinterpret_cast<const int4 *>(sidx + kb + 4);
        const int n[8] = {i0.x, i0.y, i0.z, i0.w, i1.x, i1.y, i1.z, i1.w};
#pragma unroll
        for (int j = 0; j < 8; ++j) cc.w[j] = load8(a.wd + static_cast<size_t>(n[j]) * a.d + col);
    };

#ifndef RM_DOWN_PD
#define RM_DOWN_PD 2
#endif
    constexpr int PD = RM_DOWN_PD < CPW ? RM_DOWN_PD : CPW;  // chunks in flight per wave
    DnChunk<NT> cb[PD];
#pragma unroll
    for (int k = 0; k < PD; ++k) load_h(cb[k], k, 0);
    __builtin_amdgcn_sched_barrier(0);  // then the H tiles, before the wait for the indices
#pragma unroll
    for (int q = 0; q < kIdxPerThread; ++q) {
        const int i = tid + q * kDnThreads;
        if (i < cps * rm::kBfChunk) sidx[i] = clamp_neuron(iv[q], a.d_ff);
    }
    __syncthreads();

    __shared__ rm_f32x4 red[kDnWaves][NT][4][64];
    for (int t0 = 0;;) {
        rm_f32x4 acc[NT][4];
#pragma unroll
        for (int tt = 0; tt < NT; ++tt)
#pragma unroll
            for (int q = 0; q < 4; ++q) acc[tt][q] = rm_f32x4{0.f, 0.f, 0.f, 0.f};

        // PD chunks in flight: chunk k + PD is loaded into chunk k's registers right after chunk k's products.
#pragma unroll
        for (int k = 0; k < PD; ++k) load_w(cb[k], k);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int k = 0; k < CPW; ++k) {
            if (c_begin + wave + k * kDnWaves <= c_last) dn_mma(cb[k % PD], acc);
            if (k + PD < CPW) {
                load_h(cb[k % PD], k + PD, t0);
                load_w(cb[k % PD], k + PD);
            }
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
                        *reinterpret_cast<float4 *>(P + static_cast<size_t>(t) * a.d + colw) = o;
                    }
                }
            }
        }
        t0 += rm::kBfTokBlock;
        if (kOneBlock || t0 >= a.T) break;
        __syncthreads();
#pragma unroll
        for (int k = 0; k < PD; ++k) load_h(cb[k], k, t0);
    }
}

// ------------------------------------------------------------------------------------------ layer, per XCD

// One sample's list at d = 2048 with 257 .. 768 groups of 8 listed slots (the spread plan's range), or a single
// layer's list of 8 .. 192 chunks at d = 1024: the FFN input's bf16 rounding, the gate/up and the down projection
// in one launch of 256 workgroups, one per compute unit, so no prologue launch precedes it.  The list's 32-slot
// chunks are cut into 8 slices of cps chunks, slice x for the 32 workgroups i with i mod 8 = x.  The dispatcher
// deals a launch's workgroups to the 8 XCDs in turn, starting where the previous launch stopped, so such a group
// shares one XCD and its L2; each workgroup checks this against the hardware's XCC_ID register at meeting 1.
//   Phase 0: the XCD's 32 workgroups write the XCD's own copy of xn = bf16(x g) (and, with a norm, its per-token
//            partial sums of squares, in the prologue's order), one (token row, 256-column block) unit per wave.
//   Phase 1: the spread gate/up over the slice's quads of 4 slots (dealt round-robin over the XCD's 32
//            workgroups), reading the XCD's xn copy and writing h into H.
//   Phase 2: the down projection of the same slice for column tile i / 8 (64 columns at d = 2048, 32 at
//            d = 1024), whose float32 partial goes to the slice's row of the partials as the split down
//            projection writes it, so the epilogue launch is unchanged.
// Between the phases the XCD's workgroups meet; everything a phase reads was written by compute units of the same
// XCD, so no hand-off needs the device-wide L2 write-back that makes a hand-off between XCDs cost more than a
// kernel boundary.  Inside one launch a plain load can be served a stale copy of a line that another compute unit
// stores to, an atomic does not see plain stores' lines, and a plain store can stay in an L2 that a device-scope
// load reads past; a device-scope store and a device-scope load meet.
//   Meeting 1 (after phase 0): each workgroup stores the launch's tag in its flag with a device-scope store (tag:
//            the dispatch packet's id mixed with the queue's address, different for every launch, so the flags
//            need no reset and the workspace no initialization) once its phase-0 stores are complete, and waits
//            until the XCD's 32 flags hold the tag: at d = 2048 with scalar loads issued behind its first weight
//            loads (they have their own counter), at d = 1024 with device-scope vector loads before any weight
//            load (a vector poll issued behind them would wait for them).  Rank 0 first resets the XCD's counter
//            for meeting 2 with an atomic swap.
//   Meeting 2 (after phase 1): an atomic add on that counter (executed past the L1, where the polls, also
//            atomic adds, read it) until it reaches 32.
// The xn copy and H are read with plain loads: no line of them is read in the launch before it is written.  A
// wait gives up after spin_ticks of the 100 MHz real-time clock (as meeting 1 does when a group's workgroups are
// not on one XCD); then the workgroup writes NaN partials, so the layer's output is NaN rather than wrong.
constexpr int kXlPerXcd = 32;  // workgroups per XCD: 256 compute units / 8 XCDs

struct XlArgs {
    GuArgs g;            // the gate/up arguments (one sample); g.xn / g.ssq: XCD 0's copies, XCD x's at + x stride
    const float *x;      // the FFN input, float32 [T][d]
    const float *norm_g; // the norm gain [d], or null
    uint16_t *xn8;       // [8][T][d] bf16: XCD x's copy of xn
    float *ssq8;         // [8][T][ssq_stride(d)]: XCD x's copy of the partial sums of squares (norm only)
    const uint16_t *wd;  // neuron-major W_down [d_ff][d]
    float *part;         // float32 partials [slices][T][d], slice x = chunks [x cps, (x + 1) cps)
    unsigned long long *flags;  // [8][32]: meeting 1's flag of workgroup (XCD x, rank r) at flags[32 x + r]
    unsigned *ctr;       // [8][64]: meeting 2's counter of XCD x at ctr[64 x] (its own 256-byte line)
    unsigned zero;       // 0, an operand the compiler cannot see, so that a poll stays an atomic add
    int cps;             // chunks per slice, at most 8 CPW
    long long spin_ticks;
};

__device__ __forceinline__ unsigned xcc_id() {
    unsigned v;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(v));
    return v & 0xfu;
}

extern "C" __device__ unsigned long long rm_llvm_dispatch_id() __asm("llvm.amdgcn.dispatch.id");

// A 64-bit value that differs between launches: the dispatch packet's id in its queue (a counter) times an odd
// constant (a bijection), xor the queue's address.
__device__ __forceinline__ unsigned long long launch_tag() {
    const unsigned long long q = reinterpret_cast<unsigned long long>(__builtin_amdgcn_queue_ptr());
    return (rm_llvm_dispatch_id() + 1ull) * 0x9E3779B97F4A7C15ull ^ q;
}

// NCH: 256-column chunks of d (8 at d = 2048); CPW: chunks per wave in phase 2 (cps <= 8 CPW).  The phase-2
// rows of W_down are requested inside phase 1, behind the loads of its chunk RM_XCD_PRE_AT - 1 (the last
// chunk's weights are then in flight, so no product waits for them), and held in registers until meeting 2;
// after it only H (from this XCD's L2) is read.  Requested at the start instead, they delayed the first input
// chunk by 2.7 us; requested after the meeting, the down phase waited for them.  RM_XCD_PX: input chunks in flight
// (all of them: the XCD's copy of xn is requested at once after meeting 1, 0.2 us faster than 6 at a time).
#ifndef RM_XCD_PX
#define RM_XCD_PX 8
#endif
#ifndef RM_XCD_PRE_AT
#define RM_XCD_PRE_AT 7
#endif
// CW: columns per lane in phase 2 (4 at d = 2048, 2 at d = 1024): column tiles of 16 CW columns, 32 per XCD.
template <int NCH, int CPW, int CW>
__global__ __launch_bounds__(kGuThreads) void layer_xcd_kernel(XlArgs a) {
    constexpr int NT = 4;
    constexpr bool kScalarPoll = NCH == 8;  // meeting 1's wait: scalar loads behind the first weights (d = 2048)
    constexpr int kXsBytes = 2 * 64 * kRowPitch * 2;            // phase 1: the staged input chunks
    constexpr int kRed2Bytes = kGuWaves * NT * 64 * 16;          // phase 1: the third tile's wave partials
    constexpr int kRedBytes = kGuWaves * NT * 4 * 64 * 16;       // phase 2: the 8 waves' 64-token x 16 CW tiles (CW <= 4)
    static_assert(kXsBytes + kRed2Bytes <= kRedBytes, "phase 1's buffers fit phase 2's");
    constexpr int kSlots = CPW * kGuWaves * rm::kBfChunk;        // indices of a slice
    constexpr int kIdxPer = (kSlots + kGuThreads - 1) / kGuThreads;
    constexpr int kUnits = 2;                                    // phase-0 units per wave: 64 rows x NCH blocks / 256
    __shared__ __attribute__((aligned(16))) unsigned char lds[kRedBytes];
    __shared__ float spans[(NCH + 1) * 64];
    __shared__ __attribute__((aligned(16))) int sidx[kSlots];
    __shared__ int s_fail;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int x = blockIdx.x & 7;
    const int rank = blockIdx.x >> 3;  // the workgroup's place on its XCD, and its phase-2 column tile
    GuArgs g = a.g;
    g.xn = a.xn8 + static_cast<size_t>(x) * g.T * g.d;
    if (g.ssq != nullptr) g.ssq = a.ssq8 + static_cast<size_t>(x) * g.T * rm::ssq_stride(g.d);
    const int nchunks = g.kcap / rm::kBfChunk;
    const int c0 = x * a.cps;
    const int n = max(0, min(c0 + a.cps, nchunks) - c0);  // chunks of this XCD's slice

    // Phase 0's input: unit u = row * NCH + block of the XCD's T * NCH units, u = 8 rank + wave + 256 k; the loads
    // are unconditional (a unit past the rows reloads the last one, whose results are not stored).
    const int units = g.T * NCH;
    float4 xin[kUnits], gin[kUnits];
#pragma unroll
    for (int k = 0; k < kUnits; ++k) {
        const int u = min(rank * kGuWaves + wave + k * kXlPerXcd * kGuWaves, units - 1);
        const size_t o = static_cast<size_t>(u / NCH) * g.d + (u % NCH) * kChunkCols + lane * 4;
        xin[k] = *reinterpret_cast<const float4 *>(a.x + o);
        gin[k] = *reinterpret_cast<const float4 *>((a.norm_g != nullptr ? a.norm_g : a.x) + (u % NCH) * kChunkCols +
                                                   lane * 4);
    }

    const int grp = lane >> 4;  // phase 2: slots 8 grp .. 8 grp + 7 of a chunk
    const int nn = lane & 15;   // phase 2: token in tile, and physical columns CW nn + q
    const int colw = rank * 16 * CW + nn * CW;
    const bool colok = colw < g.d;
    const int col = min(colw, g.d - CW);  // columns past d re-read the last ones; those outputs are not stored
    // Phase 2's chunk k of this wave: slice chunk wave + 8 k (clamped to the slice; the products of a chunk past
    // it are skipped), counted from a start that differs by column tile, so that the XCD's 32 workgroups do not
    // all read the same chunk of H from the L2 at the same time.
    const int rot = rank % max(n, 1);
    auto chunk_of = [&](int k) {
        const int j = min(wave + k * kGuWaves, max(n, 1) - 1);
        return c0 + (j + rot < max(n, 1) ? j + rot : j + rot - max(n, 1));
    };
    // The slice's indices go out with the input (two coalesced loads per thread) and are staged in LDS when the
    // rows they name are requested.
    int iv[kIdxPer];
#pragma unroll
    for (int q = 0; q < kIdxPer; ++q) {
        const int i = min(tid + q * kGuThreads, max(n * rm::kBfChunk, 1) - 1);
        iv[q] = g.idx[min(c0 * rm::kBfChunk + i, g.d_ff - 1)];
    }
    uint2 wdn[CPW][8];
    auto pre = [&]() {
#pragma unroll
        for (int q = 0; q < kIdxPer; ++q) {
            const int i = tid + q * kGuThreads;
            if (i < kSlots) sidx[i] = clamp_neuron(iv[q], g.d_ff);
        }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < CPW; ++k) {
            const int kb = (chunk_of(k) - c0) * rm::kBfChunk + grp * 8;
            const int4 i0 = *reinterpret_cast<const int4 *>(sidx + kb);
            const int4 i1 = *reinterpret_cast<const int4 *>(sidx + kb + 4);
            const int nr[8] = {i0.x, i0.y, i0.z, i0.w, i1.x, i1.y, i1.z, i1.w};
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const uint16_t *src = a.wd + static_cast<size_t>(nr[j]) * g.d + col;
                if constexpr (CW == 4)
                    wdn[k][j] = load8(src);
                else  // two columns: the row's 4 bytes in the low dword, which is all dn_mma<NT, 2> reads
                    wdn[k][j] = uint2{*reinterpret_cast<const uint32_t *>(src), 0u};
            }
        }
    };
    // The flag this workgroup stores: the launch's tag with its low 4 bits replaced by the XCD it runs on, so that
    // a group's flags agree only if all 32 of its workgroups share one XCD (and thus one L2).
    const unsigned long long tag = (launch_tag() & ~0xfull) | xcc_id();
    unsigned long long *fl = a.flags + x * kXlPerXcd;
    unsigned *ctr = a.ctr + x * 64;
    if (tid == 0) s_fail = 0;
    // Phase 0 (behind the index loads, before the input and weight loads): round x g to bf16 into this XCD's copy
    // of xn, as the prologue does, then meeting 1.
    auto early = [&]() {
#pragma unroll
        for (int k = 0; k < kUnits; ++k) {
            const int u = rank * kGuWaves + wave + k * kXlPerXcd * kGuWaves;
            const int row = u / NCH, blk = u % NCH;
            float4 v = xin[k];
            if (g.ssq != nullptr) {  // partial sums of squares of the row's 32-column blocks
                const float ss = rm_ssq32(v, true);
                if (u < units && (lane & 7) == 0)
                    const_cast<float *>(g.ssq)[static_cast<size_t>(row) * rm::ssq_stride(g.d) + blk * 8 + (lane >> 3)] = ss;
                v.x *= gin[k].x;
                v.y *= gin[k].y;
                v.z *= gin[k].z;
                v.w *= gin[k].w;
            }
            uint2 packed;
            packed.x = rm_f32_to_bf16_bits(v.x) | (rm_f32_to_bf16_bits(v.y) << 16);
            packed.y = rm_f32_to_bf16_bits(v.z) | (rm_f32_to_bf16_bits(v.w) << 16);
            if (u < units)
                *reinterpret_cast<uint2 *>(const_cast<uint16_t *>(g.xn) + static_cast<size_t>(row) * g.d +
                                           blk * kChunkCols + lane * 4) = packed;
        }
        if (tid == 0 && rank == 0) __hip_atomic_exchange(ctr, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        // This wave's stores are complete (vmcnt(0); the builtin, unlike an asm statement, tells the compiler
        // that the index loads are complete too, so the weight loads behind the flag's store need no wait).
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_waitcnt(0x0f70);
        __syncthreads();
        // Meeting 1: arrive; at d = 1024 also wait here, before any weight load is in flight (a vector poll would
        // wait behind them), until the XCD's 32 flags hold the tag.
        if (tid == 0) __hip_atomic_store(fl + rank, tag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if constexpr (!kScalarPoll) {
            if (wave == 0) {
                bool fail = false;
                const unsigned long long t0 = __builtin_amdgcn_s_memrealtime();
                for (;;) {
                    const unsigned long long f =
                        __hip_atomic_load(fl + (lane & (kXlPerXcd - 1)), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    if (__builtin_amdgcn_ballot_w64(f != tag) == 0) break;
                    if (static_cast<long long>(__builtin_amdgcn_s_memrealtime() - t0) > a.spin_ticks) {
                        fail = true;
                        break;
                    }
                    __builtin_amdgcn_s_sleep(1);
                }
                if (lane == 0 && fail) s_fail = 1;
            }
            __syncthreads();
        }
    };
    // At d = 2048 the wait of meeting 1 comes behind the first weight loads: wave 0 polls with scalar loads that
    // bypass the scalar cache (their own counter, so they do not wait for the weights in flight) until the XCD's
    // 32 flags hold the tag, 8 flags (64 bytes) per load.  (Measured: config 4 at 30 % 27.6 -> 26.6 us per
    // step; at d = 1024, with less weight per compute unit, 13.8 -> 14.1, so there the vector poll stays.)
    auto meet = [&]() {
        if (wave == 0) {
            bool fail = false;
            const unsigned long long t0 = __builtin_amdgcn_s_memrealtime();
            for (;;) {
                typedef unsigned u32x16 __attribute__((ext_vector_type(16)));
                u32x16 f0, f1, f2, f3;
                asm volatile(
                    "s_load_dwordx16 %0, %4, 0x0 glc\n\t"
                    "s_load_dwordx16 %1, %4, 0x40 glc\n\t"
                    "s_load_dwordx16 %2, %4, 0x80 glc\n\t"
                    "s_load_dwordx16 %3, %4, 0xc0 glc\n\t"
                    "s_waitcnt lgkmcnt(0)"
                    : "=s"(f0), "=s"(f1), "=s"(f2), "=s"(f3)
                    : "s"(fl)
                    : "memory");
                const unsigned lo = static_cast<unsigned>(tag), hi = static_cast<unsigned>(tag >> 32);
                bool all = true;
#pragma unroll
                for (int i = 0; i < 8; ++i)
                    all = all && f0[2 * i] == lo && f0[2 * i + 1] == hi && f1[2 * i] == lo && f1[2 * i + 1] == hi &&
                          f2[2 * i] == lo && f2[2 * i + 1] == hi && f3[2 * i] == lo && f3[2 * i + 1] == hi;
                if (all) break;
                if (static_cast<long long>(__builtin_amdgcn_s_memrealtime() - t0) > a.spin_ticks) {
                    fail = true;
                    break;
                }
                __builtin_amdgcn_s_sleep(1);
            }
            if (lane == 0 && fail) s_fail = 1;
        }
        __syncthreads();
    };

    // Phase 1: gate/up of the slice's quads q0, q0 + 32, ...
    const int nq = n * (rm::kBfChunk / 4);
    const int mine = nq > rank ? (nq - rank + kXlPerXcd - 1) / kXlPerXcd : 0;
    auto xs = reinterpret_cast<uint16_t(*)[64 * kRowPitch]>(lds);
    auto red2 = reinterpret_cast<rm_f32x4 *>(lds + kXsBytes);
    const int q0 = c0 * (rm::kBfChunk / 4) + rank;
    auto phase1 = [&](auto wait) {  // wait: the scalar poll, or nothing (early() has polled)
        switch ((mine + 1) / 2) {
            case 0:
                early();
                wait();
                pre();
                break;
            case 1:
                gateup_spread_body<1, NCH, RM_XCD_PX, RM_XCD_PRE_AT, true>(g, q0, kXlPerXcd, mine, xs, red2, spans,
                                                                           pre, early, wait);
                break;
            case 2:
                gateup_spread_body<2, NCH, RM_XCD_PX, RM_XCD_PRE_AT, true>(g, q0, kXlPerXcd, mine, xs, red2, spans,
                                                                           pre, early, wait);
                break;
            default:
                gateup_spread_body<3, NCH, RM_XCD_PX, RM_XCD_PRE_AT, true>(g, q0, kXlPerXcd, mine, xs, red2, spans,
                                                                           pre, early, wait);
                break;
        }
    };
    if constexpr (kScalarPoll)
        phase1(meet);
    else
        phase1(NoPre{});

    // Meeting 2: this workgroup's stores of h are complete before it arrives.
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (tid == 0) {
        unsigned now = __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) + 1u;
        const unsigned long long t0 = __builtin_amdgcn_s_memrealtime();
        while (now < kXlPerXcd) {
            __builtin_amdgcn_s_sleep(1);
            now = __hip_atomic_fetch_add(ctr, a.zero, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (static_cast<long long>(__builtin_amdgcn_s_memrealtime() - t0) > a.spin_ticks) {
                s_fail = 1;
                break;
            }
        }
    }
    __syncthreads();
    asm volatile("buffer_inv sc0" ::: "memory");  // this compute unit's L1 holds no line of H
    if (n == 0) return;

    // Phase 2: the slice's chunks for column tile `rank`, the rows already in registers; H from the L2.
    DnChunk<NT> cb[CPW];
#pragma unroll
    for (int k = 0; k < CPW; ++k) {
        const int ce = chunk_of(k);
#pragma unroll
        for (int tt = 0; tt < NT; ++tt)
            cb[k].a[tt] = load16(g.H + (static_cast<size_t>(ce) * g.tpad + tt * 16 + nn) * rm::kBfChunk + grp * 8);
#pragma unroll
        for (int j = 0; j < 8; ++j) cb[k].w[j] = wdn[k][j];
    }
    __builtin_amdgcn_sched_barrier(0);
    rm_f32x4 acc[NT][4];
#pragma unroll
    for (int tt = 0; tt < NT; ++tt)
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[tt][q] = rm_f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int k = 0; k < CPW; ++k)
        if (wave + k * kGuWaves < n) dn_mma<NT, CW>(cb[k], acc);
    auto red = reinterpret_cast<rm_f32x4(*)[NT][CW][64]>(lds);  // [wave][token tile][column call][lane]
#pragma unroll
    for (int tt = 0; tt < NT; ++tt)
#pragma unroll
        for (int q = 0; q < CW; ++q) red[wave][tt][q][lane] = acc[tt][q];
    __syncthreads();
    // Wave w sums token tile w / 2 and column calls qc .. qc + CW / 2 - 1 (qc = (w % 2) CW / 2) over the 8 waves in
    // wave order and stores that part of the slice's partial.
    constexpr int QW = CW / 2;  // column calls per wave
    const int tt = wave >> 1;
    const int qc = (wave & 1) * QW;
    rm_f32x4 v[QW];
#pragma unroll
    for (int j = 0; j < QW; ++j) {
        v[j] = red[0][tt][qc + j][lane];
#pragma unroll
        for (int w = 1; w < kGuWaves; ++w) v[j] += red[w][tt][qc + j][lane];
    }
    if (!colok) return;
    const float nan = __builtin_nanf("");
    const bool bad = s_fail != 0;
    float *P = a.part + static_cast<size_t>(x) * g.T * g.d + colw + qc;  // physical columns CW nn + qc + j
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int t = tt * 16 + grp * 4 + i;  // lane L, register i: token 4 (L / 16) + i of the tile
        if (t < g.T) {
            if constexpr (QW == 2) {
                float2 o;
                o.x = bad ? nan : v[0][i];
                o.y = bad ? nan : v[1][i];
                *reinterpret_cast<float2 *>(P + static_cast<size_t>(t) * g.d) = o;
            } else {
                P[static_cast<size_t>(t) * g.d] = bad ? nan : v[0][i];
            }
        }
    }
}

// Down projection with the epilogue fused, for lists of at most kDfMaxChunks chunks.  Workgroup: one column
// tile of 16 CW columns (CW = 2 or 4 per lane), NT tiles of 16 tokens, one sample; its 8 waves take the list's
// chunks in turn (chunk wave + 8 k, k < CPW: every load is issued before the first product), each keeping NT x CW
// 16 x 16 fp32 tiles, and the 8 waves' tiles are summed in wave order through LDS, one token tile at a time.
// Then y = x + acc (x + (y_a + acc) for Eq. 4), y_a = acc on an anchor step, and inside a stack the next layer's
// input xn = y * g in bf16 with the row's partial sums of squares for its 32-column blocks.  No partials leave
// the workgroup, so no epilogue launch follows.
struct DfArgs {
    const uint16_t *H, *wd;
    const int32_t *idx, *count;
    int d_ff, d, T, tpad, kcap, max_count, B, ncol, ntt;
    const float *x;
    float *y;
    const float *ya_in;
    float *ya_out;
    const float *out_gate;  // [B][d] adaptive output gate, or null
    const float *g_next;    // with xn_next: the next layer's norm gain, or null for no norm
    uint16_t *xn_next;    // the next layer's FFN input, or null
    float *ssq;
};

template <int N>
using f32v = float __attribute__((ext_vector_type(N)));

// CPS < CPW: the chunks go in stages of CPS (each stage's loads, then its products), so that the four 16-token
// tiles of a whole 64-token block (several samples) fit the registers: one workgroup per (sample, column tile)
// then reads the sample's listed rows of its columns once, and the grid is one round.
template <int CPW, int NT, int CW, int CPS = CPW>
__global__ __launch_bounds__(kDfThreads) void down_fused_kernel(DfArgs a) {
    static_assert(CW == 2 || CW == 4, "two or four columns per lane");
    constexpr int STAGES = (CPW + CPS - 1) / CPS;
    using vec = f32v<CW>;
    const int q = xcd_logical(blockIdx.x, gridDim.x);  // = (sample * ncol + column tile) * ntt + token tile
    const int tt = q % a.ntt;
    const int ct = (q / a.ntt) % a.ncol;
    const int b = q / (a.ntt * a.ncol);
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int grp = lane >> 4;  // K group: slots 8*grp .. 8*grp+7 of a chunk
    const int nn = lane & 15;   // A row (token in tile) and B column group (physical columns CW*nn + q)
    const int colw = (ct * 16 + nn) * CW;
    const bool colok = colw < a.d;
    const int col = min(colw, a.d - CW);  // columns past d re-read the last CW columns; those are not stored
    const int nchunks = a.kcap / rm::kBfChunk;
    const int t0 = tt * 16 * NT;  // NT tiles of 16 tokens
    const uint16_t *Hb = a.H + static_cast<size_t>(b) * a.tpad * a.kcap;

    // The list's neuron indices (clamped into [0, d_ff)) are staged once in LDS.
    constexpr int kIdxPerThread = rm::kDfMaxChunks * rm::kBfChunk / kDfThreads;
    __shared__ __attribute__((aligned(16))) int sidx[rm::kDfMaxChunks * rm::kBfChunk];
    int iv[kIdxPerThread];
#pragma unroll
    for (int i = 0; i < kIdxPerThread; ++i)
        iv[i] = a.idx[static_cast<size_t>(b) * a.d_ff + min(min(tid + i * kDfThreads, a.kcap - 1), a.d_ff - 1)];
    int cnt = a.count[b];
    // The epilogue's inputs depend on nothing computed here, so they are loaded now and the epilogue does not
    // wait for memory a second time.  Wave w < 4 finishes token t0 + 16 j + 4 grp + w of tile j (waves 4-7 load
    // the same rows and drop them).  An anchor's y_a goes out first, right behind the indices: the compiler waits
    // for the loads before it inside that branch, and the indices are needed next anyway.
    size_t ro[NT];
    vec x_in[NT], ya_in[NT];
#pragma unroll
    for (int j = 0; j < NT; ++j)
        ro[j] = (static_cast<size_t>(b) * a.T + min(t0 + j * 16 + grp * 4 + (wave & 3), a.T - 1)) * a.d + col;
    if (a.ya_in != nullptr)
#pragma unroll
        for (int j = 0; j < NT; ++j) ya_in[j] = *reinterpret_cast<const vec *>(a.ya_in + ro[j]);
    __builtin_amdgcn_sched_barrier(0);  // the index loads go out first

    auto chunk_of = [&](int k) { return min(wave + k * rm::kDfWaves, nchunks - 1); };
    DnChunk<NT> cb[CPS];
    auto load_h = [&](int stage) {  // chunk-major H: 16 tokens x 64 bytes, one contiguous kilobyte per tile
#pragma unroll
        for (int k = 0; k < CPS; ++k)
            if (stage * CPS + k < CPW)
#pragma unroll
                for (int j = 0; j < NT; ++j)
                    cb[k].a[j] = load16(Hb +
                                        (static_cast<size_t>(chunk_of(stage * CPS + k)) * a.tpad + t0 + j * 16 + nn) *
                                            rm::kBfChunk +
                                        grp * 8);
    };
    load_h(0);
#pragma unroll
    for (int j = 0; j < NT; ++j) x_in[j] = *reinterpret_cast<const vec *>(a.x + ro[j]);
    // The gates load unconditionally (under its branch the compiler waited there for every load in flight): a
    // gate the call does not have reads x instead, and its value is not used.
    const vec gate =
        *reinterpret_cast<const vec *>((a.out_gate != nullptr ? a.out_gate + static_cast<size_t>(b) * a.d : a.x) + col);
    const vec g_next = *reinterpret_cast<const vec *>((a.g_next != nullptr ? a.g_next : a.x) + col);
    __builtin_amdgcn_sched_barrier(0);  // then the H tiles, before the wait for the indices
#pragma unroll
    for (int i = 0; i < kIdxPerThread; ++i) {
        const int s = tid + i * kDfThreads;
        if (s < a.kcap) sidx[s] = clamp_neuron(iv[i], a.d_ff);
    }
    __syncthreads();
    auto load_w = [&](int stage) {
#pragma unroll
        for (int k = 0; k < CPS; ++k) {
            if (stage * CPS + k >= CPW) continue;
            const int kb = chunk_of(stage * CPS + k) * rm::kBfChunk + grp * 8;
            const int4 i0 = *reinterpret_cast<const int4 *>(sidx + kb);
            const int4 i1 = *reinterpret_cast<const int4 *>(sidx + kb + 4);
            const int n[8] = {i0.x, i0.y, i0.z, i0.w, i1.x, i1.y, i1.z, i1.w};
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const uint16_t *wp = a.wd + static_cast<size_t>(n[j]) * a.d + col;
                if constexpr (CW == 4) cb[k].w[j] = load8(wp);
                else cb[k].w[j] = make_uint2(*reinterpret_cast<const uint32_t *>(wp), 0u);
            }
        }
    };

    rm_f32x4 acc[NT][4];
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
        for (int c = 0; c < CW; ++c) acc[j][c] = rm_f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int stage = 0; stage < STAGES; ++stage) {
        if (stage > 0) load_h(stage);
        load_w(stage);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int k = 0; k < CPS; ++k) {
            const int kk = stage * CPS + k;
            if (kk >= CPW) continue;
            if constexpr (STAGES == 1) {
                if (wave + kk * rm::kDfWaves < nchunks) dn_mma<NT, CW>(cb[k], acc);
            } else {  // a chunk past the list enters with a zero H tile (exact zeros) rather than under a branch,
                      // which would let the compiler move this stage's loads into it
                if (wave + kk * rm::kDfWaves >= nchunks)
#pragma unroll
                    for (int j = 0; j < NT; ++j) cb[k].a[j] = zero16();
                dn_mma<NT, CW>(cb[k], acc);
            }
        }
        __builtin_amdgcn_sched_barrier(0);
    }

    __shared__ rm_f32x4 red[rm::kDfWaves][CW][64];
    cnt = cnt < 0 ? 0 : (cnt > a.max_count ? a.max_count : cnt);
    const int ssq_stride = rm::ssq_stride(a.d);
    // The 32-column block of this lane's columns, and whether the lane is its first (it stores the sum).
    const int part = colw / rm::kSsqCols;
    const bool part_lead = (nn & (rm::kSsqCols / CW - 1)) == 0;
#pragma unroll
    for (int j = 0; j < NT; ++j) {
        if (j > 0) __syncthreads();  // tile j - 1's sums have been read
#pragma unroll
        for (int c = 0; c < CW; ++c) red[wave][c][lane] = acc[j][c];
        __syncthreads();
        if (wave >= 4) continue;
        // Wave i finishes token 4 * grp + i of tile j (lane L, register i of a tile: token 4*(L/16)+i,
        // physical column CW*(L%16) + q of call q): the 8 waves' sums in wave order.
        const int i = wave;
        vec acc_v;
#pragma unroll
        for (int c = 0; c < CW; ++c) {
            float v = red[0][c][lane][i];
#pragma unroll
            for (int w = 1; w < rm::kDfWaves; ++w) v += red[w][c][lane][i];
            acc_v[c] = v;
        }
        const int t = t0 + j * 16 + grp * 4 + i;
        const bool live = t < a.T;
        vec out = x_in[j];
        if (a.ya_in != nullptr || cnt > 0) {  // an empty list without an anchor leaves y = x bit for bit
            vec f = acc_v;
            if (a.ya_in != nullptr) f = ya_in[j] + acc_v;  // Eq. 4: the FFN output is y_a + (h - h_a) W_down
            if (a.out_gate != nullptr) f = f * gate;       // the adaptive output gate, before the residual
            out = out + f;
        }
        const bool st = live && colok;
        if (st) {
            *reinterpret_cast<vec *>(a.y + ro[j]) = out;
            if (a.ya_out != nullptr) *reinterpret_cast<vec *>(a.ya_out + ro[j]) = acc_v;
        }
        if (a.xn_next == nullptr) continue;
        if (a.g_next != nullptr) {
            float ss;
            if constexpr (CW == 4) ss = rm_ssq32(make_float4(out[0], out[1], out[2], out[3]), colok);
            else ss = rm_ssq32_pairs(out[0], out[1], colok);
            const int row = b * a.T + t;
            if (part_lead && st) a.ssq[static_cast<size_t>(row) * ssq_stride + part] = ss;
            out = out * g_next;
        }
        if (st) {
            if constexpr (CW == 4) {
                uint2 packed;
                packed.x = rm_f32_to_bf16_bits(out[0]) | (rm_f32_to_bf16_bits(out[1]) << 16);
                packed.y = rm_f32_to_bf16_bits(out[2]) | (rm_f32_to_bf16_bits(out[3]) << 16);
                *reinterpret_cast<uint2 *>(a.xn_next + ro[j]) = packed;
            } else {
                *reinterpret_cast<uint32_t *>(a.xn_next + ro[j]) =
                    rm_f32_to_bf16_bits(out[0]) | (rm_f32_to_bf16_bits(out[1]) << 16);
            }
        }
    }
}

int token_tiles(int T) {
    const int tiles = (T + 15) / 16;
    return tiles >= 4 ? 4 : tiles;
}

template <int NT>
hipError_t launch_gateup_nt(const rm::Plan &p, const GuArgs &a, hipStream_t st) {
    hipError_t e = hipSuccess;
    const dim3 block(kGuThreads);
    const dim3 grid(p.gate_blocks * p.B);
    if (p.gate_groups == 1) {
        if (p.T <= rm::kBfTokBlock) {
            switch (p.d / 256) {  // the plan picks the direct kernel only for d = 256, 512, 1024, 2048
                case 1:
                    e = launch_timed(RM_KERNEL_GATEUP, gateup_direct_kernel<NT, 1, true>, grid, block, st, a);
                    break;
                case 2:
                    e = launch_timed(RM_KERNEL_GATEUP, gateup_direct_kernel<NT, 2, true>, grid, block, st, a);
                    break;
                case 4:
                    e = launch_timed(RM_KERNEL_GATEUP, gateup_direct_kernel<NT, 4, true>, grid, block, st, a);
                    break;
                default:
                    e = launch_timed(RM_KERNEL_GATEUP, gateup_direct_kernel<NT, 8, true>, grid, block, st, a);
                    break;
            }
        } else {
            switch (p.d / 256) {
                case 1:
                    e = launch_timed(RM_KERNEL_GATEUP, gateup_direct_kernel<NT, 1, false>, grid, block, st, a);
                    break;
                case 2:
                    e = launch_timed(RM_KERNEL_GATEUP, gateup_direct_kernel<NT, 2, false>, grid, block, st, a);
                    break;
                case 4:
                    e = launch_timed(RM_KERNEL_GATEUP, gateup_direct_kernel<NT, 4, false>, grid, block, st, a);
                    break;
                default:
                    e = launch_timed(RM_KERNEL_GATEUP, gateup_direct_kernel<NT, 8, false>, grid, block, st, a);
                    break;
            }
        }
        return e;
    }
    const int nch = (p.d + kChunkCols - 1) / kChunkCols;
    if (p.T <= rm::kBfTokBlock && p.d % kChunkCols == 0 && (nch == 1 || nch == 2 || nch == 4 || nch == 8)) {
#define RM_PIPE(NG, TWO)                                                                                    \
    switch (nch) {                                                                                          \
        case 1: e = launch_timed(RM_KERNEL_GATEUP, gateup_pipe_kernel<NG, 1, TWO>, grid, block, st, a); break; \
        case 2: e = launch_timed(RM_KERNEL_GATEUP, gateup_pipe_kernel<NG, 2, TWO>, grid, block, st, a); break; \
        case 4: e = launch_timed(RM_KERNEL_GATEUP, gateup_pipe_kernel<NG, 4, TWO>, grid, block, st, a); break; \
        default: e = launch_timed(RM_KERNEL_GATEUP, gateup_pipe_kernel<NG, 8, TWO>, grid, block, st, a); break; \
    }
        const bool two = static_cast<long long>(p.gate_blocks) * p.B > 256;  // more workgroups than compute units
        switch (p.gate_groups) {
            case 2: RM_PIPE(2, true) break;
            case 4:
                if (two) RM_PIPE(4, true) else RM_PIPE(4, false)
                break;
            default:
                if (two) RM_PIPE(8, true) else RM_PIPE(8, false)
                break;
        }
#undef RM_PIPE
        return e;
    }
#define RM_STAGED(NG)                                                                                    \
    switch (nch) {                                                                                       \
        case 1: e = launch_timed(RM_KERNEL_GATEUP, gateup_staged_unrolled_kernel<NT, NG, 1>, grid, block, st, a); \
            break;                                                                                       \
        case 2: e = launch_timed(RM_KERNEL_GATEUP, gateup_staged_unrolled_kernel<NT, NG, 2>, grid, block, st, a); \
            break;                                                                                       \
        case 3: e = launch_timed(RM_KERNEL_GATEUP, gateup_staged_unrolled_kernel<NT, NG, 3>, grid, block, st, a); \
            break;                                                                                       \
        case 4: e = launch_timed(RM_KERNEL_GATEUP, gateup_staged_unrolled_kernel<NT, NG, 4>, grid, block, st, a); \
            break;                                                                                       \
        case 8: /* 8 chunks x 8 groups: the unrolled form spills */                                      \
            if (NG < 8)                                                                                  \
                e = launch_timed(RM_KERNEL_GATEUP, gateup_staged_unrolled_kernel<NT, NG, 8>, grid, block, st, a); \
            else                                                                                         \
                e = launch_timed(RM_KERNEL_GATEUP, gateup_staged_kernel<NT, NG>, grid, block, st, a);         \
            break;                                                                                       \
        default: e = launch_timed(RM_KERNEL_GATEUP, gateup_staged_kernel<NT, NG>, grid, block, st, a); break; \
    }
    switch (p.gate_groups) {
        case 2: RM_STAGED(2) break;
        case 4: RM_STAGED(4) break;
        default: RM_STAGED(8) break;
    }
#undef RM_STAGED
    return e;
}

}  // namespace

namespace rm {

static hipError_t launch_gateup_args(const Plan &p, const GuArgs &a, hipStream_t st);

hipError_t launch_gateup_bf16(const Plan &p, const void *w_gate, const void *w_up, const int32_t *idx,
                              const int32_t *count, bool norm, const float *h_anchor, float *h_out, void *ws,
                              hipStream_t st) {
    char *base = static_cast<char *>(ws);
    GuArgs a{};
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
    a.B = p.B;
    a.act = p.act;
    a.H = reinterpret_cast<uint16_t *>(base + p.off_h);
    a.h_anchor = h_anchor;
    a.h_out = h_out;
    return launch_gateup_args(p, a, st);
}

static hipError_t launch_gateup_args(const Plan &p, const GuArgs &a, hipStream_t st) {
    hipError_t e;
    if (p.gate_spread > 0) {  // one sample, T <= 64, d = 256 NCH (the plan's conditions)
        const dim3 grid(p.gate_blocks), block(kGuThreads);
#define RM_SPREAD(NG)                                                                                       \
    switch (p.d / kChunkCols) {                                                                             \
        case 1: e = launch_timed(RM_KERNEL_GATEUP, gateup_spread_kernel<NG, 1>, grid, block, st, a); break; \
        case 2: e = launch_timed(RM_KERNEL_GATEUP, gateup_spread_kernel<NG, 2>, grid, block, st, a); break; \
        case 4: e = launch_timed(RM_KERNEL_GATEUP, gateup_spread_kernel<NG, 4>, grid, block, st, a); break; \
        default: e = launch_timed(RM_KERNEL_GATEUP, gateup_spread_kernel<NG, 8>, grid, block, st, a); break; \
    }
        if (p.gate_spread == 1)  // the plan's range: 1 to 3 tiles
            RM_SPREAD(1)
        else if (p.gate_spread == 2)
            RM_SPREAD(2)
        else
            RM_SPREAD(3)
#undef RM_SPREAD
        return e != hipSuccess ? e : hipGetLastError();
    }
    switch (token_tiles(p.T)) {
        case 1: e = launch_gateup_nt<1>(p, a, st); break;
        case 2: e = launch_gateup_nt<2>(p, a, st); break;
        case 3: e = launch_gateup_nt<3>(p, a, st); break;
        default: e = launch_gateup_nt<4>(p, a, st); break;
    }
    return e != hipSuccess ? e : hipGetLastError();
}

hipError_t launch_down_fused(const Plan &p, const void *w_down, const int32_t *idx, const int32_t *count,
                             const float *x, float *y, const float *g_next, bool emit_xn, const float *ya_in,
                             float *ya_out, const float *out_gate, void *ws, hipStream_t st) {
    char *base = static_cast<char *>(ws);
    DfArgs a;
    a.H = reinterpret_cast<const uint16_t *>(base + p.off_h);
    a.wd = static_cast<const uint16_t *>(w_down);
    a.idx = idx;
    a.count = count;
    a.d_ff = p.d_ff;
    a.d = p.d;
    a.T = p.T;
    a.tpad = p.tpad;
    a.kcap = p.kcap;
    a.max_count = p.max_count;
    a.B = p.B;
    a.ncol = p.df_ncol;
    a.ntt = p.ntt;
    a.x = x;
    a.y = y;
    a.ya_in = ya_in;
    a.ya_out = ya_out;
    a.out_gate = out_gate;
    a.g_next = emit_xn ? g_next : nullptr;
    a.xn_next = emit_xn ? reinterpret_cast<uint16_t *>(base + p.off_xn) : nullptr;
    a.ssq = reinterpret_cast<float *>(base + p.off_ssq);
    const dim3 grid(p.df_ncol * p.ntt * p.B);
    const dim3 block(kDfThreads);
    hipError_t e;
#define RM_DF(NT, CW)                                                                                         \
    switch (p.dn_cpw) {                                                                                       \
        case 1: e = launch_timed(RM_KERNEL_DOWN, down_fused_kernel<1, NT, CW>, grid, block, st, a); break;    \
        case 2: e = launch_timed(RM_KERNEL_DOWN, down_fused_kernel<2, NT, CW>, grid, block, st, a); break;    \
        case 3: e = launch_timed(RM_KERNEL_DOWN, down_fused_kernel<3, NT, CW>, grid, block, st, a); break;    \
        case 4: e = launch_timed(RM_KERNEL_DOWN, down_fused_kernel<4, NT, CW>, grid, block, st, a); break;    \
        case 5: e = launch_timed(RM_KERNEL_DOWN, down_fused_kernel<5, NT, CW>, grid, block, st, a); break;    \
        case 6: e = launch_timed(RM_KERNEL_DOWN, down_fused_kernel<6, NT, CW>, grid, block, st, a); break;    \
        case 7: e = launch_timed(RM_KERNEL_DOWN, down_fused_kernel<7, NT, CW>, grid, block, st, a); break;    \
        default: e = launch_timed(RM_KERNEL_DOWN, down_fused_kernel<8, NT, CW>, grid, block, st, a); break;   \
    }
    // The plan pairs one 16-token tile with 2 columns per lane (one sample) and four with 4 (several samples).
    if (p.df_nt == 4 && p.df_cw == 4) {
        // Several samples: one 64-token block per workgroup, chunks in stages of 3 (at most 8 per wave).
        switch (p.dn_cpw) {
            case 1: e = launch_timed(RM_KERNEL_DOWN, down_fused_kernel<1, 4, 4, 3>, grid, block, st, a); break;
            case 2: e = launch_timed(RM_KERNEL_DOWN, down_fused_kernel<2, 4, 4, 3>, grid, block, st, a); break;
            case 3: e = launch_timed(RM_KERNEL_DOWN, down_fused_kernel<3, 4, 4, 3>, grid, block, st, a); break;
            case 4: e = launch_timed(RM_KERNEL_DOWN, down_fused_kernel<4, 4, 4, 3>, grid, block, st, a); break;
            case 5: e = launch_timed(RM_KERNEL_DOWN, down_fused_kernel<5, 4, 4, 3>, grid, block, st, a); break;
            case 6: e = launch_timed(RM_KERNEL_DOWN, down_fused_kernel<6, 4, 4, 3>, grid, block, st, a); break;
            case 7: e = launch_timed(RM_KERNEL_DOWN, down_fused_kernel<7, 4, 4, 3>, grid, block, st, a); break;
            default: e = launch_timed(RM_KERNEL_DOWN, down_fused_kernel<8, 4, 4, 3>, grid, block, st, a); break;
        }
    } else if (p.df_nt == 1 && p.df_cw == 2) {
        RM_DF(1, 2)
    }
    else
        return hipErrorInvalidValue;
#undef RM_DF
    return e != hipSuccess ? e : hipGetLastError();
}

hipError_t launch_layer_xcd(const Plan &p, const void *w_gate, const void *w_up, const void *w_down,
                            const int32_t *idx, const int32_t *count, const float *xin, const float *norm_g,
                            const float *h_anchor, void *ws, hipStream_t st) {
    char *base = static_cast<char *>(ws);
    XlArgs a{};
    GuArgs &g = a.g;
    g.wg = static_cast<const uint16_t *>(w_gate);
    g.wu = static_cast<const uint16_t *>(w_up);
    g.xn = reinterpret_cast<const uint16_t *>(base + p.off_xn8);
    g.idx = idx;
    g.count = count;
    g.ssq = norm_g != nullptr ? reinterpret_cast<const float *>(base + p.off_ssq8) : nullptr;
    g.eps = p.eps;
    g.max_count = p.max_count;
    g.d_ff = p.d_ff;
    g.d = p.d;
    g.T = p.T;
    g.tpad = p.tpad;
    g.kcap = p.kcap;
    g.B = 1;
    g.act = p.act;
    g.H = reinterpret_cast<uint16_t *>(base + p.off_h);
    g.h_anchor = h_anchor;
    g.h_out = nullptr;
    a.x = xin;
    a.norm_g = norm_g;
    a.xn8 = reinterpret_cast<uint16_t *>(base + p.off_xn8);
    a.ssq8 = reinterpret_cast<float *>(base + p.off_ssq8);
    a.wd = static_cast<const uint16_t *>(w_down);
    a.part = reinterpret_cast<float *>(base + p.off_part);
    a.flags = reinterpret_cast<unsigned long long *>(base + p.off_sync);
    a.ctr = reinterpret_cast<unsigned *>(base + p.off_sync + kXcdFlagBytes);
    a.zero = 0u;
    a.cps = p.slice_units;
    a.spin_ticks = kXcdSpinTicks;
    // The plan's conditions: B = 1, T <= 64, d = 2048 or 1024 (32 column tiles of 64 or 32 columns, one per
    // workgroup of an XCD), slices of at most 24 chunks, 256 workgroups.
    if (p.B != 1 || p.T > kBfTokBlock || (p.d != 8 * kChunkCols && p.d != 4 * kChunkCols) || p.slice_units < 1 ||
        p.slice_units > 3 * kGuWaves || p.slices > 8)
        return hipErrorInvalidValue;
    const dim3 grid(8 * kXlPerXcd), block(kGuThreads);
    const int cpw = (p.slice_units + kGuWaves - 1) / kGuWaves;
    hipError_t e;
#define RM_XL(NCH, CW)                                                                                   \
    switch (cpw) {                                                                                       \
        case 1: e = launch_timed(RM_KERNEL_LAYER, layer_xcd_kernel<NCH, 1, CW>, grid, block, st, a); break; \
        case 2: e = launch_timed(RM_KERNEL_LAYER, layer_xcd_kernel<NCH, 2, CW>, grid, block, st, a); break; \
        default: e = launch_timed(RM_KERNEL_LAYER, layer_xcd_kernel<NCH, 3, CW>, grid, block, st, a); break; \
    }
    if (p.d == 8 * kChunkCols) {
        RM_XL(8, 4)
    } else {
        RM_XL(4, 2)
    }
#undef RM_XL
    return e != hipSuccess ? e : hipGetLastError();
}

hipError_t launch_down_bf16(const Plan &p, const void *w_down, const int32_t *idx, void *ws, hipStream_t st) {
    char *base = static_cast<char *>(ws);
    DnArgs a;
    a.H = reinterpret_cast<const uint16_t *>(base + p.off_h);
    a.wd = static_cast<const uint16_t *>(w_down);
    a.idx = idx;
    a.d_ff = p.d_ff;
    a.d = p.d;
    a.T = p.T;
    a.tpad = p.tpad;
    a.kcap = p.kcap;
    a.slices = p.slices;
    a.chunks_per_slice = p.slice_units;
    a.B = p.B;
    a.ncol = p.ncol;
    a.part = reinterpret_cast<float *>(base + p.off_part);
    const dim3 grid(p.ncol * p.slices * p.B), block(kDnThreads);
    hipError_t e = hipSuccess;
#define RM_DOWN_CPW(NT, ONE)                                                                              \
    switch (p.slice_units / kDnWaves) {                                                                  \
        case 1: e = launch_timed(RM_KERNEL_DOWN, down_bf16_kernel<NT, 1, ONE>, grid, block, st, a); break;    \
        case 2: e = launch_timed(RM_KERNEL_DOWN, down_bf16_kernel<NT, 2, ONE>, grid, block, st, a); break;    \
        case 3: e = launch_timed(RM_KERNEL_DOWN, down_bf16_kernel<NT, 3, ONE>, grid, block, st, a); break;    \
        case 4: e = launch_timed(RM_KERNEL_DOWN, down_bf16_kernel<NT, 4, ONE>, grid, block, st, a); break;    \
        case 5: e = launch_timed(RM_KERNEL_DOWN, down_bf16_kernel<NT, 5, ONE>, grid, block, st, a); break;    \
        case 6: e = launch_timed(RM_KERNEL_DOWN, down_bf16_kernel<NT, 6, ONE>, grid, block, st, a); break;    \
        case 7: e = launch_timed(RM_KERNEL_DOWN, down_bf16_kernel<NT, 7, ONE>, grid, block, st, a); break;    \
        default: e = launch_timed(RM_KERNEL_DOWN, down_bf16_kernel<NT, 8, ONE>, grid, block, st, a); break;   \
    }
#define RM_DOWN(NT)                          \
    if (p.T <= rm::kBfTokBlock) {            \
        RM_DOWN_CPW(NT, true)                \
    } else {                                 \
        RM_DOWN_CPW(NT, false)               \
    }
    switch (token_tiles(p.T)) {
        case 1: RM_DOWN(1) break;
        case 2: RM_DOWN(2) break;
        case 3: RM_DOWN(3) break;
        default: RM_DOWN(4) break;
    }
#undef RM_DOWN
#undef RM_DOWN_CPW
    return e != hipSuccess ? e : hipGetLastError();
}

}  // namespace rm
