// C ABI entry points: argument validation, launch plan / workspace layout, and the layer and stack drivers.
//
// A call enqueues on the caller's stream: the prologue (the first layer's FFN input and its sums of squares),
// then per layer the gathered gate/up projection (H), the gathered down projection (per-K-slice partials) and
// the epilogue (y = x + the partials in slice order, plus the next layer's FFN input inside a stack).  Layers
// after the first run in place on y.  Nothing here synchronizes or allocates.
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <mutex>

#include "rm_select.h"

#define RM_EXPORT extern "C" __attribute__((visibility("default")))

// Scratch of rm_sparse_ffn_layer_noalloc, for callers that cannot allocate a workspace: every GPU the library
// runs on holds its own copy of this array until the process ends, and every call of that entry point on the GPU
// shares it.  Host code never uses the name itself (on the host it is only a stand-in for the symbol): kernels
// get the device address that hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) unsigned char scratch[RM_NOALLOC_SCRATCH_BYTES];

namespace {

thread_local char g_last_error[512] = "";

struct ProfileSlot {
    hipEvent_t begin = nullptr;
    hipEvent_t end = nullptr;
};
thread_local ProfileSlot g_profile[5];

rm_status fail(rm_status st, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
    va_end(ap);
    return st;
}

rm_status ok() {
    g_last_error[0] = '\0';
    return RM_OK;
}

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }
int ceil_div(int a, int b) { return (a + b - 1) / b; }
bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

rm_status check_shape(const rm_ffn_shape *s) {
    if (s == nullptr) return fail(RM_ERR_INVALID_ARG, "shape pointer is NULL");
    if (s->d <= 0 || s->d_ff <= 0) return fail(RM_ERR_INVALID_ARG, "d=%d and d_ff=%d must be positive", s->d, s->d_ff);
    if (s->d % 32 != 0) return fail(RM_ERR_SHAPE, "d=%d must be a multiple of 32", s->d);
    if (s->wdtype != RM_F32 && s->wdtype != RM_BF16) return fail(RM_ERR_DTYPE, "unknown weight dtype %d", s->wdtype);
    if (!(s->norm_eps >= 0.0f)) return fail(RM_ERR_INVALID_ARG, "norm_eps must be >= 0");
    if (s->act != RM_ACT_SILU && s->act != RM_ACT_GELU_TANH) return fail(RM_ERR_INVALID_ARG, "unknown act %d", s->act);
    return RM_OK;
}

rm_status check_layer(const rm_ffn_layer_weights *w, int l) {
    if (w == nullptr) return fail(RM_ERR_INVALID_ARG, "weights pointer is NULL");
    if (!w->w_gate || !w->w_up || !w->w_down)
        return fail(RM_ERR_INVALID_ARG, "layer %d: a weight pointer is NULL", l);
    if (!aligned(w->w_gate, 16) || !aligned(w->w_up, 16) || !aligned(w->w_down, 16) ||
        (w->norm_g && !aligned(w->norm_g, 16)) || (w->out_gate && !aligned(w->out_gate, 16)))
        return fail(RM_ERR_ALIGN, "layer %d: weight, gain and gate pointers must be 16-byte aligned", l);
    return RM_OK;
}

bool ranges_overlap(const void *a, size_t na, const void *b, size_t nb) {
    const uintptr_t pa = reinterpret_cast<uintptr_t>(a), pb = reinterpret_cast<uintptr_t>(b);
    return pa < pb + nb && pb < pa + na;
}

// Common checks of a layer / stack / dense call; fills the plan.
rm_status check_call(const rm_ffn_shape *s, int B, int T, const float *x, float *y, const int32_t *idx,
                     const int32_t *count, bool sparse, int max_count, void *ws, size_t ws_bytes, rm::Plan *p,
                     unsigned form = 0) {
    rm_status st = check_shape(s);
    if (st != RM_OK) return st;
    if (B <= 0 || T <= 0) return fail(RM_ERR_INVALID_ARG, "B=%d and T=%d must be positive", B, T);
    if (B > 65535) return fail(RM_ERR_SHAPE, "B=%d exceeds 65535", B);
    if (!x || !y) return fail(RM_ERR_INVALID_ARG, "x or y is NULL");
    if (!aligned(x, 16) || !aligned(y, 16)) return fail(RM_ERR_ALIGN, "x and y must be 16-byte aligned");
    const size_t act_bytes = static_cast<size_t>(B) * T * s->d * sizeof(float);
    if (x != y && ranges_overlap(x, act_bytes, y, act_bytes))
        return fail(RM_ERR_INVALID_ARG, "y overlaps x without being equal to it");
    if (sparse) {
        if (!idx || !count) return fail(RM_ERR_INVALID_ARG, "idx or count is NULL");
        if (!aligned(idx, 4) || !aligned(count, 4)) return fail(RM_ERR_ALIGN, "idx and count must be 4-byte aligned");
        if (max_count < 0 || max_count > s->d_ff)
            return fail(RM_ERR_SHAPE, "max_count=%d outside [0, d_ff=%d]", max_count, s->d_ff);
    }
    st = rm::make_plan(s, B, T, sparse ? max_count : s->d_ff, p, form);
    if (st != RM_OK) return st;
    if (!ws) return fail(RM_ERR_INVALID_ARG, "workspace is NULL");
    if (!aligned(ws, 16)) return fail(RM_ERR_ALIGN, "workspace must be 16-byte aligned");
    if (ws_bytes < p->total)
        return fail(RM_ERR_WORKSPACE, "workspace of %zu bytes is smaller than the %zu required", ws_bytes, p->total);
    if (ranges_overlap(ws, p->total, x, act_bytes) || ranges_overlap(ws, p->total, y, act_bytes))
        return fail(RM_ERR_INVALID_ARG, "workspace overlaps x or y");
    return RM_OK;
}

// The lists are read while y and the workspace are written: idx ([lists][B][d_ff]) and count ([lists][B]) must
// not overlap either (lists = 1 for a layer, L for a stack).  Checked last, after the per-argument checks.
rm_status check_lists(const rm_ffn_shape *s, int lists, int B, int T, const float *y, const int32_t *idx,
                      const int32_t *count, const void *ws, size_t ws_bytes) {
    const size_t act_bytes = static_cast<size_t>(B) * T * s->d * sizeof(float);
    const size_t ib = static_cast<size_t>(lists) * B * s->d_ff * 4, cb = static_cast<size_t>(lists) * B * 4;
    if (ranges_overlap(idx, ib, y, act_bytes) || ranges_overlap(idx, ib, ws, ws_bytes) ||
        ranges_overlap(count, cb, y, act_bytes) || ranges_overlap(count, cb, ws, ws_bytes))
        return fail(RM_ERR_INVALID_ARG, "idx or count overlaps y or the workspace");
    return RM_OK;
}

rm_status hip_fail(hipError_t e, const char *what) {
    return fail(RM_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// Device address of `scratch` on the current device, looked up once per device (the first call of the no-alloc
// entry point there) and kept.  The stream must belong to the current device, since each device has its own copy.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

rm_status noalloc_scratch(hipStream_t st, void **out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices) return fail(RM_ERR_INVALID_ARG, "device %d outside [0, %d)", dev, kMaxDevices);
    if (st != nullptr) {
        int sdev = -1;
        e = hipStreamGetDevice(st, &sdev);
        if (e != hipSuccess) return hip_fail(e, "hipStreamGetDevice");
        if (sdev != dev)
            return fail(RM_ERR_INVALID_ARG, "the stream belongs to device %d but device %d is current", sdev, dev);
    }
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[dev] == nullptr) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress of the no-alloc scratch");
        if (p == nullptr) return fail(RM_ERR_HIP, "hipGetSymbolAddress returned NULL for the no-alloc scratch");
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return RM_OK;
}

// The layers' output gates must not overlap y (they are read while y is written); checked by every FFN entry
// point before it enqueues anything.
rm_status check_gates(const rm_ffn_layer_weights *w, int L, int B, int T, int d, const float *y) {
    const size_t act_bytes = static_cast<size_t>(B) * T * d * sizeof(float);
    for (int l = 0; l < L; ++l)
        if (w[l].out_gate && ranges_overlap(w[l].out_gate, static_cast<size_t>(B) * d * sizeof(float), y, act_bytes))
            return fail(RM_ERR_INVALID_ARG, "layer %d: out_gate overlaps y", l);
    return RM_OK;
}

// Checks shared by the anchor and delta stacks: L, weights, the anchor buffers' sizes and overlaps.
rm_status check_anchor_buffers(const rm_ffn_shape *s, const rm_ffn_layer_weights *w, int L, int B, int T,
                               const float *x, float *y, int max_count, const void *y_anchor, const void *h_anchor,
                               const void *ws, size_t ws_bytes) {
    if (L <= 0) return fail(RM_ERR_INVALID_ARG, "L=%d must be positive", L);
    if (!w) return fail(RM_ERR_INVALID_ARG, "weights pointer is NULL");
    for (int l = 0; l < L; ++l) {
        const rm_status st = check_layer(&w[l], l);
        if (st != RM_OK) return st;
    }
    const rm_status sg = check_gates(w, L, B, T, s->d, y);
    if (sg != RM_OK) return sg;
    if (!y_anchor) return fail(RM_ERR_INVALID_ARG, "y_anchor is NULL");
    if (!h_anchor && max_count > 0) return fail(RM_ERR_INVALID_ARG, "h_anchor is NULL with max_count=%d", max_count);
    if (!aligned(y_anchor, 16) || !aligned(h_anchor, 4))
        return fail(RM_ERR_ALIGN, "y_anchor must be 16-byte and h_anchor 4-byte aligned");
    const size_t act = static_cast<size_t>(B) * T * s->d * sizeof(float);
    const size_t ya_bytes = act * L;
    const size_t ha_bytes = static_cast<size_t>(L) * B * max_count * T * sizeof(float);
    if (ranges_overlap(y_anchor, ya_bytes, h_anchor, ha_bytes) || ranges_overlap(y_anchor, ya_bytes, x, act) ||
        ranges_overlap(y_anchor, ya_bytes, y, act) || ranges_overlap(h_anchor, ha_bytes, x, act) ||
        ranges_overlap(h_anchor, ha_bytes, y, act) || ranges_overlap(y_anchor, ya_bytes, ws, ws_bytes) ||
        ranges_overlap(h_anchor, ha_bytes, ws, ws_bytes))
        return fail(RM_ERR_INVALID_ARG, "y_anchor and h_anchor must not overlap each other, x, y or the workspace");
    return RM_OK;
}

// Eq. 4 terms of an anchor or delta stack (all null for a plain call).  Per layer l:
//   ya_in  + l * B T d: y_a, added to the masked sum (delta step);
//   ya_out + l * B T d: receives the FFN output before the residual (anchor step);
//   ha_in  + l * h_stride: h_a^M, subtracted from h (delta step);
//   ha_out + l * h_stride: receives h^M of the lists cap_idx / cap_count (anchor step), computed with cap_plan,
//          which sizes the lists (its max_count) and shares the call's FFN input and sums of squares.
struct AnchorTerms {
    const float *ya_in = nullptr;
    float *ya_out = nullptr;
    const float *ha_in = nullptr;
    float *ha_out = nullptr;
    const int32_t *cap_idx = nullptr;
    const int32_t *cap_count = nullptr;
    const rm::Plan *cap_plan = nullptr;
    size_t h_stride = 0;
};

// Layers 0..L-1 of one call; w[l] are the layers' weights, lists at idx + l * list_stride and counts at
// count + l * count_stride (both strides 0 when every layer uses the same lists, as the dense calls do).
// A non-null mask ([n_masks][d_ff]) is compacted into idx / count in the prologue's launch.
rm_status run_layers(const rm::Plan &p, const rm_ffn_layer_weights *w, int L, const float *x, float *y,
                     const int32_t *idx, const int32_t *count, size_t list_stride, size_t count_stride, void *ws,
                     hipStream_t st, const AnchorTerms &at = AnchorTerms{}, const uint8_t *mask = nullptr,
                     int n_masks = 0) {
    // The one-launch layer form reads the float32 input itself: only a mask's compaction precedes it.
    hipError_t e = hipSuccess;
    if (p.xcd_layer) {
        if (mask) e = rm::launch_mask_compact(mask, n_masks, p.d_ff, const_cast<int32_t *>(idx),
                                              const_cast<int32_t *>(count), st);
    } else {
        e = mask ? rm::launch_compact_prologue(p, mask, n_masks, const_cast<int32_t *>(idx),
                                               const_cast<int32_t *>(count), x, w[0].norm_g, ws, st)
                 : rm::launch_prologue(p, x, w[0].norm_g, ws, st);
    }
    if (e != hipSuccess) return hip_fail(e, "prologue launch");
    const bool bf = p.wdtype == RM_BF16;
    const size_t y_stride = static_cast<size_t>(p.B) * p.T * p.d;
    // The fused down projection sums the whole list in each workgroup: fewer, longer workgroups than the split
    // over K, and no epilogue launch.  With one sample's 32-column tiles it is the faster form for every list
    // it takes, a single d = 1024 layer included (d_ff = 4096, 1229 neurons, T = 51: 15.6 -> 15.3 us per step).
    const bool fused = p.fused_down;
    for (int l = 0; l < L; ++l) {
        const int32_t *il = idx + l * list_stride;
        const int32_t *cl = count + l * count_stride;
        const bool norm = w[l].norm_g != nullptr;
        const float *ha = at.ha_in ? at.ha_in + l * at.h_stride : nullptr;
        if (p.xcd_layer)  // gate/up and down in one launch from the float32 input; partials to the epilogue
            e = rm::launch_layer_xcd(p, w[l].w_gate, w[l].w_up, w[l].w_down, il, cl, l == 0 ? x : y, w[l].norm_g,
                                     ha, ws, st);
        else
            e = bf ? rm::launch_gateup_bf16(p, w[l].w_gate, w[l].w_up, il, cl, norm, ha, nullptr, ws, st)
                   : rm::launch_gateup_f32(p, w[l].w_gate, w[l].w_up, il, cl, norm, ha, nullptr, ws, st);
        if (e != hipSuccess) return hip_fail(e, p.xcd_layer ? "layer launch" : "gate/up launch");
        if (at.ha_out != nullptr) {  // the anchor keeps h^M of the group's lists (same input, same norm)
            const rm::Plan &q = *at.cap_plan;
            const int32_t *ci = at.cap_idx + static_cast<size_t>(l) * p.B * p.d_ff;
            const int32_t *cc = at.cap_count + static_cast<size_t>(l) * p.B;
            float *ho = at.ha_out + l * at.h_stride;
            e = bf ? rm::launch_gateup_bf16(q, w[l].w_gate, w[l].w_up, ci, cc, norm, nullptr, ho, ws, st)
                   : rm::launch_gateup_f32(q, w[l].w_gate, w[l].w_up, ci, cc, norm, nullptr, ho, ws, st);
            if (e != hipSuccess) return hip_fail(e, "anchor h capture launch");
        }
        const bool next = l + 1 < L && !p.xcd_layer;  // the one-launch form needs no xn for the next layer
        const float *g_next = next ? w[l + 1].norm_g : nullptr;
        const float *xin = l == 0 ? x : y;
        const float *ya_in = at.ya_in ? at.ya_in + l * y_stride : nullptr;
        float *ya_out = at.ya_out ? at.ya_out + l * y_stride : nullptr;
        if (fused) {  // down projection and epilogue in one launch
            e = rm::launch_down_fused(p, w[l].w_down, il, cl, xin, y, g_next, next, ya_in, ya_out, w[l].out_gate,
                                      ws, st);
            if (e != hipSuccess) return hip_fail(e, "down launch");
            continue;
        }
        if (!p.xcd_layer) {
            e = bf ? rm::launch_down_bf16(p, w[l].w_down, il, ws, st)
                   : rm::launch_down_f32(p, w[l].w_down, il, cl, ws, st);
            if (e != hipSuccess) return hip_fail(e, "down launch");
        }
        e = rm::launch_epilogue(p, cl, xin, y, g_next, next, ya_in, ya_out, w[l].out_gate, ws, st);
        if (e != hipSuccess) return hip_fail(e, "epilogue launch");
    }
    return RM_OK;
}

// Whether the one-launch layer form may run on the current device: it has the 256 compute units (8 XCDs of 32)
// that the form needs resident at once (asked once per device), and the environment variable RM_NO_LAYER_FORM
// was not set to a non-empty value other than "0" when the process first asked (for callers that share the GPU
// with other work that can hold compute units while the form's workgroups wait for each other).
bool device_has_256_cus() {
    static const bool off = [] {
        const char *e = getenv("RM_NO_LAYER_FORM");
        return e != nullptr && e[0] != '\0' && strcmp(e, "0") != 0;
    }();
    if (off) return false;
    static std::atomic<int> known[64];  // 0 = not asked, 1 = no, 2 = yes
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) return false;
    if (dev >= 64) return false;
    int v = known[dev].load(std::memory_order_relaxed);
    if (v == 0) {
        int cus = 0;
        const bool ok = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess;
        v = ok && cus == 256 ? 2 : 1;
        known[dev].store(v, std::memory_order_relaxed);
    }
    return v == 2;
}

}  // namespace

namespace rm {

rm_status make_plan(const rm_ffn_shape *s, int B, int T, int max_count, Plan *p, unsigned form) {
    Plan q;
    q.d = s->d;
    q.d_ff = s->d_ff;
    q.wdtype = s->wdtype;
    q.B = B;
    q.T = T;
    q.max_count = max_count;
    q.eps = s->norm_eps;
    q.act = s->act;
    const int kmax = max_count > 0 ? max_count : 1;
    size_t xn_elem, h_elem;
    bool xcd_shape = false, xcd_room = false;
    int part_slices = 0;  // partial slices the workspace holds (at least q.slices)
    // Aim for one down-projection workgroup per compute unit (256 CUs): a grid just past a multiple of the unit
    // count leaves the units with one more workgroup setting the time (d = 2048, 4916 neurons: 8 slices of 20 chunks,
    // 256 workgroups, instead of 10 slices of 16, 320: down 10.0 -> 8.1 us), and fewer K-slices mean fewer
    // float32 partials written and read back by the epilogue.
    constexpr int kCUs = 256;
#ifndef RM_DOWN_TARGET
#define RM_DOWN_TARGET 256
#endif
    constexpr int kTargetDownGroups = RM_DOWN_TARGET;
    if (s->wdtype == RM_BF16) {
        q.tpad = ceil_div(T, kBfTokBlock) * kBfTokBlock;
        // Gate/up workgroups of 8 * NG neurons.  Measured at d = 2048 (one sample) and d = 1024 (16 samples):
        // one round of workgroups that fills most compute units is best (the widest NG with 150 .. 256
        // workgroups); a grid just past the compute units (256 .. 384 workgroups) is the worst case, since the
        // compute units that get a second workgroup set the time, so a grid there takes the next narrower NG
        // (more, lighter workgroups); otherwise the widest NG that still gives every compute unit one
        // workgroup, or one group of 8 per workgroup (the direct kernel, when d allows) for short lists.
        const int k32 = ceil_div(kmax, kBfChunk) * kBfChunk;
        const bool direct_ok = s->d == 256 || s->d == 512 || s->d == 1024 || s->d == 2048;
        // One sample with more groups of 8 slots than compute units (up to 3 per unit): the spread kernel, one
        // workgroup per compute unit taking quads of 4 slots round-robin, so that every unit streams weights and
        // the units' weight bytes differ by one quad at most.
        const int n8 = k32 / 8;
        const bool spread = RM_GATEUP_SPREAD && B == 1 && T <= kBfTokBlock && direct_ok && n8 > kCUs &&
                            n8 <= 3 * kCUs;
        auto groups_of = [&](int ng) { return static_cast<long long>(B) * ceil_div(k32, 8 * ng); };
        q.gate_groups = 0;
        for (int ng : {8, 4, 2})
            if (q.gate_groups == 0 && groups_of(ng) >= 150 && groups_of(ng) <= kCUs) q.gate_groups = ng;
        if (q.gate_groups == 0) {
            q.gate_groups = direct_ok ? 1 : 2;
            for (int ng : {8, 4, 2}) {
                if (groups_of(ng) >= kCUs) {
                    q.gate_groups = (groups_of(ng) <= kCUs * 3 / 2 && ng > 2) ? ng / 2 : ng;
                    break;
                }
            }
        }
        q.kcap = ceil_div(k32, std::max(kBfChunk, 8 * q.gate_groups)) * std::max(kBfChunk, 8 * q.gate_groups);
        q.gate_blocks = q.kcap / (8 * q.gate_groups);
        if (spread) {
            q.gate_groups = 1;
            q.kcap = k32;
            q.gate_spread = (ceil_div(k32 / 4, kCUs) + 1) / 2;  // 16-row tiles of the fullest workgroup
            q.gate_blocks = kCUs;
        }
        q.col_tile = kBfColTile;
        q.ncol = ceil_div(s->d, q.col_tile);
        const int nchunks = q.kcap / kBfChunk;
        // Chunks per slice: a multiple of 4 (1 to 8 per wave), the fewest that keep the slice count within the
        // target; lists longer than 8 chunks per wave at the target get more slices.
        const int s_target = std::max(1, ceil_div(kTargetDownGroups, q.ncol * B));
        const int cps = kBfWaves * std::min(kBfMaxChunksPerSlice / kBfWaves,
                                            std::max(1, ceil_div(ceil_div(nchunks, s_target), kBfWaves)));
        q.slice_units = cps;
        q.slices = ceil_div(nchunks, cps);
        // One sample's list in the spread range at d = 2048, or of 8 .. 192 chunks at d = 1024: gate/up and down
        // in one launch, the list's chunks cut into 8 slices, one per XCD (at most 3 chunks per wave of the down
        // phase, at most 6 quads per workgroup of the gate/up phase).  It pays where it removes launches: at
        // d = 2048 it replaces prologue (or epilogue-emitted input), gate/up, split down and epilogue by two
        // launches, in a stack too; at d = 1024 only for a single layer on given lists (prologue, gate/up and
        // fused down become two launches; a stack's layer is already gate/up + fused down, and a call that
        // compacts its mask does so in the prologue's launch).  Measured on one box: config 2 14.3 -> 13.7 us
        // per layer, its masked call 15.3 -> 16.5; a d = 1024 stack (config 3) 12.55 -> 14.7 and config 4 at
        // 10 % 17.0 -> 18.2 with it, so those keep the other kernels.  The workspace holds the buffers and the
        // partials of either plan, so its size does not depend on the device or the call; the launch form needs
        // 256 compute units (all 256 workgroups resident, 32 per XCD).
        const int cps8 = ceil_div(nchunks, 8);
        const bool xcd_d = s->d == 8 * 256 || s->d == 4 * 256;
        xcd_shape = RM_LAYER_XCD && B == 1 && T <= kBfTokBlock && cps8 <= 3 * 8 && nchunks >= 8 &&
                    ((spread && s->d == 8 * 256) || s->d == 4 * 256);
        // The buffers are reserved for every such d and T, whatever B and max_count, so that the workspace size
        // stays monotone in them (a workspace sized for more samples or a longer list serves this call).
        xcd_room = RM_LAYER_XCD && T <= kBfTokBlock && xcd_d;
        if (xcd_shape) part_slices = std::max(q.slices, ceil_div(nchunks, cps8));
        // Short lists (up to kDfMaxChunks chunks): one workgroup per (column tile, token tile) can sum the whole
        // list.  One sample: 16-token tiles.  Several samples: one 64-token tile, so each sample's listed rows of
        // a column tile are read once (16 samples of 51 tokens, d = 1024: down 17.8 -> 14.8 us against two 32-token tiles).
        q.dn_cpw = ceil_div(nchunks, kDfWaves);
        q.df_nt = B == 1 ? 1 : 4;
        q.fused_down = nchunks <= kDfMaxChunks;
        if (xcd_shape && (s->d == 8 * 256 || form == 0) && device_has_256_cus()) {  // the one-launch form
            q.xcd_layer = true;
            q.fused_down = false;
            q.slice_units = cps8;
            q.slices = ceil_div(nchunks, cps8);
            // A separate gate/up launch on this plan (an anchor's capture of h_a) runs the spread kernel: the
            // same per-neuron arithmetic and chunk order as the one-launch form's gate/up phase, so a delta step
            // at the anchor's own input finds h - h_a = 0 exactly.
            q.gate_groups = 1;
            q.gate_blocks = kCUs;
            q.gate_spread = (ceil_div(q.kcap / 4, kCUs) + 1) / 2;
        }
        q.ntt = ceil_div(T, 16 * q.df_nt);
        // One sample's tiles are 32 columns wide (two per lane), so that the 16-token tiles of a short prompt
        // still give the chip a workgroup per compute unit or more; with several samples, 64 columns.
        q.df_cw = B == 1 ? 2 : 4;
        q.df_ncol = ceil_div(s->d, 16 * q.df_cw);
        xn_elem = 2;
        h_elem = 2;
    } else {
        q.tpad = ceil_div(T, kF32TokBlock) * kF32TokBlock;
        q.kcap = ceil_div(kmax, kF32NeurPerBlk) * kF32NeurPerBlk;
        q.gate_blocks = q.kcap / kF32NeurPerBlk;
        q.col_tile = kF32ColTile;
        q.ncol = ceil_div(s->d, kF32ColTile);
        const long long work = static_cast<long long>(kmax) * q.ncol * B;
        const int su =
            static_cast<int>(std::max<long long>(kF32SliceNeur, (work + kTargetDownGroups - 1) / kTargetDownGroups));
        q.slice_units = su;
        q.slices = ceil_div(kmax, su);
        xn_elem = 4;
        h_elem = 4;
    }
    if (q.slices > 65535 || static_cast<long long>(q.gate_blocks) * B > 0x7fffffffLL ||
        static_cast<long long>(q.ncol) * q.slices * B > 0x7fffffffLL ||
        static_cast<long long>(q.ncol) * ceil_div(T, 16) * B > 0x7fffffffLL ||
        static_cast<long long>(q.df_ncol) * q.ntt * B > 0x7fffffffLL)
        return fail(RM_ERR_SHAPE, "launch grid too large");
    if (static_cast<long long>(B) * T * ceil_div(s->d, kRowBlock) > 0x7fffffffLL)
        return fail(RM_ERR_SHAPE, "B=%d x T=%d rows are too many for one launch", B, T);
    size_t off = 0;
    q.off_xn = off;
    off = align_up(off + static_cast<size_t>(B) * T * s->d * xn_elem, 256);
    q.off_h = off;
    off = align_up(off + static_cast<size_t>(B) * q.tpad * q.kcap * h_elem, 256);
    q.off_part = off;
    off = align_up(off + static_cast<size_t>(B) * std::max(q.slices, part_slices) * static_cast<size_t>(T) * s->d * 4,
                   256);
    q.off_ssq = off;
    off = align_up(off + static_cast<size_t>(B) * T * ssq_stride(s->d) * sizeof(float), 256);
    q.off_ident = off;
    off = align_up(off + static_cast<size_t>(B) * s->d_ff * sizeof(int32_t), 256);
    q.off_ident_count = off;
    off = align_up(off + static_cast<size_t>(B) * sizeof(int32_t), 256);
    q.off_xn8 = off;
    if (xcd_room) off = align_up(off + static_cast<size_t>(8) * T * s->d * 2, 256);
    q.off_ssq8 = off;
    if (xcd_room) off = align_up(off + static_cast<size_t>(8) * T * ssq_stride(s->d) * sizeof(float), 256);
    q.off_sync = off;
    if (xcd_room) off = align_up(off + kXcdFlagBytes + kXcdCtrBytes, 256);
    q.total = off;
    *p = q;
    return RM_OK;
}

void profile_take(int kernel, hipEvent_t *begin, hipEvent_t *end) {
    *begin = g_profile[kernel].begin;
    *end = g_profile[kernel].end;
    g_profile[kernel] = ProfileSlot{};
}

}  // namespace rm

// ---------------------------------------------------------------------------------------------------------
// Exported C ABI
// ---------------------------------------------------------------------------------------------------------

RM_EXPORT rm_status rm_mask_compact(const uint8_t *mask, int32_t n_masks, int32_t d_ff, int32_t *idx, int32_t *count,
                                    void *stream) {
    if (!mask || !idx || !count) return fail(RM_ERR_INVALID_ARG, "mask, idx or count is NULL");
    if (n_masks <= 0 || d_ff <= 0)
        return fail(RM_ERR_INVALID_ARG, "n_masks=%d and d_ff=%d must be positive", n_masks, d_ff);
    if (!aligned(idx, 4) || !aligned(count, 4)) return fail(RM_ERR_ALIGN, "idx and count must be 4-byte aligned");
    if (static_cast<long long>(n_masks) * ((d_ff + 1023) / 1024) > 0x7fffffffLL)
        return fail(RM_ERR_SHAPE, "n_masks=%d x d_ff=%d is too large for one launch", n_masks, d_ff);
    const size_t mbytes = static_cast<size_t>(n_masks) * d_ff;
    if (ranges_overlap(mask, mbytes, idx, mbytes * 4) || ranges_overlap(mask, mbytes, count, n_masks * 4u) ||
        ranges_overlap(idx, mbytes * 4, count, n_masks * 4u))
        return fail(RM_ERR_INVALID_ARG, "mask, idx and count must not overlap");
    const hipError_t e = rm::launch_mask_compact(mask, n_masks, d_ff, idx, count, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "mask compaction launch");
    return ok();
}

RM_EXPORT rm_status rm_workspace_size(const rm_ffn_shape *s, int32_t B, int32_t T, int32_t max_count, size_t *bytes) {
    if (!bytes) return fail(RM_ERR_INVALID_ARG, "bytes is NULL");
    rm_status st = check_shape(s);
    if (st != RM_OK) return st;
    if (B <= 0 || T <= 0) return fail(RM_ERR_INVALID_ARG, "B=%d and T=%d must be positive", B, T);
    if (max_count < 0 || max_count > s->d_ff)
        return fail(RM_ERR_SHAPE, "max_count=%d outside [0, d_ff=%d]", max_count, s->d_ff);
    rm::Plan p;
    st = rm::make_plan(s, B, T, max_count, &p);
    if (st != RM_OK) return st;
    *bytes = p.total;
    return ok();
}

RM_EXPORT rm_status rm_sparse_ffn_layer(const rm_ffn_shape *s, const rm_ffn_layer_weights *w, int32_t B, int32_t T,
                                        const float *x, float *y, const int32_t *idx, const int32_t *count,
                                        int32_t max_count, void *ws, size_t ws_bytes, void *stream) {
    rm::Plan p;
    rm_status st = check_call(s, B, T, x, y, idx, count, true, max_count, ws, ws_bytes, &p);
    if (st != RM_OK) return st;
    st = check_layer(w, 0);
    if (st != RM_OK) return st;
    st = check_gates(w, 1, B, T, s->d, y);
    if (st != RM_OK) return st;
    st = check_lists(s, 1, B, T, y, idx, count, ws, p.total);
    if (st != RM_OK) return st;
    st = run_layers(p, w, 1, x, y, idx, count, 0, 0, ws, static_cast<hipStream_t>(stream));
    return st == RM_OK ? ok() : st;
}

RM_EXPORT rm_status rm_sparse_ffn_layer_noalloc(const rm_ffn_shape *s, const rm_ffn_layer_weights *w, int32_t B,
                                                int32_t T, const float *x, float *y, const int32_t *idx,
                                                const int32_t *count, int32_t max_count, void *stream) {
    // The scratch the call needs is known from the shape alone: a call that needs more than the array holds
    // fails here, before anything touches the device.
    rm_status st = check_shape(s);
    if (st != RM_OK) return st;
    if (B <= 0 || T <= 0) return fail(RM_ERR_INVALID_ARG, "B=%d and T=%d must be positive", B, T);
    if (max_count < 0 || max_count > s->d_ff)
        return fail(RM_ERR_SHAPE, "max_count=%d outside [0, d_ff=%d]", max_count, s->d_ff);
    rm::Plan p;
    st = rm::make_plan(s, B, T, max_count, &p);
    if (st != RM_OK) return st;
    if (p.total > RM_NOALLOC_SCRATCH_BYTES)
        return fail(RM_ERR_WORKSPACE,
                    "this call needs %zu bytes of scratch; rm_sparse_ffn_layer_noalloc holds %zu (use "
                    "rm_sparse_ffn_layer with a workspace)",
                    p.total, static_cast<size_t>(RM_NOALLOC_SCRATCH_BYTES));
    void *ws = nullptr;
    st = noalloc_scratch(static_cast<hipStream_t>(stream), &ws);
    if (st != RM_OK) return st;
    // The same validation and kernels as the workspace form; the layer path needs no cleared scratch.
    return rm_sparse_ffn_layer(s, w, B, T, x, y, idx, count, max_count, ws, RM_NOALLOC_SCRATCH_BYTES, stream);
}

RM_EXPORT rm_status rm_sparse_ffn_stack(const rm_ffn_shape *s, const rm_ffn_layer_weights *w, int32_t L, int32_t B,
                                        int32_t T, const float *x, float *y, const int32_t *idx,
                                        const int32_t *count, int32_t max_count, void *ws, size_t ws_bytes,
                                        void *stream) {
    if (L <= 0) return fail(RM_ERR_INVALID_ARG, "L=%d must be positive", L);
    if (!w) return fail(RM_ERR_INVALID_ARG, "weights pointer is NULL");
    rm::Plan p;
    rm_status st = check_call(s, B, T, x, y, idx, count, true, max_count, ws, ws_bytes, &p,
                              rm::kFormStack | rm::kFormMask);
    if (st != RM_OK) return st;
    for (int l = 0; l < L; ++l) {
        st = check_layer(&w[l], l);
        if (st != RM_OK) return st;
    }
    st = check_gates(w, L, B, T, s->d, y);
    if (st != RM_OK) return st;
    st = check_lists(s, L, B, T, y, idx, count, ws, p.total);
    if (st != RM_OK) return st;
    st = run_layers(p, w, L, x, y, idx, count, static_cast<size_t>(B) * s->d_ff, B, ws,
                    static_cast<hipStream_t>(stream));
    return st == RM_OK ? ok() : st;
}

// Checks of the masks of a call that compacts them (n_masks = L * B masks of d_ff bytes into idx / count).
static rm_status check_masks(const rm_ffn_shape *s, int n_masks, int B, int T, const uint8_t *mask, const int32_t *idx,
                      const int32_t *count, const float *x, const float *y, const void *ws, size_t ws_bytes) {
    if (!mask) return fail(RM_ERR_INVALID_ARG, "mask is NULL");
    const int nseg = ceil_div(s->d_ff, 1024);
    const long long units = static_cast<long long>(B) * T * ceil_div(s->d, rm::kRowBlock);
    if (static_cast<long long>(n_masks) * nseg + (units + 3) / 4 > 0x7fffffffLL)
        return fail(RM_ERR_SHAPE, "%d masks of d_ff=%d and B x T = %d x %d rows are too many for one launch",
                    n_masks, s->d_ff, B, T);
    const size_t mbytes = static_cast<size_t>(n_masks) * s->d_ff;
    const size_t act = static_cast<size_t>(B) * T * s->d * sizeof(float);
    const void *outs[2] = {idx, count};
    const size_t out_bytes[2] = {mbytes * 4, static_cast<size_t>(n_masks) * 4};
    for (int i = 0; i < 2; ++i)
        if (ranges_overlap(outs[i], out_bytes[i], mask, mbytes) || ranges_overlap(outs[i], out_bytes[i], x, act) ||
            ranges_overlap(outs[i], out_bytes[i], y, act) || ranges_overlap(outs[i], out_bytes[i], ws, ws_bytes))
            return fail(RM_ERR_INVALID_ARG, "idx and count must not overlap the masks, x, y or the workspace");
    if (ranges_overlap(idx, out_bytes[0], count, out_bytes[1]))
        return fail(RM_ERR_INVALID_ARG, "idx and count must not overlap");
    return RM_OK;
}

RM_EXPORT rm_status rm_masked_ffn_layer(const rm_ffn_shape *s, const rm_ffn_layer_weights *w, int32_t B, int32_t T,
                                        const float *x, float *y, const uint8_t *mask, int32_t *idx, int32_t *count,
                                        int32_t max_count, void *ws, size_t ws_bytes, void *stream) {
    rm::Plan p;
    rm_status st = check_call(s, B, T, x, y, idx, count, true, max_count, ws, ws_bytes, &p, rm::kFormMask);
    if (st != RM_OK) return st;
    st = check_layer(w, 0);
    if (st != RM_OK) return st;
    st = check_masks(s, B, B, T, mask, idx, count, x, y, ws, ws_bytes);
    if (st != RM_OK) return st;
    st = check_gates(w, 1, B, T, s->d, y);
    if (st != RM_OK) return st;
    st = run_layers(p, w, 1, x, y, idx, count, 0, 0, ws, static_cast<hipStream_t>(stream), AnchorTerms{}, mask, B);
    return st == RM_OK ? ok() : st;
}

RM_EXPORT rm_status rm_masked_ffn_stack(const rm_ffn_shape *s, const rm_ffn_layer_weights *w, int32_t L, int32_t B,
                                        int32_t T, const float *x, float *y, const uint8_t *mask, int32_t *idx,
                                        int32_t *count, int32_t max_count, void *ws, size_t ws_bytes, void *stream) {
    if (L <= 0) return fail(RM_ERR_INVALID_ARG, "L=%d must be positive", L);
    if (!w) return fail(RM_ERR_INVALID_ARG, "weights pointer is NULL");
    rm::Plan p;
    rm_status st = check_call(s, B, T, x, y, idx, count, true, max_count, ws, ws_bytes, &p,
                              rm::kFormStack | rm::kFormMask);
    if (st != RM_OK) return st;
    for (int l = 0; l < L; ++l) {
        st = check_layer(&w[l], l);
        if (st != RM_OK) return st;
    }
    if (static_cast<long long>(L) * B > 0x7fffffffLL) return fail(RM_ERR_SHAPE, "L x B is too large");
    st = check_masks(s, L * B, B, T, mask, idx, count, x, y, ws, ws_bytes);
    if (st != RM_OK) return st;
    st = check_gates(w, L, B, T, s->d, y);
    if (st != RM_OK) return st;
    st = run_layers(p, w, L, x, y, idx, count, static_cast<size_t>(B) * s->d_ff, B, ws,
                    static_cast<hipStream_t>(stream), AnchorTerms{}, mask, L * B);
    return st == RM_OK ? ok() : st;
}

RM_EXPORT rm_status rm_dense_ffn_ref(const rm_ffn_shape *s, const rm_ffn_layer_weights *w, int32_t B, int32_t T,
                                     const float *x, float *y, void *ws, size_t ws_bytes, void *stream) {
    rm::Plan p;
    rm_status st = check_call(s, B, T, x, y, nullptr, nullptr, false, 0, ws, ws_bytes, &p);
    if (st != RM_OK) return st;
    st = check_layer(w, 0);
    if (st != RM_OK) return st;
    st = check_gates(w, 1, B, T, s->d, y);
    if (st != RM_OK) return st;
    const hipStream_t hs = static_cast<hipStream_t>(stream);
    const hipError_t e = rm::launch_identity_lists(p, ws, hs);
    if (e != hipSuccess) return hip_fail(e, "identity list launch");
    char *base = static_cast<char *>(ws);
    st = run_layers(p, w, 1, x, y, reinterpret_cast<const int32_t *>(base + p.off_ident),
                    reinterpret_cast<const int32_t *>(base + p.off_ident_count), 0, 0, ws, hs);
    return st == RM_OK ? ok() : st;
}

RM_EXPORT rm_status rm_anchor_ffn_stack(const rm_ffn_shape *s, const rm_ffn_layer_weights *w, int32_t L, int32_t B,
                                        int32_t T, const float *x, float *y, const int32_t *idx,
                                        const int32_t *count, int32_t max_count, float *y_anchor, float *h_anchor,
                                        void *ws, size_t ws_bytes, void *stream) {
    rm::Plan p, q;
    // the dense layers
    rm_status st = check_call(s, B, T, x, y, nullptr, nullptr, false, 0, ws, ws_bytes, &p, rm::kFormStack);
    if (st != RM_OK) return st;
    // The group's lists: their plan sizes the capture launch, which uses only the dense layout's regions (its
    // own plan may ask for more, e.g. the one-launch layer form's buffers), so the dense size is what counts.
    st = check_call(s, B, T, x, y, idx, count, true, max_count, ws, SIZE_MAX, &q, rm::kFormStack);
    if (st != RM_OK) return st;
    st = check_anchor_buffers(s, w, L, B, T, x, y, max_count, y_anchor, h_anchor, ws, ws_bytes);
    if (st != RM_OK) return st;
    st = check_lists(s, L, B, T, y, idx, count, ws, p.total);
    if (st != RM_OK) return st;
    // The capture reads the dense layers' FFN input and sums of squares from the dense workspace layout (with the
    // one-launch layer form, XCD 0's copies, which that launch completes and which have the same layout for one
    // sample); it writes nothing else there.
    q.off_xn = p.xcd_layer ? p.off_xn8 : p.off_xn;
    q.off_ssq = p.xcd_layer ? p.off_ssq8 : p.off_ssq;
    q.off_h = p.off_h;  // not written by a capture
    AnchorTerms at;
    at.ya_out = y_anchor;
    at.ha_out = max_count > 0 ? h_anchor : nullptr;  // nothing to keep from empty lists
    at.cap_idx = idx;
    at.cap_count = count;
    at.cap_plan = &q;
    at.h_stride = static_cast<size_t>(B) * max_count * T;
    const hipStream_t hs = static_cast<hipStream_t>(stream);
    const hipError_t e = rm::launch_identity_lists(p, ws, hs);
    if (e != hipSuccess) return hip_fail(e, "identity list launch");
    char *base = static_cast<char *>(ws);
    st = run_layers(p, w, L, x, y, reinterpret_cast<const int32_t *>(base + p.off_ident),
                    reinterpret_cast<const int32_t *>(base + p.off_ident_count), 0, 0, ws, hs, at);
    return st == RM_OK ? ok() : st;
}

RM_EXPORT rm_status rm_delta_ffn_stack(const rm_ffn_shape *s, const rm_ffn_layer_weights *w, int32_t L, int32_t B,
                                       int32_t T, const float *x, float *y, const int32_t *idx, const int32_t *count,
                                       int32_t max_count, const float *y_anchor, const float *h_anchor, void *ws,
                                       size_t ws_bytes, void *stream) {
    rm::Plan p;
    rm_status st = check_call(s, B, T, x, y, idx, count, true, max_count, ws, ws_bytes, &p, rm::kFormStack);
    if (st != RM_OK) return st;
    st = check_anchor_buffers(s, w, L, B, T, x, y, max_count, y_anchor, h_anchor, ws, ws_bytes);
    if (st != RM_OK) return st;
    AnchorTerms at;
    at.ya_in = y_anchor;
    at.ha_in = max_count > 0 ? h_anchor : nullptr;
    at.h_stride = static_cast<size_t>(B) * max_count * T;
    st = check_lists(s, L, B, T, y, idx, count, ws, p.total);
    if (st != RM_OK) return st;
    st = run_layers(p, w, L, x, y, idx, count, static_cast<size_t>(B) * s->d_ff, B, ws,
                    static_cast<hipStream_t>(stream), at);
    return st == RM_OK ? ok() : st;
}

RM_EXPORT rm_status rm_gather_stack_rows(const rm_ffn_shape *s, const rm_ffn_layer_weights *w, int32_t L,
                                         const int32_t *idx, const int32_t *count, int32_t max_count, void *out,
                                         void *stream) {
    rm_status st = check_shape(s);
    if (st != RM_OK) return st;
    if (L <= 0) return fail(RM_ERR_INVALID_ARG, "L=%d must be positive", L);
    if (!w) return fail(RM_ERR_INVALID_ARG, "weights pointer is NULL");
    for (int l = 0; l < L; ++l) {
        st = check_layer(&w[l], l);
        if (st != RM_OK) return st;
    }
    if (!idx || !count || !out) return fail(RM_ERR_INVALID_ARG, "idx, count or out is NULL");
    if (!aligned(idx, 4) || !aligned(count, 4) || !aligned(out, 16))
        return fail(RM_ERR_ALIGN, "idx and count must be 4-byte and out 16-byte aligned");
    if (max_count <= 0 || max_count > s->d_ff)
        return fail(RM_ERR_SHAPE, "max_count=%d outside [1, d_ff=%d]", max_count, s->d_ff);
    const size_t eb = s->wdtype == RM_BF16 ? 2 : 4;
    const size_t out_bytes = static_cast<size_t>(L) * 3 * max_count * s->d * eb;
    const size_t wbytes = static_cast<size_t>(s->d_ff) * s->d * eb;
    for (int l = 0; l < L; ++l)
        if (ranges_overlap(out, out_bytes, w[l].w_gate, wbytes) || ranges_overlap(out, out_bytes, w[l].w_up, wbytes) ||
            ranges_overlap(out, out_bytes, w[l].w_down, wbytes))
            return fail(RM_ERR_INVALID_ARG, "out overlaps layer %d's weights", l);
    if (ranges_overlap(out, out_bytes, idx, static_cast<size_t>(L) * s->d_ff * 4) ||
        ranges_overlap(out, out_bytes, count, static_cast<size_t>(L) * 4))
        return fail(RM_ERR_INVALID_ARG, "out overlaps idx or count");
    const hipError_t e = rm::launch_gather_rows(w, idx, count, s->d_ff, s->d, s->wdtype, max_count, L, out,
                                                static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "row gather launch");
    return ok();
}

RM_EXPORT rm_status rm_context_select(const float *x, const float *x_ref, int32_t n_tok, int32_t d, int32_t v0,
                                      int32_t P, int32_t k, float *drift, int32_t *rows, int32_t *count,
                                      void *stream) {
    if (!x || !x_ref || !rows || !count) return fail(RM_ERR_INVALID_ARG, "x, x_ref, rows or count is NULL");
    if (n_tok <= 0 || d <= 0) return fail(RM_ERR_INVALID_ARG, "n_tok=%d and d=%d must be positive", n_tok, d);
    if (n_tok > rm_sel::kSelThreads * rm_sel::kSelPerThread)
        return fail(RM_ERR_SHAPE, "n_tok=%d exceeds %d", n_tok, rm_sel::kSelThreads * rm_sel::kSelPerThread);
    if (v0 < 0 || P < 0 || static_cast<long long>(v0) + P > n_tok)
        return fail(RM_ERR_SHAPE, "visual rows [%d, %d + %d) outside [0, n_tok=%d)", v0, v0, P, n_tok);
    if (k < 0 || k > P) return fail(RM_ERR_SHAPE, "k=%d outside [0, P=%d]", k, P);
    if (P > 0 && !drift) return fail(RM_ERR_INVALID_ARG, "drift is NULL");
    if (!aligned(x, 4) || !aligned(x_ref, 4) || !aligned(rows, 4) || !aligned(count, 4) ||
        (drift && !aligned(drift, 4)))
        return fail(RM_ERR_ALIGN, "pointers must be 4-byte aligned");
    const size_t xb = static_cast<size_t>(n_tok) * d * 4;
    const void *outs[3] = {drift, rows, count};
    const size_t ob[3] = {static_cast<size_t>(P) * 4, static_cast<size_t>(n_tok) * 4, 4};
    for (int i = 0; i < 3; ++i) {
        if (!outs[i]) continue;
        if (ranges_overlap(outs[i], ob[i], x, xb) || ranges_overlap(outs[i], ob[i], x_ref, xb))
            return fail(RM_ERR_INVALID_ARG, "drift, rows and count must not overlap x or x_ref");
        for (int j = i + 1; j < 3; ++j)
            if (outs[j] && ranges_overlap(outs[i], ob[i], outs[j], ob[j]))
                return fail(RM_ERR_INVALID_ARG, "drift, rows and count must not overlap each other");
    }
    const hipError_t e = rm::launch_context_select(x, x_ref, n_tok, d, v0, P, k, drift, rows, count,
                                                   static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "context selection launch");
    return ok();
}

static rm_status context_plan(const rm_ffn_shape *s, int n_tok, int max_rows, rm::ContextPlan *p) {
    rm_status st = check_shape(s);
    if (st != RM_OK) return st;
    if (s->wdtype != RM_BF16) return fail(RM_ERR_DTYPE, "the context FFN takes bf16 weights");
    if (s->d % 64 != 0 || s->d_ff % rm::kCtxGluBN != 0)
        return fail(RM_ERR_SHAPE, "d=%d must be a multiple of 64 and d_ff=%d of %d", s->d, s->d_ff, rm::kCtxGluBN);
    if (n_tok <= 0 || max_rows <= 0 || max_rows > n_tok)
        return fail(RM_ERR_SHAPE, "need 1 <= max_rows=%d <= n_tok=%d", max_rows, n_tok);
    rm::ContextPlan q;
    q.d = s->d;
    q.d_ff = s->d_ff;
    q.act = s->act;
    q.n_tok = n_tok;
    q.max_rows = max_rows;
    q.m_pad = ceil_div(max_rows, rm::kCtxBM) * rm::kCtxBM;
    q.down_bn = rm::ctx_down_bn(s->d);
    const long long tiles = static_cast<long long>(q.m_pad / rm::kCtxBM) * (s->d_ff / rm::kCtxGluBN);
    if (tiles > 0x7fffffffLL) return fail(RM_ERR_SHAPE, "launch grid too large");
    // The down GEMM splits K until it has about one workgroup per compute unit, keeping slices of at least 1024
    // along K (a multiple of the 64-wide K stage).
    const int out_tiles = (q.m_pad / rm::kCtxBM) * (s->d / q.down_bn);
    q.down_splits = 1;
    while (q.down_splits < 16 && out_tiles * q.down_splits < rm::kCtxDownTarget &&
           s->d_ff % (2 * q.down_splits * 64) == 0 && s->d_ff / (2 * q.down_splits) >= 1024)
        q.down_splits *= 2;
    q.off_a = 0;
    q.off_h = align_up(static_cast<size_t>(q.m_pad) * s->d * 2, 256);
    q.off_part = align_up(q.off_h + static_cast<size_t>(q.m_pad) * s->d_ff * 2, 256);
    const size_t part = q.down_splits > 1 ? static_cast<size_t>(q.down_splits) * q.m_pad * s->d * 4 : 0;
    q.total = align_up(q.off_part + part, 256);
    *p = q;
    return RM_OK;
}

RM_EXPORT rm_status rm_context_workspace_size(const rm_ffn_shape *s, int32_t n_tok, int32_t max_rows, size_t *bytes) {
    if (!bytes) return fail(RM_ERR_INVALID_ARG, "bytes is NULL");
    rm::ContextPlan p;
    const rm_status st = context_plan(s, n_tok, max_rows, &p);
    if (st != RM_OK) return st;
    *bytes = p.total;
    return ok();
}

static rm_status context_ffn(const rm_ffn_shape *s, const void *w_gate, const void *w_up, const void *w_down_t,
                             bool blocked, int32_t n_tok, const float *x, const int32_t *rows, const int32_t *count,
                             int32_t max_rows, float *y, void *ws, size_t ws_bytes, void *stream) {
    rm::ContextPlan p;
    rm_status st = context_plan(s, n_tok, max_rows, &p);
    if (st != RM_OK) return st;
    if (!w_gate || !w_up || !w_down_t || !x || !rows || !count || !y || !ws)
        return fail(RM_ERR_INVALID_ARG, "a pointer is NULL");
    if (!aligned(w_gate, 16) || !aligned(w_up, 16) || !aligned(w_down_t, 16) || !aligned(x, 16) ||
        !aligned(y, 4) || !aligned(rows, 4) || !aligned(count, 4) || !aligned(ws, 16))
        return fail(RM_ERR_ALIGN, "weights, x and the workspace must be 16-byte aligned, the rest 4-byte");
    if (ws_bytes < p.total)
        return fail(RM_ERR_WORKSPACE, "workspace of %zu bytes is smaller than the %zu required", ws_bytes, p.total);
    const size_t act_bytes = static_cast<size_t>(n_tok) * s->d * 4;
    if (ranges_overlap(x, act_bytes, y, act_bytes) || ranges_overlap(ws, p.total, x, act_bytes) ||
        ranges_overlap(ws, p.total, y, act_bytes))
        return fail(RM_ERR_INVALID_ARG, "x, y and the workspace must not overlap");
    // What the launches only read (the weights, the row list and its count) must not overlap what they write.
    const size_t mb = static_cast<size_t>(s->d) * s->d_ff * 2;
    const void *ins[5] = {w_gate, w_up, w_down_t, rows, count};
    const size_t inb[5] = {mb, mb, mb, static_cast<size_t>(max_rows) * 4, 4};
    for (int i = 0; i < 5; ++i)
        if (ranges_overlap(ins[i], inb[i], y, act_bytes) || ranges_overlap(ins[i], inb[i], ws, p.total))
            return fail(RM_ERR_INVALID_ARG, "the weights, rows and count must not overlap y or the workspace");
    const hipError_t e = rm::launch_context_ffn(p, w_gate, w_up, w_down_t, blocked, x, rows, count, y, ws,
                                                static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "context FFN launch");
    return ok();
}

RM_EXPORT rm_status rm_context_ffn(const rm_ffn_shape *s, const void *w_gate, const void *w_up, const void *w_down_t,
                                   int32_t n_tok, const float *x, const int32_t *rows, const int32_t *count,
                                   int32_t max_rows, float *y, void *ws, size_t ws_bytes, void *stream) {
    return context_ffn(s, w_gate, w_up, w_down_t, false, n_tok, x, rows, count, max_rows, y, ws, ws_bytes, stream);
}

static size_t context_matrix_bytes(const rm_ffn_shape *s) { return static_cast<size_t>(s->d) * s->d_ff * 2; }

RM_EXPORT rm_status rm_context_pack_size(const rm_ffn_shape *s, size_t *bytes) {
    if (!bytes) return fail(RM_ERR_INVALID_ARG, "bytes is NULL");
    rm::ContextPlan p;
    const rm_status st = context_plan(s, 1, 1, &p);
    if (st != RM_OK) return st;
    *bytes = 3 * context_matrix_bytes(s);
    return ok();
}

RM_EXPORT rm_status rm_context_pack(const rm_ffn_shape *s, const void *w_gate, const void *w_up, const void *w_down_t,
                                    void *packed, size_t packed_bytes, void *stream) {
    rm::ContextPlan p;
    const rm_status st = context_plan(s, 1, 1, &p);
    if (st != RM_OK) return st;
    if (!w_gate || !w_up || !w_down_t || !packed) return fail(RM_ERR_INVALID_ARG, "a pointer is NULL");
    if (!aligned(w_gate, 16) || !aligned(w_up, 16) || !aligned(w_down_t, 16) || !aligned(packed, 16))
        return fail(RM_ERR_ALIGN, "weights and the packed buffer must be 16-byte aligned");
    const size_t mb = context_matrix_bytes(s);
    if (packed_bytes < 3 * mb)
        return fail(RM_ERR_WORKSPACE, "packed buffer of %zu bytes is smaller than the %zu required", packed_bytes,
                    3 * mb);
    if (ranges_overlap(packed, 3 * mb, w_gate, mb) || ranges_overlap(packed, 3 * mb, w_up, mb) ||
        ranges_overlap(packed, 3 * mb, w_down_t, mb))
        return fail(RM_ERR_INVALID_ARG, "the packed buffer must not overlap the weights");
    const auto hs = static_cast<hipStream_t>(stream);
    char *out = static_cast<char *>(packed);
    hipError_t e = rm::launch_pack_blocked(w_gate, s->d_ff, s->d, out, hs);
    if (e == hipSuccess) e = rm::launch_pack_blocked(w_up, s->d_ff, s->d, out + mb, hs);
    if (e == hipSuccess) e = rm::launch_pack_blocked(w_down_t, s->d, s->d_ff, out + 2 * mb, hs);
    if (e != hipSuccess) return hip_fail(e, "context weight packing launch");
    return ok();
}

RM_EXPORT rm_status rm_context_ffn_packed(const rm_ffn_shape *s, const void *packed, int32_t n_tok, const float *x,
                                          const int32_t *rows, const int32_t *count, int32_t max_rows, float *y,
                                          void *ws, size_t ws_bytes, void *stream) {
    if (!packed) return fail(RM_ERR_INVALID_ARG, "packed is NULL");
    rm::ContextPlan p;
    const rm_status st = context_plan(s, n_tok, max_rows, &p);
    if (st != RM_OK) return st;
    const size_t mb = context_matrix_bytes(s);
    const char *w = static_cast<const char *>(packed);
    if (ranges_overlap(w, 3 * mb, y, static_cast<size_t>(n_tok) * s->d * 4) || ranges_overlap(w, 3 * mb, ws, ws_bytes))
        return fail(RM_ERR_INVALID_ARG, "the packed weights must not overlap y or the workspace");
    return context_ffn(s, w, w + mb, w + 2 * mb, true, n_tok, x, rows, count, max_rows, y, ws, ws_bytes, stream);
}

RM_EXPORT rm_status rm_neuron_norms(const void *w_down, int32_t d_ff, int32_t d, int32_t wdtype, float *norms,
                                    void *stream) {
    if (!w_down || !norms) return fail(RM_ERR_INVALID_ARG, "w_down or norms is NULL");
    if (d <= 0 || d_ff <= 0) return fail(RM_ERR_INVALID_ARG, "d=%d and d_ff=%d must be positive", d, d_ff);
    if (d % 32 != 0) return fail(RM_ERR_SHAPE, "d=%d must be a multiple of 32", d);
    if (wdtype != RM_F32 && wdtype != RM_BF16) return fail(RM_ERR_DTYPE, "unknown weight dtype %d", wdtype);
    if (!aligned(w_down, 16) || !aligned(norms, 4))
        return fail(RM_ERR_ALIGN, "w_down must be 16-byte and norms 4-byte aligned");
    const size_t wbytes = static_cast<size_t>(d_ff) * d * (wdtype == RM_BF16 ? 2 : 4);
    if (ranges_overlap(w_down, wbytes, norms, static_cast<size_t>(d_ff) * 4))
        return fail(RM_ERR_INVALID_ARG, "norms overlaps w_down");
    const hipError_t e = rm::launch_neuron_norms(w_down, d_ff, d, wdtype, norms, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "neuron norm launch");
    return ok();
}

RM_EXPORT rm_status rm_group_masks(const float *h, int32_t S, int32_t L, int32_t d_ff, int32_t T, const float *norms,
                                   int32_t K, float *scores, uint8_t *mask, void *stream) {
    if (!h || !norms || !scores || !mask) return fail(RM_ERR_INVALID_ARG, "h, norms, scores or mask is NULL");
    if (S <= 0 || L <= 0 || d_ff <= 0 || T <= 0)
        return fail(RM_ERR_INVALID_ARG, "S=%d, L=%d, d_ff=%d and T=%d must be positive", S, L, d_ff, T);
    if (d_ff > rm::kGroupMaxDff) return fail(RM_ERR_SHAPE, "d_ff=%d exceeds %d", d_ff, rm::kGroupMaxDff);
    if (K < 0 || K > d_ff) return fail(RM_ERR_SHAPE, "K=%d outside [0, d_ff=%d]", K, d_ff);
    if (static_cast<long long>(S) * L > 65535) return fail(RM_ERR_SHAPE, "S x L = %d x %d exceeds 65535", S, L);
    if (!aligned(h, 4) || !aligned(norms, 4) || !aligned(scores, 4))
        return fail(RM_ERR_ALIGN, "h, norms and scores must be 4-byte aligned");
    const size_t sl = static_cast<size_t>(S) * L;
    const size_t hb = sl * d_ff * T * 4, nb = static_cast<size_t>(L) * d_ff * 4, sb = sl * d_ff * 4;
    const size_t mb = static_cast<size_t>(L) * d_ff;
    if (ranges_overlap(scores, sb, h, hb) || ranges_overlap(scores, sb, norms, nb) ||
        ranges_overlap(scores, sb, mask, mb) || ranges_overlap(mask, mb, h, hb) || ranges_overlap(mask, mb, norms, nb))
        return fail(RM_ERR_INVALID_ARG, "scores and mask must not overlap each other, h or norms");
    const hipError_t e = rm::launch_group_masks(h, S, L, d_ff, T, norms, K, scores, mask,
                                                static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "group mask launch");
    return ok();
}

RM_EXPORT rm_status rm_profile_kernel_events(int32_t kernel, void *ev_begin, void *ev_end) {
    if (kernel < RM_KERNEL_GATEUP || kernel > RM_KERNEL_LAYER)
        return fail(RM_ERR_INVALID_ARG, "unknown kernel id %d", kernel);
    g_profile[kernel].begin = static_cast<hipEvent_t>(ev_begin);
    g_profile[kernel].end = static_cast<hipEvent_t>(ev_end);
    return ok();
}

RM_EXPORT rm_status rm_layer_kernels(const rm_ffn_shape *s, int32_t B, int32_t T, int32_t max_count,
                                     uint32_t *kernels) {
    if (!kernels) return fail(RM_ERR_INVALID_ARG, "kernels is NULL");
    size_t bytes = 0;
    const rm_status st = rm_workspace_size(s, B, T, max_count, &bytes);  // the same checks
    if (st != RM_OK) return st;
    rm::Plan p;
    rm::make_plan(s, B, T, max_count, &p);
    *kernels = p.xcd_layer ? (1u << RM_KERNEL_LAYER) : ((1u << RM_KERNEL_GATEUP) | (1u << RM_KERNEL_DOWN));
    return ok();
}

RM_EXPORT rm_status rm_stream_read(const void *buf, size_t bytes, int32_t workgroups, uint32_t *sink, void *stream) {
    if (!buf || !sink) return fail(RM_ERR_INVALID_ARG, "buf or sink is NULL");
    if (bytes == 0 || bytes % 16 != 0) return fail(RM_ERR_SHAPE, "bytes=%zu must be a positive multiple of 16", bytes);
    if (workgroups < 1 || workgroups > (1 << 20))
        return fail(RM_ERR_SHAPE, "workgroups=%d outside [1, %d]", workgroups, 1 << 20);
    if (!aligned(buf, 16) || !aligned(sink, 4)) return fail(RM_ERR_ALIGN, "buf must be 16-byte and sink 4-byte aligned");
    if (ranges_overlap(buf, bytes, sink, static_cast<size_t>(workgroups) * 512 * 4))
        return fail(RM_ERR_INVALID_ARG, "sink overlaps buf");
    const hipError_t e = rm::launch_stream_read(buf, bytes, workgroups, sink, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "stream read launch");
    return ok();
}

RM_EXPORT const char *rm_status_string(rm_status status) {
    switch (status) {
        case RM_OK: return "RM_OK";
        case RM_ERR_INVALID_ARG: return "RM_ERR_INVALID_ARG: invalid argument";
        case RM_ERR_SHAPE: return "RM_ERR_SHAPE: unsupported shape";
        case RM_ERR_DTYPE: return "RM_ERR_DTYPE: unsupported dtype";
        case RM_ERR_ALIGN: return "RM_ERR_ALIGN: misaligned pointer";
        case RM_ERR_WORKSPACE: return "RM_ERR_WORKSPACE: workspace too small";
        case RM_ERR_HIP: return "RM_ERR_HIP: HIP runtime error";
    }
    return "unknown rm_status";
}

RM_EXPORT const char *rm_last_error(void) { return g_last_error; }
