/*
 * rmuscle.h: C ABI of the Action Cache sparse-FFN hot path on one AMD Instinct MI355X (gfx950).
 *
 * The paper's Action Cache (section 4.1, "Group-Shared Neuron Masks" and "Anchors with Mask Recomputation")
 * keeps, per action-expert FFN layer, a mask of important intermediate neurons taken from a similar reference
 * execution.  The mask is shared by the consecutive denoising steps of a group, and at each such step only
 * the selected neurons' hidden activations h^M are computed and applied through their down-projection rows
 * (Eq. 4).  The core call is that update with a zero anchor, i.e. the masked SwiGLU FFN
 *
 *     y[b,t,:] = x[b,t,:] + sum_{i < count[b]} h[b,t,i] * w_down[idx[b][i], :]
 *     h[b,t,i] = act(<w_gate[idx[b][i]], xn[b,t]>) * <w_up[idx[b][i]], xn[b,t]>   (act: SiLU or GELU-tanh)
 *     xn       = norm_g ? x / sqrt(mean(x^2) + norm_eps) * norm_g : x
 *
 * where only the listed rows of w_gate / w_up / w_down are read.  Eq. 4 itself, with the group's dense
 * anchor, is the pair rm_anchor_ffn_stack (the anchor step) / rm_delta_ffn_stack (the other steps):
 *
 *     y[b,t,:] = x[b,t,:] + y_a[b,t,:] + sum_{i < count[b]} (h[b,t,i] - h_a[b,i,t]) * w_down[idx[b][i], :]
 *
 * with y_a the anchor's FFN output (before the residual) and h_a its activations of the listed neurons.  With an
 * output gate (rm_ffn_layer_weights.out_gate) the FFN part of each formula is multiplied by it before the
 * residual is added, and y_a is kept before the gate.
 *
 * Conventions shared by every call
 *   - Pointers are DEVICE pointers unless marked (host).  The caller owns every buffer and the stream; the
 *     library allocates nothing and never synchronizes.  Its only state is a thread-local error string, the
 *     events that rm_profile_kernel_events arms for the calling thread, a per-device record of the compute-unit
 *     count (asked once; with the RM_NO_LAYER_FORM environment variable, read once, it decides whether the
 *     one-launch layer form can run), and the noalloc entry point's per-device scratch array.
 *   - Every call is asynchronous on `stream` (a hipStream_t; NULL = the default stream).
 *   - Every argument is validated on the host before anything is enqueued; on error nothing is enqueued and
 *     the call returns a negative rm_status with a detail message in rm_last_error().
 *   - Index lists are multisets: a neuron listed twice contributes twice.  Lists made by rm_mask_compact hold
 *     no repeats.  An index outside [0, d_ff) is undefined behaviour (not checked on the device).
 *   - Activations are float32.  Weights are float32 (RM_F32) or bfloat16 (RM_BF16); accumulation is float32.
 *     On the bf16 path the FFN input xn and the activations h are rounded to bf16 before the matrix-core
 *     products.
 *   - The result is deterministic: no floating-point atomics; repeated calls give bitwise equal outputs.
 *   - The one-launch layer form (RM_KERNEL_LAYER; on a device with 256 compute units) needs all 256 of its
 *     workgroups resident at once: the 32 workgroups of each XCD wait for each other twice.  Work on other
 *     streams or processes that holds compute units while it runs delays it; a wait gives up after 200 ms,
 *     and then the affected outputs are NaN (the kernel always finishes).  Callers that share the GPU that
 *     way set the environment variable RM_NO_LAYER_FORM=1 before their first call: every call then takes
 *     the other kernels (same results up to the order of the float32 sums).
 */
#ifndef RMUSCLE_H
#define RMUSCLE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum rm_status {
    RM_OK = 0,
    RM_ERR_INVALID_ARG = -1, /* null pointer, non-positive size, bad enum value            */
    RM_ERR_SHAPE = -2,       /* d not a multiple of 32, max_count outside [0, d_ff], ...    */
    RM_ERR_DTYPE = -3,       /* unknown weight dtype                                        */
    RM_ERR_ALIGN = -4,       /* a pointer is not 16-byte aligned                            */
    RM_ERR_WORKSPACE = -5,   /* ws_bytes smaller than rm_workspace_size() asks for          */
    RM_ERR_HIP = -6          /* the HIP runtime refused a launch (see rm_last_error())      */
} rm_status;

typedef enum rm_dtype { RM_F32 = 0, RM_BF16 = 1 } rm_dtype;

/* Activation of the gated linear unit: h = act(<w_gate, xn>) * <w_up, xn>.  SiLU makes the FFN a SwiGLU, the
 * tanh form of GELU, 0.5 z (1 + tanh(sqrt(2/pi) (z + 0.044715 z^3))), a GeGLU (section 3.4 scores post-GeGLU
 * activations). */
typedef enum rm_act { RM_ACT_SILU = 0, RM_ACT_GELU_TANH = 1 } rm_act;

/* Shape of one FFN layer.  d: model width (multiple of 32).  d_ff: intermediate neurons (>= 1).
 * wdtype: an rm_dtype.  norm_eps: RMSNorm epsilon (1e-6 in the workloads); ignored without norm_g.
 * act: an rm_act. */
typedef struct rm_ffn_shape {
    int32_t d;
    int32_t d_ff;
    int32_t wdtype;
    float norm_eps;
    int32_t act;
} rm_ffn_shape;

/* Weights of one layer, all row-major [d_ff][d] in the dtype of rm_ffn_shape.wdtype.
 * Row n of every matrix belongs to intermediate neuron n:
 *   w_gate[n], w_up[n]: the gate and up projections (PyTorch nn.Linear weights of shape [d_ff][d]);
 *   w_down[n]: the neuron's down-projection row, i.e. the row-vector form W^down of Eq. 4 (the transpose of a
 *              PyTorch down_proj.weight of shape [d][d_ff]), so that a neuron's down weights are contiguous.
 * norm_g: float32 [d] RMSNorm gain applied to the FFN input, or NULL for no norm.
 * out_gate: float32 [B][d], the adaptive output gate of each sample for this layer and step (section 4.1: the
 *           FFN output goes through the model's adaptive gate before the residual addition), or NULL for none:
 *           y = x + out_gate[b] * FFN(x) elementwise over columns, for every token of sample b.
 * All pointers 16-byte aligned.  Read-only. */
typedef struct rm_ffn_layer_weights {
    const void *w_gate;
    const void *w_up;
    const void *w_down;
    const float *norm_g;
    const float *out_gate;
} rm_ffn_layer_weights;

/* Mask -> ascending active-neuron index list (section 4.1: a reference stores its selected neuron indices;
 * section 5: one mask per layer and group).
 *   mask:  uint8 [n_masks][d_ff], nonzero = active (a torch.bool tensor's storage qualifies).
 *   idx:   int32 [n_masks][d_ff] out.  Row m holds the active positions of mask m in ascending order in its
 *          first count[m] entries and -1 in the rest (the whole row is written).
 *   count: int32 [n_masks] out, the number of active neurons of each mask.
 * n_masks >= 1, d_ff >= 1.  idx and count must not overlap mask.  Errors: RM_ERR_INVALID_ARG for null
 * pointers or non-positive sizes, RM_ERR_ALIGN if idx or count is not 4-byte aligned. */
rm_status rm_mask_compact(const uint8_t *mask, int32_t n_masks, int32_t d_ff, int32_t *idx, int32_t *count,
                          void *stream);

/* Workspace bytes (written to *bytes, a host pointer) needed by the FFN calls (rm_sparse_ffn_*, rm_masked_ffn_*,
 * rm_dense_ffn_ref, rm_anchor_ffn_stack, rm_delta_ffn_stack) for B samples of T tokens with at most max_count
 * listed neurons per sample and layer (max_count = d_ff for the dense and anchor calls).  The workspace is
 * scratch owned by the caller: 256-byte aligned device memory, contents need not be initialized, reused by every
 * layer of a call, and it must not be used by two calls that may run at the same time. */
rm_status rm_workspace_size(const rm_ffn_shape *s, int32_t B, int32_t T, int32_t max_count, size_t *bytes);

/* One masked FFN layer with residual (Eq. 4 with a zero anchor; see the file comment).
 *   s, w:   host pointers to the shape and to the layer's weights.
 *   x:      float32 [B][T][d] input.   y: float32 [B][T][d] output; y == x (in place) is allowed, any other
 *           overlap is not.
 *   idx:    int32 [B][d_ff]: sample b's list in idx[b][0 .. count[b]-1] (the rm_mask_compact layout).
 *   count:  int32 [B], each in [0, max_count]; read on the device, so it may be produced by an earlier kernel.
 *   max_count: host-side upper bound of count[], in [0, d_ff]; sizes the launch and the workspace.
 *   ws, ws_bytes: workspace of at least rm_workspace_size(s, B, T, max_count) bytes.
 * The workspace must not overlap x or y, nor may idx or count overlap y or the workspace (RM_ERR_INVALID_ARG).
 * count[b] == 0 gives y[b] == x[b] bit for bit. */
rm_status rm_sparse_ffn_layer(const rm_ffn_shape *s, const rm_ffn_layer_weights *w, int32_t B, int32_t T,
                              const float *x, float *y, const int32_t *idx, const int32_t *count,
                              int32_t max_count, void *ws, size_t ws_bytes, void *stream);

/* Bytes of device scratch that rm_sparse_ffn_layer_noalloc holds per GPU (32 MiB). */
#define RM_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)

/* rm_sparse_ffn_layer without a workspace argument, for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation): the same computation, the same
 * kernels and the same results bit for bit, with the workspace taken from a device array of
 * RM_NOALLOC_SCRATCH_BYTES inside the library.  Arguments and errors as for rm_sparse_ffn_layer, minus ws and
 * ws_bytes, plus:
 *   - RM_ERR_WORKSPACE, before anything touches the device, when rm_workspace_size(s, B, T, max_count) exceeds
 *     RM_NOALLOC_SCRATCH_BYTES (every configuration of the action expert in this library fits: at most 15 MiB);
 *   - RM_ERR_INVALID_ARG when `stream` belongs to a device other than the current one.
 * The call allocates nothing.  Its first call on a device looks up that device's copy of the array (each GPU has
 * its own), which stays allocated until the process ends.  Every call on one GPU uses the same array and leaves
 * its contents behind; the layer needs none of it cleared.  Calls that may overlap on one GPU (several streams,
 * several threads) race on the array: the caller must order them. */
rm_status rm_sparse_ffn_layer_noalloc(const rm_ffn_shape *s, const rm_ffn_layer_weights *w, int32_t B, int32_t T,
                                      const float *x, float *y, const int32_t *idx, const int32_t *count,
                                      int32_t max_count, void *stream);

/* L masked FFN layers applied in order (the action expert's layer loop within one denoising step, sections
 * 2.4 and 4.1): layer l reads layer l-1's output.  w is a host array of L weight structs.  idx is
 * int32 [L][B][d_ff] and count int32 [L][B] (one rm_mask_compact call over L*B masks fills both); max_count
 * bounds every count.  x, y, ws as for rm_sparse_ffn_layer (y == x allowed).  L >= 1. */
rm_status rm_sparse_ffn_stack(const rm_ffn_shape *s, const rm_ffn_layer_weights *w, int32_t L, int32_t B,
                              int32_t T, const float *x, float *y, const int32_t *idx, const int32_t *count,
                              int32_t max_count, void *ws, size_t ws_bytes, void *stream);

/* rm_mask_compact followed by rm_sparse_ffn_layer, for a step that takes a freshly retrieved mask (section 4.1:
 * the reference's mask is compacted into its index list; section 5: one mask per layer and group).  The
 * compaction runs in the launch of the layer's first kernel (the two are independent), or ahead of the
 * one-launch layer kernel at d = 2048.  The result is rm_sparse_ffn_layer's on the written lists bit for bit,
 * except for one sample at d = 1024, where rm_sparse_ffn_layer runs the one-launch layer kernel and this call
 * the prologue (with the compaction), gate/up and fused down kernels: there the two agree up to the order of
 * the float32 sums.
 *   mask:  uint8 [B][d_ff], nonzero = active.
 *   idx, count: out, int32 [B][d_ff] and [B], written exactly as rm_mask_compact writes them, so that the
 *          group's later steps can call rm_sparse_ffn_layer with them.
 *   max_count: in [0, d_ff], at least the number of active neurons of every mask (d_ff is always safe); a mask
 *          with more active neurons than max_count contributes only its first max_count neurons.
 * Other arguments, the workspace size and the errors as for rm_sparse_ffn_layer; idx and count must not
 * overlap the masks, x, y, the workspace or each other. */
rm_status rm_masked_ffn_layer(const rm_ffn_shape *s, const rm_ffn_layer_weights *w, int32_t B, int32_t T,
                              const float *x, float *y, const uint8_t *mask, int32_t *idx, int32_t *count,
                              int32_t max_count, void *ws, size_t ws_bytes, void *stream);

/* rm_mask_compact of L * B masks followed by rm_sparse_ffn_stack (bit for bit), the compaction in the launch
 * of the stack's first kernel (ahead of the one-launch layer kernel at d = 2048).  mask: uint8 [L][B][d_ff];
 * idx int32 [L][B][d_ff] and count int32 [L][B] out.  Otherwise as rm_masked_ffn_layer and
 * rm_sparse_ffn_stack. */
rm_status rm_masked_ffn_stack(const rm_ffn_shape *s, const rm_ffn_layer_weights *w, int32_t L, int32_t B,
                              int32_t T, const float *x, float *y, const uint8_t *mask, int32_t *idx,
                              int32_t *count, int32_t max_count, void *ws, size_t ws_bytes, void *stream);

/* The dense FFN layer with residual: every neuron active (the anchor step of a group, section 4.1, and the
 * dense fallback of section 5).  Same arguments as rm_sparse_ffn_layer without the lists; the workspace is
 * sized with max_count = d_ff. */
rm_status rm_dense_ffn_ref(const rm_ffn_shape *s, const rm_ffn_layer_weights *w, int32_t B, int32_t T,
                           const float *x, float *y, void *ws, size_t ws_bytes, void *stream);

/* The anchor step of a group with Eq. 4 (section 4.1, "Anchors with Mask Recomputation"): L dense FFN layers
 * applied in order, as rm_dense_ffn_ref for each layer (norm, residual, layer l reading layer l-1's output),
 * which also keep what the group's later steps reuse:
 *   y_anchor: float32 [L][B][T][d] out, each layer's dense FFN output y_a before the residual (its y minus
 *             its input, as summed before the residual add);
 *   h_anchor: float32 [L][B][max_count][T] out, h_anchor[l][b][i][t] = the dense activation h of neuron
 *             idx[l][b][i] at token t, for i < count[l][b] (later entries are not written); may be NULL
 *             when max_count is 0.
 *   idx, count, max_count: the group's lists, as for rm_sparse_ffn_stack ([L][B][d_ff] and [L][B]).
 * x, y, w as for rm_sparse_ffn_stack.  The workspace is sized with max_count = d_ff
 * (rm_workspace_size(s, B, T, s->d_ff, ...)).  The h values kept are computed by the same kernel, with the
 * same launch geometry and summation order, as the h of rm_delta_ffn_stack with the same lists, so a delta
 * step at the anchor's own input reproduces the anchor's y bit for bit.  y_anchor and h_anchor must not
 * overlap each other, x, y or the workspace.  Errors as for rm_sparse_ffn_stack; RM_ERR_ALIGN if y_anchor is
 * not 16-byte or h_anchor not 4-byte aligned. */
rm_status rm_anchor_ffn_stack(const rm_ffn_shape *s, const rm_ffn_layer_weights *w, int32_t L, int32_t B,
                              int32_t T, const float *x, float *y, const int32_t *idx, const int32_t *count,
                              int32_t max_count, float *y_anchor, float *h_anchor, void *ws, size_t ws_bytes,
                              void *stream);

/* A non-anchor step of the group with Eq. 4 (section 4.1): L layers, layer l computing
 *     y = x + (y_anchor[l] + sum_{i < count[l][b]} (h - h_anchor[l][b][i]) * w_down[idx[l][b][i]])
 * with h the current activations of the listed neurons.  The difference h - h_anchor is formed in float32 and
 * then rounded once (to bf16 on the bf16 path) for the down projection.  y_anchor and h_anchor are what
 * rm_anchor_ffn_stack wrote for the same lists (read only).  With an empty list the layer returns
 * x + y_anchor; with the anchor taken at the same input the layer returns the anchor's y.  Arguments and
 * errors as for rm_sparse_ffn_stack, plus those of rm_anchor_ffn_stack for y_anchor and h_anchor; the
 * workspace is sized with the call's max_count. */
rm_status rm_delta_ffn_stack(const rm_ffn_shape *s, const rm_ffn_layer_weights *w, int32_t L, int32_t B, int32_t T,
                             const float *x, float *y, const int32_t *idx, const int32_t *count, int32_t max_count,
                             const float *y_anchor, const float *h_anchor, void *ws, size_t ws_bytes, void *stream);

/* Compact copies of a group's selected weight rows (section 4.1, last paragraph; section 5, "Overlapping
 * Retrieval and Weight Gathering"): each layer's listed rows copied once per group into contiguous buffers, which
 * every step of that group can then read in place of the scattered originals.  For every layer l of a stack and its list (one list per
 * layer, the group's mask: idx int32 [L][d_ff], count int32 [L], the rm_mask_compact layout with B = 1):
 *     out[l][0][i] = w[l].w_gate[idx[l][i]],  out[l][1][i] = w[l].w_up[idx[l][i]],
 *     out[l][2][i] = w[l].w_down[idx[l][i]]
 * for i < count[l] (clamped to max_count), and zero rows for count[l] <= i < max_count.
 *   out: [L][3][max_count][d] in the weights' dtype, 16-byte aligned, must not overlap the weights, idx or count.
 *   max_count in [1, d_ff].
 * Layer l's compact rows form an FFN layer of d_ff' = max_count neurons (w_gate = out[l][0] and so on) that the
 * FFN calls run with the identity lists 0 .. max_count-1 and the same counts, in the same slot order as the
 * original lists (so Eq. 4's h_anchor slots still match). */
rm_status rm_gather_stack_rows(const rm_ffn_shape *s, const rm_ffn_layer_weights *w, int32_t L, const int32_t *idx,
                               const int32_t *count, int32_t max_count, void *out, void *stream);

/* Context Cache, the rows to recompute (section 4.1, "Visual-Token Recomputation", Eq. 2).  Over a layer's N
 * token rows, of which rows [v0, v0 + P) are visual tokens:
 *   drift[p] = RMS(x[v0+p] - x_ref[v0+p]) / max(RMS(x[v0+p]), 1e-6), the Eq. 2 drift of each visual token, with
 *              x the current FFN input (after RMSNorm) and x_ref the reference execution's, both float32 [N][d];
 *   rows:      int32 [N] out: in its first count[0] entries, ascending, every non-visual row (Eq. 3 reuses a
 *              cached output only for a visual token) and the k visual rows with the largest drift (ties to the
 *              lower token); k = ceil(rho_p * P) in the paper;
 *   count:     int32 [1] out, (N - P) + k.
 * The drift is float32 (lane j of a wave adds the squares of columns j, j + 64, ...; the lanes' sums are folded
 * 32, 16, ..., 1 apart; rounded division and correctly rounded square roots), within float32 rounding of the
 * exact Eq. 2 value; the rows are the top k of these float32 values, the same on every call.  N <= 16384, 0 <= v0, v0 + P <= N, 0 <= k <= P; drift may be NULL when P = 0.
 * drift, rows and count must not overlap each other, x or x_ref.  Errors: RM_ERR_INVALID_ARG, RM_ERR_SHAPE,
 * RM_ERR_ALIGN (4-byte alignment). */
rm_status rm_context_select(const float *x, const float *x_ref, int32_t n_tok, int32_t d, int32_t v0, int32_t P,
                            int32_t k, float *drift, int32_t *rows, int32_t *count, void *stream);

/* Workspace bytes (written to *bytes, host pointer) of rm_context_ffn for n_tok rows with at most max_rows
 * recomputed. */
rm_status rm_context_workspace_size(const rm_ffn_shape *s, int32_t n_tok, int32_t max_rows, size_t *bytes);

/* Context Cache, the update of Eq. 3: the listed rows of y are replaced by F(x) of those rows, every other row
 * keeps the reference output the caller put there.  F(x) = (act(x W_gate^T) * (x W_up^T)) W_down, the VLM FFN
 * on its normalized input (no norm inside, no residual).
 *   s:        d a multiple of 64 and d_ff of 128, wdtype RM_BF16, act (GeGLU for the Gemma VLM of pi0.5); norm_eps
 *             unused.
 *   w_gate, w_up: bf16 [d_ff][d]; w_down_t: bf16 [d][d_ff], the nn.Linear layout of the down projection (this
 *             dense FFN reads every neuron, so both of its products take K-contiguous operands).
 *   x:        float32 [n_tok][d], the FFN input of every row (rounded to bf16 for the matrix cores).
 *   rows, count: the recomputed rows and their number (rm_context_select's outputs, read on the device);
 *             count is clamped to [0, max_rows] and rows outside [0, n_tok) to it.
 *   max_rows: host bound of count, in [1, n_tok]; sizes the launch and the workspace.
 *   y:        float32 [n_tok][d], in/out: the reference outputs on entry.
 *   ws, ws_bytes: at least rm_context_workspace_size(s, n_tok, max_rows) bytes, 16-byte aligned.
 * x, y and the workspace must not overlap, nor may the weights, rows or count overlap y or the workspace.
 * Errors: RM_ERR_INVALID_ARG, RM_ERR_SHAPE, RM_ERR_DTYPE, RM_ERR_ALIGN, RM_ERR_WORKSPACE, RM_ERR_HIP. */
rm_status rm_context_ffn(const rm_ffn_shape *s, const void *w_gate, const void *w_up, const void *w_down_t,
                         int32_t n_tok, const float *x, const int32_t *rows, const int32_t *count, int32_t max_rows,
                         float *y, void *ws, size_t ws_bytes, void *stream);

/* Bytes (written to *bytes, host pointer) of a layer's weights packed by rm_context_pack: 3 * d * d_ff * 2. */
rm_status rm_context_pack_size(const rm_ffn_shape *s, size_t *bytes);

/* The three matrices of one layer (the arguments of rm_context_ffn) copied into the blocked layout that
 * rm_context_ffn_packed reads: each matrix as 64-row x 64-column bf16 blocks of 8 KB, the blocks of a 64-row tile
 * consecutive along K, the 16-byte pieces of each block row permuted; w_gate, then w_up, then w_down_t.  Every
 * K stage of a weight tile is then one contiguous read.  A layout change only (no arithmetic); run it once when
 * the weights are loaded.
 *   packed, packed_bytes: device buffer of at least rm_context_pack_size bytes, 16-byte aligned, owned by the
 *             caller; it must not overlap the weights.
 * Errors: as rm_context_ffn for the shape and pointers; RM_ERR_WORKSPACE if packed_bytes is too small. */
rm_status rm_context_pack(const rm_ffn_shape *s, const void *w_gate, const void *w_up, const void *w_down_t,
                          void *packed, size_t packed_bytes, void *stream);

/* rm_context_ffn with the weights from rm_context_pack (same result bit for bit: only the weights' layout
 * differs).  packed must not overlap y or the workspace. */
rm_status rm_context_ffn_packed(const rm_ffn_shape *s, const void *packed, int32_t n_tok, const float *x,
                                const int32_t *rows, const int32_t *count, int32_t max_rows, float *y, void *ws,
                                size_t ws_bytes, void *stream);

/* Down-projection row norms ||W_down[n]||_2 of one layer (the weight factor of Eq. 1, section 3.4), float32.
 *   w_down: [d_ff][d] in wdtype (the layout of rm_ffn_layer_weights.w_down), 16-byte aligned; d a multiple of 32.
 *   norms:  float32 [d_ff] out.
 * Each norm is the correctly rounded square root of the float32 sum of the row's squares, added in column order
 * with every square and sum rounded to float32 (the order rm_group_masks' selections are defined with). */
rm_status rm_neuron_norms(const void *w_down, int32_t d_ff, int32_t d, int32_t wdtype, float *norms, void *stream);

/* Group neuron masks from the reference activations of a group of S denoising steps (section 5, "Constructing
 * Group Neuron Masks"): per layer, Eq. 1's score c[s][l][n] = (sum over t of |h[s][l][n][t]|) * norms[l][n] for
 * every step, each step's K best neurons as candidates, and as the mask the K candidates with the largest score
 * summed over the steps.
 *   h:      float32 [S][L][d_ff][T], neuron-major per step and layer (rm_anchor_ffn_stack run with the identity
 *           lists 0 .. d_ff-1 writes one step's [L][1][d_ff][T] as its h_anchor).
 *   norms:  float32 [L][d_ff] (rm_neuron_norms of each layer's w_down).
 *   K:      neurons per mask, in [0, d_ff] (section 5 takes K = ceil(rho_n * d_ff)).
 *   scores: float32 [S][L][d_ff] out, the Eq. 1 scores.
 *   mask:   uint8 [L][d_ff] out, 1 for the layer's K selected neurons, else 0 (the input of rm_mask_compact and
 *           rm_masked_ffn_*).
 * Sums run in index order in float32 with one rounding per operation; ties at the K-th place go to the lower
 * neuron index.  d_ff <= 16384, S * L <= 65535.  scores and mask must not overlap each other, h or norms.
 * Errors: RM_ERR_INVALID_ARG (null pointer, non-positive size, overlap), RM_ERR_SHAPE (d_ff, K or S * L out of
 * range), RM_ERR_ALIGN. */
rm_status rm_group_masks(const float *h, int32_t S, int32_t L, int32_t d_ff, int32_t T, const float *norms,
                         int32_t K, float *scores, uint8_t *mask, void *stream);

/* Measurement hook.  Arms two hipEvent_t (begin, end, created by the caller) for the next launch of the named
 * kernel by this thread: that launch goes through hipExtLaunchKernel, which stamps the events with the
 * kernel's own start and end, the interval a kernel trace reports.  The hook disarms after that launch;
 * passing NULL events disarms it.  kernel: an rm_kernel_id. */
typedef enum rm_kernel_id {
    RM_KERNEL_GATEUP = 0,      /* gate/up projection of the FFN calls                          */
    RM_KERNEL_DOWN = 1,        /* down projection of the FFN calls                             */
    RM_KERNEL_SCORES = 2,      /* Eq. 1 scores of rm_group_masks                               */
    RM_KERNEL_GROUP_SELECT = 3, /* top-K selection, union and rerank of rm_group_masks         */
    RM_KERNEL_LAYER = 4         /* gate/up and down of one layer in one launch (one sample's    */
                                /* long list at d = 2048, or a single layer's given list at    */
                                /* d = 1024: the workgroups of each XCD meet between the two   */
                                /* projections)                                                */
} rm_kernel_id;
rm_status rm_profile_kernel_events(int32_t kernel, void *ev_begin, void *ev_end);

/* Measurement: which of the hooked kernels a single-layer call on given lists (rm_sparse_ffn_layer) of this
 * shape launches on the current device: bit k of *kernels (a host pointer) is set for rm_kernel_id k
 * (RM_KERNEL_GATEUP and RM_KERNEL_DOWN, or RM_KERNEL_LAYER alone when the gate/up and down projections run in
 * one launch).  Host only; enqueues nothing.  Errors: those of rm_workspace_size. */
rm_status rm_layer_kernels(const rm_ffn_shape *s, int32_t B, int32_t T, int32_t max_count, uint32_t *kernels);

/* Measurement: a plain streaming read of `bytes` of `buf` (16-byte aligned, bytes a positive multiple of 16) by
 * `workgroups` workgroups of 512 threads, each lane keeping eight 16-byte loads in flight.  It computes nothing
 * the caller uses: sink (uint32 [workgroups * 512], 4-byte aligned, not overlapping buf) is written only in the
 * practically impossible case that a lane's XOR of its loads equals a fixed magic number.  Used to state the hot
 * path's bandwidth as a fraction of a bare read on the same GPU.  workgroups in [1, 1 << 20]. */
rm_status rm_stream_read(const void *buf, size_t bytes, int32_t workgroups, uint32_t *sink, void *stream);

/* Static description of a status code. */
const char *rm_status_string(rm_status status);

/* Detail of this thread's last failed call ("" if none). */
const char *rm_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* RMUSCLE_H */
