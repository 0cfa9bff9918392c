"""Benchmark of the Action Cache sparse-FFN hot path on one MI355X.

Workload (default): the wide FFN layer, the largest single-GPU configuration: bf16 weights / float32
activations, d = 2048, d_ff = 16384, T = 51 tokens (50 actions + 1 state), mask = top 30% of neurons (K = 4916) by
mean |SiLU(g) * u| on a reference input, evaluated on that input + 0.1 N(0,1).  One step is the whole hot path for
one batch: rm_masked_ffn_layer, i.e. the compaction of the layer's mask into its index list (in the launch of the
layer's first kernel) and the masked layer.

Weights are cold: every step reads a different one of R copies of the layer (>= 1 GiB together), so neither
L2 nor the 256 MB Infinity Cache can serve them and the weight bytes come from HBM.  Activations, mask and
index list are small and stay resident.

Steps are replayed from HIP graphs (captured through torch.cuda.CUDAGraph), the way a denoising loop is run in
deployment: a graph of one step per weight copy, plus a graph of the remainder so that exactly K steps are
timed.  Every kernel of every step runs; the graph only removes per-launch host and dispatch overhead.  The
same steps launched one call at a time are reported as eager_us_per_layer.

The printed JSON line gives value = achieved GB/s on active weight bytes (3 K d * 2 B per step) over the timed
steps, the roofline of the dominant kernel (its algorithmic bytes / its average duration from HIP events
recorded around its launches by the library's measurement hook, on the launch stream), and the float64 CPU
oracle timed on a bounded sample of the same workload.  Beside them: the distribution of single-step times (each
step a graph replay between two events), the mask compaction timed on its own, the bandwidth of a plain streaming
read on the same GPU (rm_stream_read) and the fraction of it the step reaches, and, for the default workload, the
per-layer figures of configurations 2, 3 and 5 (secondary; one graph-replayed run each).

Other workloads (--workload): config 2's layer d = 1024, d_ff = 4096 (c2); the wide layer at 10/50/100% (c4-*);
the 18-layer stack
run through a 10-step denoising schedule, one step of the benchmark being the whole sequence (c3); the same
sequence with Eq. 4's dense anchors at steps 0 and 5 and anchor-delta updates at the other steps (c3-eq4), also
with the group's rows copied into compact buffers first (c3-eq4-compact); and
16 independent executions through the stack with per-sample lists (c5); and the construction of one group's
neuron masks from 5 reference steps of the stack (gm); and the Context Cache's token recomputation on one VLM
FFN layer (cc).

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W]
                       [--workload c4-30|c2|c4-10|c4-50|c4-100|c3|c3-eq4|c3-eq4-compact|c5|gm|cc]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, 8 TB/s
BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix cores (no sparsity)
PROFILES = os.path.join(ROOT, "profiles")
CSRC = os.path.join(ROOT, "paper_2609_19104_amd", "csrc")
COLD_BYTES = 1 << 30   # weight copies rotated through per timed run


# ----------------------------------------------------------------------------------------------------------
# Byte / FLOP accounting (algorithmic: active weights only)
# ----------------------------------------------------------------------------------------------------------

def projection_flops(tokens: int, d: int, d_ff: int) -> int:
    """FLOPs of one dense projection between widths d and d_ff at `tokens` tokens (multiply + add)."""
    return 2 * tokens * d * d_ff


def matrix_bytes(d: int, d_ff: int, elem_bytes: int) -> int:
    return d * d_ff * elem_bytes


def gateup_bytes(k: int, d: int, elem_bytes: int) -> int:
    """Active weight bytes of the gate/up kernel: two rows of d weights per listed neuron."""
    return 2 * k * d * elem_bytes


def down_bytes(k: int, d: int, elem_bytes: int) -> int:
    """Active weight bytes of the down kernel: one neuron-major row of d weights per listed neuron."""
    return k * d * elem_bytes


def active_weight_bytes(k: int, d: int, elem_bytes: int) -> int:
    return gateup_bytes(k, d, elem_bytes) + down_bytes(k, d, elem_bytes)


# ----------------------------------------------------------------------------------------------------------
# Workloads
# ----------------------------------------------------------------------------------------------------------

WORKLOADS = {
    "c2": dict(name="pi0 action-expert FFN layer, bf16, d=1024 d_ff=4096 T=51, top-30% mask", cfg=2, percent=30),
    "c4-10": dict(name="wide FFN layer, bf16, d=2048 d_ff=16384 T=51, top-10% mask", cfg=4, percent=10),
    "c4-30": dict(name="wide FFN layer, bf16, d=2048 d_ff=16384 T=51, top-30% mask", cfg=4, percent=30),
    "c4-50": dict(name="wide FFN layer, bf16, d=2048 d_ff=16384 T=51, top-50% mask", cfg=4, percent=50),
    "c4-100": dict(name="wide FFN layer, bf16, d=2048 d_ff=16384 T=51, all neurons", cfg=4, percent=100),
    "c3": dict(name="action-expert FFN stack, 18 layers, RMSNorm, d=1024 d_ff=4096 T=51, 10 denoising steps "
                    "(step 0 dense; top-30% masks refreshed at steps 1, 3, 5, 7, 9)", cfg=3, percent=30),
    "c3-eq4": dict(name="action-expert FFN stack, 18 layers, RMSNorm, d=1024 d_ff=4096 T=51, 10 denoising steps "
                        "with Eq. 4: dense anchors at steps 0 and 5, each shared by the next 4 steps with top-30% "
                        "group masks", cfg=3, percent=30),
    "c3-eq4-compact": dict(name="the c3-eq4 sequence with the group's selected rows copied into compact buffers "
                                "(on a side stream, during the anchor step) and the delta steps run on them",
                           cfg=3, percent=30),
    "cc": dict(name="Context Cache, one VLM FFN layer: 850 rows (768 visual), d=2048 d_ff=16384, GeGLU, bf16, "
                    "rho_p=0.4 (308 visual + 82 other rows recomputed)", cfg=6, percent=40),
    "gm": dict(name="group neuron masks for the config-3 stack: 5 reference steps x 18 layers, d_ff=4096, T=51, "
                    "K=1229 (top 30%)", cfg=3, percent=30),
    "c5": dict(name="16 independent executions x 18 layers, RMSNorm, d=1024 d_ff=4096 T=51, per-sample top-30% "
                    "masks (18% shared core + random remainder)", cfg=5, percent=30),
}


STEP_TEXT = {
    "c2": "rm_sparse_ffn_layer on the mask's list, compacted once at set-up (the group's cached list, shared by its "
          "steps), replayed from HIP graphs; masked_us_per_layer: rm_masked_ffn_layer (compaction + layer) per step",
    "c4": "rm_sparse_ffn_layer on the mask's list, compacted once at set-up (the group's cached list, shared by its "
          "steps), replayed from HIP graphs; masked_us_per_layer: rm_masked_ffn_layer (compaction + layer) per step",
    "c3": "one 10-step sequence: rm_sparse_ffn_stack (L=18) over identity lists (the dense step), then 5 "
          "rm_masked_ffn_stack (L=18, compacting the refreshed 18 masks) alternating with 4 rm_sparse_ffn_stack "
          "(L=18), replayed from HIP graphs; "
          "us_per_layer = sequence time / 180",
    "c3-eq4": "one 10-step sequence: per group (anchors 0 and 5) rm_mask_compact (18 masks) + "
              "rm_anchor_ffn_stack (L=18) + 4 rm_delta_ffn_stack (L=18), replayed from HIP graphs; "
              "us_per_layer = sequence time / 180",
    "c3-eq4-compact": "one 10-step sequence: per group rm_mask_compact (18 masks), then rm_gather_stack_rows "
                      "(18 layers x 3 matrices) on a side stream beside rm_anchor_ffn_stack (L=18), then 4 "
                      "rm_delta_ffn_stack (L=18) on the compact layers; replayed from HIP graphs; "
                      "us_per_layer = sequence time / 180",
    "cc": "rm_context_select (Eq. 2 drift of the 768 visual rows, top 308 + the 82 other rows) + "
          "rm_context_ffn_packed (gathered rows through the gate/up and down GEMMs on the weights packed once by "
          "rm_context_pack, scattered into the reference outputs), replayed from HIP graphs",
    "gm": "rm_group_masks: Eq. 1 scores of 5 steps x 18 layers from their dense activations (float32 "
          "[5][18][4096][51], written by rm_anchor_ffn_stack with identity lists at set-up), per-step top-K, union "
          "and rerank; replayed from HIP graphs; us_per_layer = step time / 18",
    "c5": "rm_masked_ffn_stack (L=18, B=16: compaction of the 288 masks + the stack), replayed from HIP graphs; "
          "us_per_layer = step time / 18; value on the union of the samples' rows, per_sample_value on all rows",
}


def ffn_hooks(rm, gu_bytes: int, dn_bytes: int):
    """The kernels a FFN step's timing hook follows: (kernel id, description, key, algorithmic bytes per launch)."""
    return [(rm.RM_KERNEL_GATEUP, "gate/up projection (gateup_*_kernel)", "gateup", gu_bytes),
            (rm.RM_KERNEL_DOWN, "down projection (down_*_kernel)", "down", dn_bytes)]


def _bf16_tensor(bits, device):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(device)


def score_mask_on_device(x_ref, wg, wu, k: int):
    """Top-k neurons by mean |SiLU(x_ref Wg^T) * (x_ref Wu^T)| over tokens, float64 on the GPU (input setup).

    Ties go to the lower neuron index (stable sort)."""
    import torch
    import torch.nn.functional as F
    xr = x_ref.to(torch.float64)
    h = F.silu(xr @ wg.to(torch.float64).T) * (xr @ wu.to(torch.float64).T)
    score = h.abs().mean(dim=0)
    order = torch.sort(score, descending=True, stable=True).indices
    mask = torch.zeros(score.shape[0], dtype=torch.uint8, device=score.device)
    mask[order[:k]] = 1
    return mask


class Setup:
    """Device-resident inputs of a workload, with R rotating weight copies."""

    def __init__(self, key: str, device, cold: bool = True):
        import torch
        import workloads as wl
        import paper_2609_19104_amd as rm

        spec = WORKLOADS[key]
        w = wl.config2() if spec["cfg"] == 2 else wl.config4(percents=(spec["percent"],))
        self.key, self.spec, self.wl = key, spec, w
        layer = w.layers[0]
        self.d, self.d_ff, self.T, self.B = w.d, w.d_ff, w.T, w.B
        self.k = wl.count_for_percent(spec["percent"], w.d_ff)
        self.layer_np = layer
        base = (_bf16_tensor(layer.w_gate, device), _bf16_tensor(layer.w_up, device),
                _bf16_tensor(layer.w_down, device), None)
        self.x = torch.from_numpy(w.x.reshape(self.B, self.T, self.d)).to(device)
        self.x_ref = torch.from_numpy(w.x_ref.reshape(self.B * self.T, self.d)).to(device)
        self.mask = score_mask_on_device(self.x_ref, base[0], base[1], self.k).reshape(1, self.d_ff)
        dense_bytes = 3 * matrix_bytes(self.d, self.d_ff, 2)
        self.copies = max(2, math.ceil(COLD_BYTES / dense_bytes)) if cold else 1
        self.layers = [base] + [tuple(t.clone() if t is not None else None for t in base)
                                for _ in range(self.copies - 1)]
        self.rotate = self.copies  # copies cycled through by step(); 1 = warm (same weights every step)
        self.y = torch.empty_like(self.x)
        self.idx = torch.empty((1, self.d_ff), dtype=torch.int32, device=device)
        self.cnt = torch.empty((1,), dtype=torch.int32, device=device)
        self.ws = rm.workspace(self.d, self.d_ff, rm.RM_BF16, self.B, self.T, self.k, device=device)
        self.rm = rm
        self.L, self.layer_steps = 1, 1
        # A step is the layer on the group's cached list (compacted here, once); with lists = False it is the
        # call that compacts the mask too.
        self.lists = True
        rm.rm_mask_compact(self.mask, self.idx, self.cnt)

    def step(self, i: int) -> None:
        if self.lists:  # the group's cached list (compacted once at set-up): the layer alone
            self.rm.rm_sparse_ffn_layer(self.x, self.y, self.layers[i % self.rotate], self.idx, self.cnt, self.k,
                                        self.ws)
        else:
            self.rm.rm_masked_ffn_layer(self.x, self.y, self.layers[i % self.rotate], self.mask, self.idx, self.cnt,
                                        self.k, self.ws)

    def compact(self) -> None:  # the step's mask compaction alone
        self.rm.rm_mask_compact(self.mask, self.idx, self.cnt)

    @property
    def active_bytes(self) -> int:
        return active_weight_bytes(self.k, self.d, 2)

    def hooks(self):
        gu, dn = gateup_bytes(self.k, self.d, 2), down_bytes(self.k, self.d, 2)
        if self.rm.rm_layer_kernels(self.d, self.d_ff, self.rm.RM_BF16, self.B, self.T, self.k) == \
                1 << self.rm.RM_KERNEL_LAYER:  # gate/up and down in one launch (layer_xcd_kernel)
            return [(self.rm.RM_KERNEL_LAYER, "gate/up + down projections in one launch (layer_xcd_kernel)",
                     "layer", gu + dn)]
        return ffn_hooks(self.rm, gu, dn)


def _stack_copies(layers, device, cold: bool):
    """Device weights of every layer ((w_gate, w_up, w_down, g) per layer), repeated in enough copies to rotate
    over >= 1 GiB when cold."""
    import torch
    base = [(_bf16_tensor(l.w_gate, device), _bf16_tensor(l.w_up, device), _bf16_tensor(l.w_down, device),
             torch.from_numpy(l.norm_g).to(device) if l.norm_g is not None else None) for l in layers]
    dense = sum(3 * matrix_bytes(l.d, l.d_ff, 2) for l in layers)
    copies = max(2, math.ceil(COLD_BYTES / dense)) if cold else 1
    return [base] + [[tuple(t.clone() if t is not None else None for t in lw) for lw in base]
                     for _ in range(copies - 1)], copies


class StackSetup5:
    """Config 5: B = 16 executions through an 18-layer stack, each with its own list per layer.  One step is one
    rm_masked_ffn_stack call: the compaction of all L B masks and the stack."""

    def __init__(self, key: str, device, cold: bool = True):
        import torch
        import workloads as wl
        import paper_2609_19104_amd as rm
        w = wl.config5()
        self.key, self.spec, self.rm = key, WORKLOADS[key], rm
        self.d, self.d_ff, self.T, self.B, self.L, self.k = w.d, w.d_ff, w.T, w.B, w.L, w.k
        self.layer_copies, self.copies = _stack_copies(w.layers, device, cold)
        self.rotate = self.copies
        self.mask = torch.from_numpy(w.masks.reshape(self.L * self.B, self.d_ff)).to(device)
        self.idx = torch.empty((self.L * self.B, self.d_ff), dtype=torch.int32, device=device)
        self.cnt = torch.empty((self.L * self.B,), dtype=torch.int32, device=device)
        self.x = torch.from_numpy(w.x).to(device)
        self.y = torch.empty_like(self.x)
        self.ws = rm.workspace(self.d, self.d_ff, rm.RM_BF16, self.B, self.T, self.k, device=device)
        self.union = [int((w.masks[l] != 0).any(axis=0).sum()) for l in range(self.L)]
        self.layer_steps = self.L

    def step(self, i: int) -> None:
        self.rm.rm_masked_ffn_stack(self.x, self.y, self.layer_copies[i % self.rotate], self.mask, self.idx, self.cnt,
                                    self.k, self.ws)

    def compact(self) -> None:  # the compaction of the step's L B masks alone
        self.rm.rm_mask_compact(self.mask, self.idx, self.cnt)

    def useful_flops(self) -> int:  # 3 projections x 2 FLOP per weight per token, each sample's own list
        return self.L * self.B * 3 * projection_flops(self.T, self.d, self.k)

    @property
    def active_bytes(self) -> int:  # distinct rows per layer call (the union of the samples' lists)
        return sum(active_weight_bytes(u, self.d, 2) for u in self.union)

    @property
    def per_sample_bytes(self) -> int:
        return self.L * self.B * active_weight_bytes(self.k, self.d, 2)

    def hooks(self):  # the first gate/up and down launches of a step: layer 0, all samples
        return ffn_hooks(self.rm, gateup_bytes(self.union[0], self.d, 2), down_bytes(self.union[0], self.d, 2))


class StackSetup3:
    """Config 3: one step is a whole 10-step denoising sequence through the 18-layer stack: step 0 dense (one
    rm_sparse_ffn_stack over identity lists, every neuron in order), steps 1..9 sparse, with the 18 per-layer
    masks compacted at steps 1, 3, 5, 7, 9 (rm_masked_ffn_stack) and their lists reused by the following step
    (rm_sparse_ffn_stack).  The masks are the top-30% neurons by mean |SiLU(g) u| of a float32 dense pass on the
    previous step's input (input setup, on the GPU)."""

    def __init__(self, key: str, device, cold: bool = True):
        import torch
        import torch.nn.functional as F
        import workloads as wl
        import paper_2609_19104_amd as rm
        w = wl.config3()
        self.key, self.spec, self.rm = key, WORKLOADS[key], rm
        self.d, self.d_ff, self.T, self.B, self.L, self.k = w.d, w.d_ff, w.T, 1, w.L, w.k
        self.steps, self.refresh = w.steps, list(w.refresh_steps)
        self.layer_copies, self.copies = _stack_copies(w.layers, device, cold)
        self.rotate = self.copies
        self.xs = [torch.from_numpy(x).to(device) for x in w.x_steps]
        masks = []
        base = self.layer_copies[0]
        for s in self.refresh:
            xl = self.xs[s - 1][0].to(torch.float32)
            m = []
            for (wg, wu, wd, g) in base:
                xn = xl * torch.rsqrt((xl * xl).mean(dim=-1, keepdim=True) + 1e-6) * g
                h = F.silu(xn @ wg.float().T) * (xn @ wu.float().T)
                order = torch.sort(h.abs().mean(dim=0), descending=True, stable=True).indices
                mk = torch.zeros(self.d_ff, dtype=torch.uint8, device=device)
                mk[order[:self.k]] = 1
                m.append(mk)
                xl = xl + h @ wd.float()
            masks.append(torch.stack(m))
        self.masks = masks  # [refreshes] x [L][d_ff]
        self.idx = [torch.empty((self.L, self.d_ff), dtype=torch.int32, device=device) for _ in self.refresh]
        self.cnt = [torch.empty((self.L,), dtype=torch.int32, device=device) for _ in self.refresh]
        self.y = torch.empty_like(self.xs[0])
        self.ws = rm.workspace(self.d, self.d_ff, rm.RM_BF16, 1, self.T, self.k, device=device)
        self.ws_dense = rm.workspace(self.d, self.d_ff, rm.RM_BF16, 1, self.T, self.d_ff, device=device)
        self.ident = torch.arange(self.d_ff, dtype=torch.int32, device=device).repeat(self.L, 1).contiguous()
        self.ident_cnt = torch.full((self.L,), self.d_ff, dtype=torch.int32, device=device)
        self.layer_steps = self.steps * self.L

    # The measurement hook is armed inside the step, right before step 2's stack (the first step that only reads
    # its lists), so the timed launches are layer 0's sparse gate/up and down.
    arm_inside = True

    def step(self, i: int) -> None:
        rm, layers = self.rm, self.layer_copies[i % self.rotate]
        rm.rm_sparse_ffn_stack(self.xs[0], self.y, layers, self.ident, self.ident_cnt, self.d_ff, self.ws_dense)
        for s in range(1, self.steps):
            r = (s - 1) // 2
            if s == 2:
                _arm(self)
            if s in self.refresh:
                rm.rm_masked_ffn_stack(self.xs[s], self.y, layers, self.masks[r], self.idx[r], self.cnt[r], self.k,
                                       self.ws)
            else:
                rm.rm_sparse_ffn_stack(self.xs[s], self.y, layers, self.idx[r], self.cnt[r], self.k, self.ws)

    @property
    def active_bytes(self) -> int:  # dense step + sparse steps
        return self.L * (active_weight_bytes(self.d_ff, self.d, 2)
                         + (self.steps - 1) * active_weight_bytes(self.k, self.d, 2))

    def compact(self) -> None:  # one refresh's compaction of the 18 layer masks alone
        self.rm.rm_mask_compact(self.masks[0], self.idx[0], self.cnt[0])

    def hooks(self):  # layer 0's gate/up and down of step 2 (a sparse step on the refreshed lists)
        return ffn_hooks(self.rm, gateup_bytes(self.k, self.d, 2), down_bytes(self.k, self.d, 2))


class StackSetupEq4:
    """The paper's anchored schedule (section 4.1) on the config-3 stack: one step is a 10-step sequence of two
    groups.  Each group compacts its 18 layer masks, runs its anchor step densely with rm_anchor_ffn_stack
    (keeping y_a and the listed h_a) and its 4 later steps with rm_delta_ffn_stack (Eq. 4).  A group's masks
    are the top-30% neurons by mean |SiLU(g) u| of a float32 dense pass on a similar input (the anchor input +
    0.1 N(0,1)), computed on the GPU at set-up."""

    ANCHORS = (0, 5)

    def __init__(self, key: str, device, cold: bool = True):
        import torch
        import torch.nn.functional as F
        import workloads as wl
        import paper_2609_19104_amd as rm
        w = wl.config3()
        self.key, self.spec, self.rm = key, WORKLOADS[key], rm
        self.d, self.d_ff, self.T, self.B, self.L, self.k = w.d, w.d_ff, w.T, 1, w.L, w.k
        self.steps = w.steps
        self.layer_copies, self.copies = _stack_copies(w.layers, device, cold)
        self.rotate = self.copies
        self.xs = [torch.from_numpy(x).to(device) for x in w.x_steps]
        base = self.layer_copies[0]
        self.masks = []
        for xr in wl.group_reference_inputs(w, self.ANCHORS):
            xl = torch.from_numpy(xr[0]).to(device)
            m = []
            for (wg, wu, wd, g) in base:
                xn = xl * torch.rsqrt((xl * xl).mean(dim=-1, keepdim=True) + 1e-6) * g
                h = F.silu(xn @ wg.float().T) * (xn @ wu.float().T)
                order = torch.sort(h.abs().mean(dim=0), descending=True, stable=True).indices
                mk = torch.zeros(self.d_ff, dtype=torch.uint8, device=device)
                mk[order[:self.k]] = 1
                m.append(mk)
                xl = xl + h @ wd.float()
            self.masks.append(torch.stack(m))
        self.idx = [torch.empty((self.L, self.d_ff), dtype=torch.int32, device=device) for _ in self.ANCHORS]
        self.cnt = [torch.empty((self.L,), dtype=torch.int32, device=device) for _ in self.ANCHORS]
        self.ya = torch.empty((self.L, 1, self.T, self.d), dtype=torch.float32, device=device)
        self.ha = torch.empty((self.L, 1, self.k, self.T), dtype=torch.float32, device=device)
        self.y = torch.empty_like(self.xs[0])
        self.ws = rm.workspace(self.d, self.d_ff, rm.RM_BF16, 1, self.T, self.k, device=device)
        self.ws_dense = rm.workspace(self.d, self.d_ff, rm.RM_BF16, 1, self.T, self.d_ff, device=device)
        self.layer_steps = self.steps * self.L

    def step(self, i: int) -> None:
        rm, layers = self.rm, self.layer_copies[i % self.rotate]
        for s in range(self.steps):
            if s in self.ANCHORS:
                g = self.ANCHORS.index(s)
                rm.rm_mask_compact(self.masks[g], self.idx[g], self.cnt[g])
                rm.rm_anchor_ffn_stack(self.xs[s], self.y, layers, self.idx[g], self.cnt[g], self.k, self.ya,
                                       self.ha, self.ws_dense)
            else:
                if s == 1:
                    _arm(self)
                rm.rm_delta_ffn_stack(self.xs[s], self.y, layers, self.idx[g], self.cnt[g], self.k, self.ya,
                                      self.ha, self.ws)

    # The measurement hook is armed inside the step, right before step 1 (the first Eq. 4 delta step).
    arm_inside = True

    def compact(self) -> None:  # one group's compaction of the 18 layer masks alone
        self.rm.rm_mask_compact(self.masks[0], self.idx[0], self.cnt[0])

    @property
    def active_bytes(self) -> int:  # anchors read every row, later steps the listed rows
        n_anchor = len(self.ANCHORS)
        return self.L * (n_anchor * active_weight_bytes(self.d_ff, self.d, 2)
                         + (self.steps - n_anchor) * active_weight_bytes(self.k, self.d, 2))

    def hooks(self):  # layer 0's gate/up and down of step 1 (the first delta step, on the group's lists)
        return ffn_hooks(self.rm, gateup_bytes(self.k, self.d, 2), down_bytes(self.k, self.d, 2))


class StackSetupEq4Compact(StackSetupEq4):
    """The anchored schedule with section 4.1's compact buffers: each group's selected rows of the 18 layers are
    copied once (rm_gather_stack_rows, on a side stream while the main stream runs the dense anchor step) and the
    group's delta steps read those contiguous rows through the identity lists."""

    def __init__(self, key: str, device, cold: bool = True):
        import torch
        super().__init__(key, device, cold)
        # One compact buffer per group (the two groups' copies would alternate in a deployment; here each group
        # keeps its own so that replays need no ordering between them).
        self.rows = [torch.empty((self.L, 3, self.k, self.d), dtype=torch.bfloat16, device=device)
                        for _ in self.ANCHORS]
        self.ident = torch.arange(self.k, dtype=torch.int32, device=device).repeat(self.L, 1).contiguous()
        self.ws_c = self.rm.workspace(self.d, self.k, self.rm.RM_BF16, 1, self.T, self.k, device=device)
        self.side = torch.cuda.Stream(device=device)

    def step(self, i: int) -> None:
        import torch
        rm, layers = self.rm, self.layer_copies[i % self.rotate]
        main = torch.cuda.current_stream()
        for s in range(self.steps):
            if s in self.ANCHORS:
                g = self.ANCHORS.index(s)
                rm.rm_mask_compact(self.masks[g], self.idx[g], self.cnt[g])
                self.side.wait_stream(main)
                with torch.cuda.stream(self.side):
                    rm.rm_gather_stack_rows(layers, self.idx[g], self.cnt[g], self.k, self.rows[g])
                rm.rm_anchor_ffn_stack(self.xs[s], self.y, layers, self.idx[g], self.cnt[g], self.k, self.ya,
                                       self.ha, self.ws_dense)
                main.wait_stream(self.side)
                clayers = [(self.rows[g][l, 0], self.rows[g][l, 1], self.rows[g][l, 2], layers[l][3])
                           for l in range(self.L)]
            else:
                if s == 1:
                    _arm(self)
                rm.rm_delta_ffn_stack(self.xs[s], self.y, clayers, self.ident, self.cnt[g], self.k, self.ya,
                                      self.ha, self.ws_c)


class ContextSetup:
    """The Context Cache step (section 4.1, Eq. 2 and Eq. 3) on one VLM FFN layer: select the rows to recompute
    from the drift of the current FFN inputs against the reference's, then recompute them (all weights read;
    the copies rotate over >= 1 GiB so the reads are cold)."""

    bound = "mfma"

    def __init__(self, key: str, device, cold: bool = True):
        import torch
        import workloads as wl
        import paper_2609_19104_amd as rm
        w = wl.context_workload()
        self.key, self.spec, self.rm, self.w = key, WORKLOADS[key], rm, w
        self.d, self.d_ff, self.T, self.B, self.L, self.k = w.d, w.d_ff, w.n_tok, 1, 1, w.k
        self.rows_max = w.n_tok - w.P + w.k
        base = (_bf16_tensor(w.layer.w_gate, device), _bf16_tensor(w.layer.w_up, device),
                _bf16_tensor(w.w_down_t, device))
        self.copies = max(2, math.ceil(COLD_BYTES / (3 * matrix_bytes(self.d, self.d_ff, 2)))) if cold else 1
        # The weights packed once, as at model load (rm_context_pack: a layout change only); each copy is packed
        # from its own clone so that no two copies share memory.
        self.weights = [rm.rm_context_pack(*base)]
        for _ in range(self.copies - 1):
            self.weights.append(rm.rm_context_pack(*(t.clone() for t in base)))
        del base
        self.rotate = self.copies
        self.x = torch.from_numpy(w.x).to(device)
        self.x_ref = torch.from_numpy(w.x_ref).to(device)
        self.y = torch.from_numpy(w.y_ref).to(device)
        self.drift = torch.empty((w.P,), dtype=torch.float32, device=device)
        self.rows = torch.empty((w.n_tok,), dtype=torch.int32, device=device)
        self.count = torch.empty((1,), dtype=torch.int32, device=device)
        self.ws = rm.context_workspace(self.d, self.d_ff, w.n_tok, self.rows_max, device=device)
        self.layer_steps = 1
        self.cold_text = (f"cold: {self.copies} rotating copies of the layer's weights "
                          f"({self.copies * 3 * matrix_bytes(self.d, self.d_ff, 2) / 2**30:.2f} GiB)")

    def step(self, i: int) -> None:
        w, packed = self.w, self.weights[i % self.rotate]
        self.rm.rm_context_select(self.x, self.x_ref, w.v0, w.P, w.k, self.drift, self.rows, self.count)
        self.rm.rm_context_ffn_packed(self.x, self.y, packed, self.rows, self.count, self.rows_max, self.ws)

    @property
    def active_bytes(self) -> int:  # every weight of the layer is read
        return 3 * matrix_bytes(self.d, self.d_ff, 2)

    def hooks(self):  # matrix-core FLOPs of the two GEMMs over the recomputed rows
        rm, r = self.rm, self.rows_max
        return [(rm.RM_KERNEL_GATEUP, "gate/up GEMM over the gathered rows (gemm_nt_kernel, GLU)", "gateup",
                 2 * projection_flops(r, self.d, self.d_ff)),
                (rm.RM_KERNEL_DOWN, "down GEMM with the scatter (gemm_nt_kernel, scatter)", "down",
                 projection_flops(r, self.d, self.d_ff))]


class GroupMaskSetup:
    """Group-mask construction (section 5) for one group of the config-3 stack: the dense activations of 5
    reference steps (inputs x_0 .. x_4 of config 3, each run through rm_anchor_ffn_stack with the identity lists,
    at set-up) -> rm_group_masks.  The activations rotate over copies (>= 1 GiB) so the timed reads are cold."""

    STEPS = 5

    def __init__(self, key: str, device, cold: bool = True):
        import torch
        import workloads as wl
        import paper_2609_19104_amd as rm
        w = wl.config3()
        self.key, self.spec, self.rm = key, WORKLOADS[key], rm
        self.d, self.d_ff, self.T, self.B, self.L, self.k = w.d, w.d_ff, w.T, 1, w.L, w.k
        layers, _ = _stack_copies(w.layers, device, cold=False)
        layers = layers[0]
        idx = torch.arange(self.d_ff, dtype=torch.int32, device=device).repeat(self.L, 1).contiguous()
        cnt = torch.full((self.L,), self.d_ff, dtype=torch.int32, device=device)
        ws = rm.workspace(self.d, self.d_ff, rm.RM_BF16, 1, self.T, self.d_ff, device=device)
        h = torch.empty((self.STEPS, self.L, self.d_ff, self.T), dtype=torch.float32, device=device)
        ya = torch.empty((self.L, 1, self.T, self.d), dtype=torch.float32, device=device)
        ha = torch.empty((self.L, 1, self.d_ff, self.T), dtype=torch.float32, device=device)
        for s in range(self.STEPS):
            x = torch.from_numpy(w.x_steps[s]).to(device)
            rm.rm_anchor_ffn_stack(x, torch.empty_like(x), layers, idx, cnt, self.d_ff, ya, ha, ws)
            h[s] = ha[:, 0]
        self.norms = torch.empty((self.L, self.d_ff), dtype=torch.float32, device=device)
        for l in range(self.L):
            rm.rm_neuron_norms(layers[l][2], self.norms[l])
        torch.cuda.synchronize()
        del layers, ws
        self.h_bytes = h.numel() * 4
        self.copies = max(2, math.ceil(COLD_BYTES / self.h_bytes)) if cold else 1
        self.hs = [h] + [h.clone() for _ in range(self.copies - 1)]
        self.rotate = self.copies
        self.cold_text = (f"cold: {self.copies} rotating copies of the activations "
                          f"({self.copies * self.h_bytes / 2**30:.2f} GiB)")
        self.scores = torch.empty((self.STEPS, self.L, self.d_ff), dtype=torch.float32, device=device)
        self.mask = torch.empty((self.L, self.d_ff), dtype=torch.uint8, device=device)
        self.layer_steps = self.L

    def step(self, i: int) -> None:
        self.rm.rm_group_masks(self.hs[i % self.rotate], self.norms, self.k, self.scores, self.mask)

    def coverage(self) -> dict:
        """Section 3.4's coverage (share of a step's summed Eq. 1 contribution inside a mask) of the group's shared
        mask and of each step's own top-K mask (rm_group_masks over that step alone), over the 5 steps x 18
        layers.  Untimed; the ratio is a property of the synthetic activations, not of a trained model."""
        import torch
        h = self.hs[0]
        self.rm.rm_group_masks(h, self.norms, self.k, self.scores, self.mask)
        sc = self.scores.double()
        tot = sc.sum(-1)
        shared = (sc * (self.mask != 0)).sum(-1) / tot
        own = torch.empty_like(shared)
        s_scores = torch.empty((1, self.L, self.d_ff), dtype=torch.float32, device=h.device)
        s_mask = torch.empty_like(self.mask)
        for s in range(self.STEPS):
            self.rm.rm_group_masks(h[s:s + 1], self.norms, self.k, s_scores, s_mask)
            own[s] = (sc[s] * (s_mask != 0)).sum(-1) / tot[s]
        return {"k": self.k, "step_specific_mean": round(own.mean().item(), 4),
                "group_shared_mean": round(shared.mean().item(), 4),
                "group_shared_min": round(shared.min().item(), 4),
                "shared_over_specific_min": round((shared / own).min().item(), 4)}

    @property
    def active_bytes(self) -> int:  # the activations read (the norms, scores and masks are < 2% more)
        return self.h_bytes

    def hooks(self):
        rm, sl = self.rm, self.STEPS * self.L
        score_bytes = self.h_bytes + 4 * self.L * self.d_ff + 4 * sl * self.d_ff
        select_bytes = 4 * sl * self.d_ff + self.L * self.d_ff
        return [(rm.RM_KERNEL_SCORES, "Eq. 1 scores (scores_kernel)", "scores", score_bytes),
                (rm.RM_KERNEL_GROUP_SELECT, "top-K, union and rerank (group_select_kernel)", "select", select_bytes)]


def _arm(setup) -> None:
    """Arms the measurement hook's events for the current step, where a setup does so inside its step."""
    fn = getattr(setup, "arm", None)
    if fn is not None:
        fn()
        setup.arm = None


def time_steps(setup: Setup, steps: int, warmup: int, hook: bool = False):
    """Time `steps` steps after `warmup` untimed ones.  With hook=True, also hand the library a pair of HIP events
    for every gate/up and down launch (it launches them with hipExtLaunchKernel, which stamps the kernel's own
    start and end on its stream) and return their average durations in microseconds."""
    import torch
    rm = setup.rm
    for i in range(warmup):
        setup.step(i)
    torch.cuda.synchronize()
    evs = None
    if hook:
        evs = {kk: [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                    for _ in range(steps)] for kk, _, _, _ in setup.hooks()}
        for pairs in evs.values():  # create the underlying events before handing them to the library
            for a, b in pairs:
                a.record()
                b.record()
        torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    if hook:
        # A spin kernel ahead of the hooked steps keeps the device busy while the host enqueues them, so the
        # steps then run back to back as in the graph replay instead of one kernel per host call.
        torch.cuda._sleep(int(2e6) * steps)
    start.record()
    for i in range(steps):
        if hook:
            def arm(i=i):
                for kk, pairs in evs.items():
                    rm.rm_profile_kernel_events(kk, pairs[i][0].cuda_event, pairs[i][1].cuda_event)
            if getattr(setup, "arm_inside", False):
                setup.arm = arm
            else:
                arm()
        setup.step(warmup + i)
    end.record()
    torch.cuda.synchronize()
    if hook:  # disarm: a slot armed for a kernel the step did not launch must not catch a later launch
        for kk in evs:
            rm.rm_profile_kernel_events(kk, None, None)
    ms = start.elapsed_time(end) / steps
    kern = None
    if hook:
        kern = {}
        for kk, pairs in evs.items():
            us = np.array([a.elapsed_time(b) for a, b in pairs]) * 1e3
            kern[kk] = {"mean": float(us.mean()), "median": float(np.median(us)), "min": float(us.min()),
                        "p10": float(np.percentile(us, 10)), "p90": float(np.percentile(us, 90))}
    return ms, kern


def _capture(setup: Setup, first: int, n: int):
    """A CUDA/HIP graph of n consecutive steps starting at step index `first`."""
    import torch
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm the calls on a side stream before capture
        for i in range(n):
            setup.step(first + i)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for i in range(n):
            setup.step(first + i)
    torch.cuda.synchronize()
    return g


def time_graph(setup: Setup, steps: int, warmup: int):
    """Exactly `steps` steps replayed from graphs (after `warmup` eager steps); returns ms per step."""
    import torch
    for i in range(warmup):
        setup.step(i)
    # Graphs of a whole number of rotations and, for single-layer steps, at least 32 steps, so that one replay's
    # launch is spread over many steps (a stack step is long enough by itself).
    per = setup.rotate * (max(1, math.ceil(32 / setup.rotate)) if setup.layer_steps == 1 else 1)
    full, tail = divmod(steps, per)
    g_full = _capture(setup, 0, per) if full else None
    g_tail = _capture(setup, 0, tail) if tail else None
    if g_full is not None:
        g_full.replay()
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(full):
        g_full.replay()
    if g_tail is not None:
        g_tail.replay()
    end.record()
    torch.cuda.synchronize()
    return start.elapsed_time(end) / steps


def time_step_distribution(setup, blocks: int = 40):
    """Per-step times: graphs of `block` consecutive steps (8 for a single layer, whose step is tens of
    microseconds, so that one graph launch and one pair of events are spread over 8 steps; 1 for a stack), each of
    `blocks` replays between two events, all queued behind a spin kernel so that they run back to back.  Returns
    (median, p10, p90) of the per-step mean of each block in microseconds, and the block length."""
    import torch
    block = 8 if setup.layer_steps == 1 else 1
    n_graphs = max(1, setup.rotate // block) if setup.rotate % block == 0 else setup.rotate
    graphs = [_capture(setup, j * block, block) for j in range(n_graphs)]
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(blocks)]
    torch.cuda.synchronize()
    torch.cuda._sleep(int(2e6) * max(1, blocks // 4))
    for i, (a, b) in enumerate(evs):
        a.record()
        graphs[i % n_graphs].replay()
        b.record()
    torch.cuda.synchronize()
    us = np.array([a.elapsed_time(b) for a, b in evs]) * 1e3 / block
    del graphs
    return float(np.median(us)), float(np.percentile(us, 10)), float(np.percentile(us, 90)), block


def time_compaction(setup, reps: int = 64) -> float:
    """Microseconds per call of the step's mask compaction alone (rm_mask_compact of its masks), from a graph of
    `reps` calls replayed a few times."""
    import torch
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        setup.compact()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(reps):
            setup.compact()
    g.replay()
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(4):
        g.replay()
    end.record()
    torch.cuda.synchronize()
    return start.elapsed_time(end) * 1e3 / (4 * reps)


def stream_read_gbs(device, gib: int = 2, reps: int = 8) -> dict:
    """Bandwidth of a plain streaming read (rm_stream_read) of a `gib` GiB buffer on this GPU: the best of a few
    grid sizes, each the median of `reps` timed reads (every read is cold: the buffer is 8x the Infinity Cache)."""
    import torch
    import paper_2609_19104_amd as rm
    buf = torch.empty(gib << 30, dtype=torch.uint8, device=device)
    best = None
    for wg in (1024, 2048, 4096, 8192):
        sink = torch.empty(wg * 512, dtype=torch.int32, device=device)
        rm.rm_stream_read(buf, wg, sink)
        torch.cuda.synchronize()
        times = []
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            rm.rm_stream_read(buf, wg, sink)
            b.record()
            torch.cuda.synchronize()
            times.append(a.elapsed_time(b))
        gbs = buf.numel() / (float(np.median(times)) * 1e-3) / 1e9
        if best is None or gbs > best["gbs"]:
            best = {"gbs": round(gbs, 1), "workgroups": wg}
    del buf
    torch.cuda.empty_cache()
    best["bytes"] = gib << 30
    return best


def secondary_lines(device, steps: int, warmup: int) -> dict:
    """Per-layer figures of configurations 2, 3 and 5, one graph-replayed timing each (cold weights)."""
    import torch
    out = {}
    for key, cls in (("c2", Setup), ("c3", StackSetup3), ("c5", StackSetup5)):
        setup = cls(key, device, cold=True)
        ms = time_graph(setup, steps, warmup)
        gbs = setup.active_bytes / (ms * 1e-3) / 1e9
        line = {"workload": setup.spec["name"], "us_per_layer": round(ms * 1e3 / setup.layer_steps, 3),
                "gbs_active": round(gbs, 1), "pct_of_peak": round(100.0 * gbs / HBM_PEAK_GBS, 2),
                "compaction_us": round(time_compaction(setup), 3)}
        if isinstance(setup, Setup):
            setup.lists = False
            line["masked_us_per_layer"] = round(time_graph(setup, steps, warmup) * 1e3, 3)
        if isinstance(setup, StackSetup5):
            line["per_sample_gbs"] = round(setup.per_sample_bytes / (ms * 1e-3) / 1e9, 1)
            line["mfma_frac"] = round(setup.useful_flops() / (ms * 1e-3) / (BF16_PEAK_TFLOPS * 1e12), 4)
        out[key] = line
        del setup
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
    return out


def _code_only(text: str) -> str:
    """C/C++ source without its comments and trailing blanks (string and character literals kept), so that an
    edit of comments alone leaves the digest below unchanged."""
    out, i, n = [], 0, len(text)
    while i < n:
        c = text[i]
        if c in "\"'":  # a literal: copied through, escapes included
            j = i + 1
            while j < n and text[j] != c:
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        elif text.startswith("//", i):
            j = text.find("\n", i)
            i = n if j < 0 else j
        elif text.startswith("/*", i):
            j = text.find("*/", i + 2)
            i = n if j < 0 else j + 2
        else:
            out.append(c)
            i += 1
    return "\n".join(line.rstrip() for line in "".join(out).split("\n") if line.strip())


def kernel_source_digest() -> str:
    """sha256 over the HIP sources' code (names and code without comments, files sorted): identifies the kernels
    a counter run measured."""
    import hashlib
    h = hashlib.sha256()
    for name in sorted(os.listdir(CSRC)):
        if name.endswith((".hip", ".h")):
            h.update(name.encode())
            with open(os.path.join(CSRC, name), encoding="utf-8") as f:
                h.update(_code_only(f.read()).encode())
    return h.hexdigest()


def counted_traffic(workload: str, kernel_key: str):
    """HBM bytes per launch of a kernel from the committed rocprofv3 counter summary of this workload
    (FETCH_SIZE and WRITE_SIZE, each scaled by what the counter reads for a plain copy of known size), or None
    when there is no summary or the kernels have changed since it was taken."""
    path = os.path.join(PROFILES, f"pmc_traffic_{workload}.md")
    if not os.path.exists(path):
        return None
    fields = {}
    with open(path) as f:
        for line in f:
            if line.startswith("- ") and ": " in line:
                k, v = line[2:].strip().split(": ", 1)
                fields[k.strip("`")] = v.strip().strip("`")
    if fields.get("kernel_source_sha256") != kernel_source_digest():
        return None
    v = fields.get(f"traffic_bytes_per_launch.{kernel_key}")
    return int(float(v)) if v else None


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(setup: Setup, seconds: float):
    """The float64 oracle on the same layer, mask and input, repeated for about `seconds` of CPU time with the
    BLAS threads it gets by default (all the cores it may use), then for about a quarter of that on one thread.
    Each figure uses the median time per evaluation."""
    import oracle

    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        threads = max([p.get("num_threads", 1) for p in threadpool_info() if p.get("user_api") == "blas"] or [1])
    except Exception:  # threadpoolctl missing: report the affinity size NumPy's BLAS defaults to
        threadpool_limits = None
        threads = len(os.sched_getaffinity(0))
    wg, wu, wd, g = setup.layer_np.f64()
    mult = setup.mask.cpu().numpy()[0].astype(np.float64)
    x = setup.x.cpu().numpy()[0]

    def run(budget: float):
        oracle.masked_ffn(x, wg, wu, wd, mult, g)  # warm
        times, t0 = [], time.perf_counter()
        while True:
            t = time.perf_counter()
            oracle.masked_ffn(x, wg, wu, wd, mult, g)
            times.append(time.perf_counter() - t)
            el = time.perf_counter() - t0
            if el >= budget and len(times) >= 5:
                return float(np.median(times)), len(times), el

    per, reps, el = run(seconds)
    out = {"value": round(setup.active_bytes / per / 1e9, 4), "unit": "GB/s", "cores": int(threads),
           "kind": "oracle", "cpu_model": _cpu_model(),
           "sample": f"{reps} float64 oracle evaluations of the same layer (dense SwiGLU over all {setup.d_ff} "
                     f"neurons, inactive ones zeroed) on the same input and mask, {el:.1f} s; median "
                     f"{per * 1e3:.2f} ms per layer; value = active weight bytes / median oracle time"}
    if threadpool_limits is not None:
        with threadpool_limits(limits=1):
            per1, reps1, _ = run(seconds / 4)
        out["single_thread"] = {"value": round(setup.active_bytes / per1 / 1e9, 4), "unit": "GB/s",
                                "ms_per_layer": round(per1 * 1e3, 2), "evaluations": reps1}
    return out


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="c4-30", choices=sorted(WORKLOADS))
    ap.add_argument("--no-secondary", action="store_true",
                    help="skip the per-layer figures of configurations 2, 3 and 5 (default workload only)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--profile-only", action="store_true",
                    help="run warmup + steps with no event hooks and no CPU leg (for rocprofv3)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run `steps` device-to-device copies of MIB MiB (the plain copy kernel whose "
                         "FETCH_SIZE / WRITE_SIZE counters scale the hot path's)")
    args = ap.parse_args(argv)

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: the library has no multi-GPU path "
              "(the hot path would shard by sample, with no communication between GPUs).", file=sys.stderr)
        return 2

    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    dev = torch.device("cuda:0")
    if args.copy_calibration:
        n = args.copy_calibration << 20
        src = torch.ones(n // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": n, "copies": args.steps}))
        return 0
    setup = {"c3": StackSetup3, "c3-eq4": StackSetupEq4, "c3-eq4-compact": StackSetupEq4Compact, "c5": StackSetup5,
             "gm": GroupMaskSetup, "cc": ContextSetup}.get(
        args.workload, Setup)(
        args.workload, dev, cold=True)

    if args.profile_only:
        time_graph(setup, args.steps, args.warmup)
        print(json.dumps({"profile_only": True, "workload": args.workload, "steps": args.steps}))
        return 0

    eager_ms, _ = time_steps(setup, args.steps, args.warmup)
    _, kern = time_steps(setup, args.steps, 5, hook=True)
    ms = time_graph(setup, args.steps, args.warmup)
    # The dominant kernel: the hooked kernel with the longest average launch duration (kernel start to end).
    hooks = setup.hooks()
    dom_id, dom, dom_key, dom_bytes = max(hooks, key=lambda h: kern[h[0]]["mean"])[:4]
    dom_us = kern[dom_id]["mean"]
    bound = getattr(setup, "bound", "hbm")
    if bound == "mfma":  # the dominant kernel's amount is FLOPs: matrix-core roofline
        achieved, peak, unit = dom_bytes / (dom_us * 1e-6) / 1e12, BF16_PEAK_TFLOPS, "TFLOP/s"
    else:
        achieved, peak, unit = dom_bytes / (dom_us * 1e-6) / 1e9, HBM_PEAK_GBS, "GB/s"
    value = setup.active_bytes / (ms * 1e-3) / 1e9

    step_med, step_p10, step_p90, step_block = time_step_distribution(setup)
    compact_us = time_compaction(setup) if hasattr(setup, "compact") else None
    masked_ms = None
    if isinstance(setup, Setup):  # the same step with the compaction of its mask (rm_masked_ffn_layer)
        setup.lists = False
        masked_ms = time_graph(setup, args.steps, args.warmup)
        setup.lists = True

    setup.rotate = 1
    warm_ms = time_graph(setup, args.steps, args.warmup)
    setup.rotate = setup.copies
    stream = stream_read_gbs(dev)

    out = {
        "metric": "µs per sparse FFN layer + achieved HBM GB/s (% of peak) on active weights",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": setup.spec["name"], "d": setup.d, "d_ff": setup.d_ff, "T": setup.T, "B": setup.B,
                   "active_neurons": setup.k, "layers": setup.L,
                   "step": STEP_TEXT.get(setup.key, STEP_TEXT[setup.key[:2]]),
                   "weights": getattr(setup, "cold_text", None) or
                              f"cold: {setup.copies} rotating copies "
                              f"({setup.copies * setup.L * 3 * setup.d * setup.d_ff * 2 / 2**30:.2f} GiB)"},
        "us_per_layer": round(ms * 1e3 / setup.layer_steps, 3),
        "eager_us_per_layer": round(eager_ms * 1e3 / setup.layer_steps, 3),
        "pct_of_peak": round(100.0 * value / HBM_PEAK_GBS, 2),
        "tokens_per_s": round(setup.B * setup.T * setup.layer_steps / (ms * 1e-3), 1),
        "active_weight_bytes": setup.active_bytes,
        "warm_us_per_layer": round(warm_ms * 1e3 / setup.layer_steps, 3),
        "step_us": {"median": round(step_med, 3), "p10": round(step_p10, 3), "p90": round(step_p90, 3),
                    "how": f"40 graph replays of {step_block} consecutive step(s), each between two events and "
                           f"divided by {step_block}, queued back to back"},
        "compaction_us": None if compact_us is None else round(compact_us, 3),
        "masked_us_per_layer": None if masked_ms is None else round(masked_ms * 1e3, 3),
        "stream_read": {"gbs": stream["gbs"], "workgroups": stream["workgroups"], "bytes": stream["bytes"],
                        "pct_of_peak": round(100.0 * stream["gbs"] / HBM_PEAK_GBS, 2),
                        "kernel": "rm_stream_read (plain streaming read, 16 B per lane, 8 loads in flight)"},
        "pct_of_stream_read": round(100.0 * value / stream["gbs"], 2),
        "kernel_us": {f"{key}{suffix}": round(kern[kid][stat], 3) for kid, _, key, _ in hooks
                      for suffix, stat in (("", "mean"), ("_median", "median"), ("_min", "min"), ("_p10", "p10"),
                                           ("_p90", "p90"))},
        "roofline": {"bound": bound, "kernel": dom, "achieved": round(achieved, 2), "peak": peak,
                     "unit": unit, "frac": round(achieved / peak, 4),
                     "traffic": counted_traffic(args.workload, dom_key),
                     ("flops_per_launch" if bound == "mfma" else "bytes_per_launch"): dom_bytes,
                     "avg_launch_us": round(dom_us, 3),
                     "traffic_unit": "bytes per launch (HBM, from rocprofv3 counters)"},
    }
    if isinstance(setup, StackSetup5):
        out["per_sample_weight_bytes"] = setup.per_sample_bytes
        out["per_sample_value"] = round(setup.per_sample_bytes / (ms * 1e-3) / 1e9, 2)
        out["mfma_frac"] = round(setup.useful_flops() / (ms * 1e-3) / (BF16_PEAK_TFLOPS * 1e12), 4)
    if isinstance(setup, GroupMaskSetup):
        out["coverage"] = setup.coverage()
    if not args.no_cpu_baseline and isinstance(setup, Setup):
        out["cpu_baseline"] = cpu_baseline(setup, args.cpu_seconds)
    if args.workload == ap.get_default("workload") and not args.no_secondary:
        del setup
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        out["secondary"] = secondary_lines(dev, args.steps, args.warmup)
    print(json.dumps(out))
    return 0


if __name__ == "__main__":
    sys.exit(main())
