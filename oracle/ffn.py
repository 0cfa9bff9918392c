"""Plain float64 CPU oracle for the Action Cache sparse-FFN hot path.

TEST INFRASTRUCTURE.  Only the tests, the smoke check and the benchmark's CPU-baseline leg may import this
module.  The GPU library never calls it, and it shares no code with the GPU path.

What is computed (the paper's Action Cache, section 4.1):

* Each intermediate neuron n of a SwiGLU FFN has gate and up rows W_gate[n], W_up[n] and a down-projection row
  W_down[n] (the row-vector form of the down projection in Eq. 4, which multiplies h^M by W^down_M).
* A cached mask M names the neurons to recompute.  The masked FFN keeps every neuron's activation
  h[t,n] = SiLU(<W_gate[n], xn_t>) * <W_up[n], xn_t> for n in M and zeroes the rest:
  y = x + (h * 1_M) W_down.  It is Eq. 4 with a zero anchor (y_a = 0, h_a = 0).
* The oracle evaluates it as a *dense* FFN over all d_ff neurons whose inactive neurons are then zeroed, the
  plain definition, not the gathered form the GPU path uses.

All arithmetic is float64 on exact widenings of the stored float32 / bfloat16 inputs.
"""
from __future__ import annotations

import math
from typing import Optional, Sequence

import numpy as np

RMS_EPS = 1e-6


def silu(z: np.ndarray) -> np.ndarray:
    """SiLU(z) = z * sigmoid(z) = z / (1 + exp(-z)), the SwiGLU gate activation.

    Written in two branches so that exp never overflows: for z < 0, z * e^z / (1 + e^z).
    """
    z = np.asarray(z, dtype=np.float64)
    out = np.empty_like(z)
    pos = z >= 0
    out[pos] = z[pos] / (1.0 + np.exp(-z[pos]))
    ez = np.exp(z[~pos])
    out[~pos] = z[~pos] * ez / (1.0 + ez)
    return out


def gelu_tanh(z: np.ndarray) -> np.ndarray:
    """GELU in its tanh form, 0.5 z (1 + tanh(sqrt(2/pi) (z + 0.044715 z^3))), the gate activation of a GeGLU FFN
    (section 3.4 names the scored activations post-GeGLU)."""
    z = np.asarray(z, dtype=np.float64)
    return 0.5 * z * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (z + 0.044715 * z * z * z)))


ACTIVATIONS = {"silu": silu, "gelu_tanh": gelu_tanh}


def rms_norm(x: np.ndarray, g: np.ndarray, eps: float = RMS_EPS) -> np.ndarray:
    """RMSNorm over the last axis: x / sqrt(mean(x^2) + eps) * g.

    The paper names the FFN input after normalization but gives no action-expert formula; the eps of 1e-6 is the
    only one it states (Eq. 2's denominator guard).
    """
    x = np.asarray(x, dtype=np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(g, dtype=np.float64)


def compact_mask(masks: np.ndarray):
    """Mask -> ascending active-neuron index list (the indices stored with a reference, section 4.1).

    masks: [N][d_ff] (or [d_ff]) of any integer type, nonzero = active.
    Returns (idx, count): idx int32 [N][d_ff] holds the active positions in ascending order in its first
    count[n] entries and -1 after them; count int32 [N].
    """
    m = np.asarray(masks)
    squeeze = m.ndim == 1
    m = m.reshape(-1, m.shape[-1])
    n, d_ff = m.shape
    idx = np.full((n, d_ff), -1, dtype=np.int32)
    count = np.zeros(n, dtype=np.int32)
    for i in range(n):
        act = np.flatnonzero(m[i] != 0)
        idx[i, : act.size] = act
        count[i] = act.size
    if squeeze:
        return idx[0], count[0]
    return idx, count


def multiplicity(idx: np.ndarray, count: int, d_ff: int) -> np.ndarray:
    """How often each neuron appears in idx[:count] (a list is a multiset; a compacted mask gives 0/1)."""
    sel = np.asarray(idx[:count], dtype=np.int64)
    if sel.size and (sel.min() < 0 or sel.max() >= d_ff):
        raise ValueError("index out of range")
    return np.bincount(sel, minlength=d_ff).astype(np.float64)


def mask_multiplicity(mask: np.ndarray) -> np.ndarray:
    return (np.asarray(mask) != 0).astype(np.float64)


def ffn_input(x: np.ndarray, norm_g: Optional[np.ndarray], eps: float = RMS_EPS) -> np.ndarray:
    x = np.asarray(x, dtype=np.float64)
    return x if norm_g is None else rms_norm(x, norm_g, eps)


def hidden(x: np.ndarray, w_gate: np.ndarray, w_up: np.ndarray, norm_g: Optional[np.ndarray] = None,
           eps: float = RMS_EPS, act: str = "silu") -> np.ndarray:
    """Dense post-GLU activations h[t,n] = act(xn_t . W_gate[n]) * (xn_t . W_up[n]) for every neuron
    (act = SiLU for SwiGLU, GELU-tanh for GeGLU)."""
    xn = ffn_input(x, norm_g, eps)
    return ACTIVATIONS[act](xn @ np.asarray(w_gate, np.float64).T) * (xn @ np.asarray(w_up, np.float64).T)


def _gated(f: np.ndarray, gate: Optional[np.ndarray]) -> np.ndarray:
    """The adaptive output gate (section 4.1: the FFN output goes through the model's adaptive gate before the
    residual addition): f * gate, gate broadcast over tokens ([d] per sample), or f without a gate."""
    return f if gate is None else f * np.asarray(gate, np.float64)


def masked_ffn(x: np.ndarray, w_gate: np.ndarray, w_up: np.ndarray, w_down: np.ndarray, mult: np.ndarray,
               norm_g: Optional[np.ndarray] = None, eps: float = RMS_EPS, act: str = "silu",
               gate: Optional[np.ndarray] = None) -> np.ndarray:
    """y = x + gate * ((h * mult) W_down): the dense FFN with inactive neurons zeroed, plus the residual.

    x: [T][d] (any leading batch axes); weights [d_ff][d]; mult [d_ff] (0/1 for a mask, counts for a multiset);
    gate: [d] (or None).  The residual adds the un-normalized x (pre-norm block).  Eq. 4 with y_a = 0, h_a = 0.
    """
    x64 = np.asarray(x, dtype=np.float64)
    h = hidden(x64, w_gate, w_up, norm_g, eps, act) * np.asarray(mult, np.float64)
    return x64 + _gated(h @ np.asarray(w_down, np.float64), gate)


def dense_ffn(x, w_gate, w_up, w_down, norm_g=None, eps: float = RMS_EPS, act: str = "silu",
              gate=None) -> np.ndarray:
    """Dense GLU FFN + residual (the anchor step, section 4.1): every neuron active."""
    return masked_ffn(x, w_gate, w_up, w_down, np.ones(np.asarray(w_gate).shape[0]), norm_g, eps, act, gate)


def ffn_stack(x: np.ndarray, layers: Sequence[tuple], mults: Sequence[np.ndarray], eps: float = RMS_EPS,
              return_all: bool = False, act: str = "silu", gates: Optional[Sequence] = None):
    """Apply layers in order, feeding each layer's output to the next.

    layers: sequence of (w_gate, w_up, w_down, norm_g) float64 tuples; mults: one multiplicity per layer;
    gates: one output gate ([d] or None) per layer, or None.
    """
    y = np.asarray(x, dtype=np.float64)
    outs = []
    for l, ((wg, wu, wd, g), m) in enumerate(zip(layers, mults)):
        y = masked_ffn(y, wg, wu, wd, m, g, eps, act, None if gates is None else gates[l])
        outs.append(y)
    return outs if return_all else y


def local_update(y_anchor: np.ndarray, h_t: np.ndarray, h_anchor: np.ndarray, mult: np.ndarray,
                 w_down: np.ndarray) -> np.ndarray:
    """Eq. 4: y_hat = y_a + (h_t^M - h_a^M) W^down_M, with h restricted to the mask by mult.

    y_anchor: the anchor step's FFN output; h_t, h_anchor: dense activations [T][d_ff] of the current step and
    of the anchor step.  Only the masked neurons' difference is applied; the anchor's contribution of every
    other neuron stays in y_a.
    """
    dh = (np.asarray(h_t, np.float64) - np.asarray(h_anchor, np.float64)) * np.asarray(mult, np.float64)
    return np.asarray(y_anchor, np.float64) + dh @ np.asarray(w_down, np.float64)


def anchor_stack(x: np.ndarray, layers: Sequence[tuple], eps: float = RMS_EPS, act: str = "silu",
                 gates: Optional[Sequence] = None):
    """The anchor step of a group (section 4.1, "Anchors with Mask Recomputation"): the dense layers in order.

    Returns (y, y_a, h_a): the last layer's output, and per layer the dense FFN output before the adaptive gate
    and the residual (y_a, [L][..][T][d]) and the dense activations (h_a, [L][..][T][d_ff]) that the group's
    later steps reuse.
    """
    y = np.asarray(x, dtype=np.float64)
    ya, ha = [], []
    for l, (wg, wu, wd, g) in enumerate(layers):
        h = hidden(y, wg, wu, g, eps, act)
        f = h @ np.asarray(wd, np.float64)
        ya.append(f)
        ha.append(h)
        y = y + _gated(f, None if gates is None else gates[l])
    return y, np.stack(ya), np.stack(ha)


def delta_stack(x: np.ndarray, layers: Sequence[tuple], mults: Sequence[np.ndarray], y_anchor: np.ndarray,
                h_anchor: np.ndarray, eps: float = RMS_EPS, act: str = "silu",
                gates: Optional[Sequence] = None) -> np.ndarray:
    """A non-anchor step of the group: at each layer the FFN output is Eq. 4's estimate from the anchor's y_a and
    h_a (as returned by anchor_stack) and this step's activations of the masked neurons, then the adaptive gate
    of this step and the residual addition; layer l reads layer l-1's output.
    """
    y = np.asarray(x, dtype=np.float64)
    for l, ((wg, wu, wd, g), m) in enumerate(zip(layers, mults)):
        h_t = hidden(y, wg, wu, g, eps, act)
        y = y + _gated(local_update(y_anchor[l], h_t, h_anchor[l], m, wd), None if gates is None else gates[l])
    return y


# ----------------------------------------------------------------------------------------------------------
# Picking masks by activation score (test-input preparation)
# ----------------------------------------------------------------------------------------------------------

def mean_abs_activation(x, w_gate, w_up, norm_g=None, eps: float = RMS_EPS) -> np.ndarray:
    """Score of neuron n: mean over tokens of |h[t,n]|, on a reference execution's input.

    This is the score the test masks are picked by.  The paper's own score (Eq. 1) also multiplies by the norm
    of the neuron's down-projection row; see contribution_score.
    """
    h = hidden(np.asarray(x, np.float64).reshape(-1, np.asarray(x).shape[-1]), w_gate, w_up, norm_g, eps)
    return np.mean(np.abs(h), axis=0)


def contribution_score(h: np.ndarray, w_down: np.ndarray) -> np.ndarray:
    """Eq. 1: c_n = (sum over actions r of |h[r,n]|) * ||W_down[n]||_2."""
    h = np.asarray(h, np.float64)
    return np.sum(np.abs(h), axis=0) * np.sqrt(np.sum(np.asarray(w_down, np.float64) ** 2, axis=1))


def topk_mask(score: np.ndarray, k: int) -> np.ndarray:
    """uint8 mask of the k highest scores; ties go to the lower neuron index (stable order)."""
    score = np.asarray(score, dtype=np.float64)
    order = np.argsort(-score, kind="stable")
    m = np.zeros(score.shape[0], dtype=np.uint8)
    m[order[:k]] = 1
    return m


def nested_topk_masks(score: np.ndarray, ks: Sequence[int]) -> np.ndarray:
    """One mask per k from a single ranking, so each smaller mask is contained in each larger one."""
    return np.stack([topk_mask(score, k) for k in ks])


def ceil_budget(rho_num: int, rho_den: int, n: int) -> int:
    """K_l = ceil(rho_n * H_l), section 5 ("Constructing Group Neuron Masks"), with rho = rho_num / rho_den."""
    return -((-rho_num * n) // rho_den)


def rel_err(a: np.ndarray, ref: np.ndarray) -> float:
    """max |a - ref| / max |ref| (0 when both are all zero)."""
    a = np.asarray(a, np.float64)
    ref = np.asarray(ref, np.float64)
    den = float(np.max(np.abs(ref))) if ref.size else 0.0
    num = float(np.max(np.abs(a - ref))) if ref.size else 0.0
    if den == 0.0:
        return 0.0 if num == 0.0 else math.inf
    return num / den


def stack_masks_from_dense(x: np.ndarray, layers: Sequence[tuple], k: int, eps: float = RMS_EPS) -> np.ndarray:
    """Per-layer masks from a dense reference execution of a stack (test-input preparation).

    Runs the dense stack on x; at layer l the mask keeps the k neurons with the largest mean |h| on that
    layer's input.  Returns uint8 [L][d_ff].
    """
    y = np.asarray(x, dtype=np.float64).reshape(-1, np.asarray(x).shape[-1])
    masks = []
    for wg, wu, wd, g in layers:
        masks.append(topk_mask(mean_abs_activation(y, wg, wu, g, eps), k))
        y = dense_ffn(y, wg, wu, wd, g, eps)
    return np.stack(masks)
