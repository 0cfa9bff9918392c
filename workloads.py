"""Seeded synthetic inputs for the Action Cache sparse-FFN workloads.

This module draws random numbers and lays out shapes. It holds none of the FFN's arithmetic: no norm, no
activation, no products, no neuron scoring. The tests, the benchmark and the oracle's callers all take their
inputs from here, so the GPU path and the oracle see the same bits while sharing no computation.

Value recipe (the shapes and distributions of a pi0-style action expert; the paper's trained checkpoints and
robot suites are not used, these stand in for them):

* weights ~ N(0, 0.02), drawn in float64, stored as float32 or as bfloat16 (round to nearest even);
* activations x ~ N(0, 1) in float32, one [T][d] tile per sample;
* neuron counts K = ceil(rho * d_ff), the per-layer budget of the paper's group-mask construction (section 5,
  "Constructing Group Neuron Masks");
* masks are uint8 per neuron, nonzero = active.  Masks picked by activation score are not built here (that
  needs the FFN); callers build them and pass them in.

Every stream of numbers comes from ``numpy.random.SeedSequence([2609, 19104, cfg, *path])`` so that each
tensor can be regenerated on its own, in any order.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

SEED_ROOT = (2609, 19104)
WEIGHT_STD = 0.02

# Stream tags used in SeedSequence paths (kept stable: changing one changes every generated input).
_TAG_W = 1
_TAG_X = 2
_TAG_NOISE = 3
_TAG_MASK = 4
_TAG_GAIN = 5
_TAG_ACT = 6


def seed_sequence(cfg: int, *path: int) -> np.random.SeedSequence:
    return np.random.SeedSequence([*SEED_ROOT, int(cfg), *[int(p) for p in path]])


def rng(cfg: int, *path: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed_sequence(cfg, *path)))


# ----------------------------------------------------------------------------------------------------------
# Storage formats
# ----------------------------------------------------------------------------------------------------------

def bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float values to bfloat16 (nearest, ties to even) and return the raw uint16 bit patterns."""
    u = np.ascontiguousarray(np.asarray(a, dtype=np.float32)).view(np.uint32).astype(np.uint64)
    if np.any((u & 0x7F800000) == 0x7F800000):
        raise ValueError("bf16_bits: non-finite input")
    lsb = (u >> 16) & 1
    return ((u + 0x7FFF + lsb) >> 16).astype(np.uint16)


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float64."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def storage_to_f64(a: np.ndarray) -> np.ndarray:
    """Exact float64 value of a stored weight array (uint16 = bfloat16 bits, float32 otherwise)."""
    if a.dtype == np.uint16:
        return bf16_bits_to_f64(a)
    return np.asarray(a, dtype=np.float64)


def count_for_percent(percent: int, d_ff: int) -> int:
    """K = ceil(percent/100 * d_ff), in exact integer arithmetic."""
    return (int(percent) * int(d_ff) + 99) // 100


# ----------------------------------------------------------------------------------------------------------
# Layers and activations
# ----------------------------------------------------------------------------------------------------------

@dataclass
class Layer:
    """One SwiGLU FFN layer's weights, in the storage the GPU path reads.

    w_gate, w_up, w_down: [d_ff][d]; row n belongs to intermediate neuron n.  w_down row n is that neuron's
    down-projection weight vector (the row-vector form of the down projection used by Eq. 4), i.e. the transpose
    of a PyTorch ``down_proj.weight`` of shape [d][d_ff].  dtype uint16 = bfloat16 bits, else float32.
    norm_g: [d] float32 RMSNorm gain applied to the FFN input, or None for no norm.
    """
    w_gate: np.ndarray
    w_up: np.ndarray
    w_down: np.ndarray
    norm_g: Optional[np.ndarray] = None

    @property
    def d(self) -> int:
        return int(self.w_gate.shape[1])

    @property
    def d_ff(self) -> int:
        return int(self.w_gate.shape[0])

    @property
    def wdtype(self) -> str:
        return "bf16" if self.w_gate.dtype == np.uint16 else "f32"

    def f64(self):
        """(w_gate, w_up, w_down, norm_g) as exact float64 arrays."""
        g = None if self.norm_g is None else np.asarray(self.norm_g, dtype=np.float64)
        return (storage_to_f64(self.w_gate), storage_to_f64(self.w_up), storage_to_f64(self.w_down), g)


def _store(a64: np.ndarray, wdtype: str) -> np.ndarray:
    if wdtype == "bf16":
        return bf16_bits(a64)
    if wdtype == "f32":
        return np.ascontiguousarray(a64, dtype=np.float32)
    raise ValueError(f"unknown weight dtype {wdtype!r}")


def make_layer(cfg: int, layer: int, d: int, d_ff: int, wdtype: str, *, norm: str = "none",
               std: float = WEIGHT_STD) -> Layer:
    """Seeded weights of one layer.  norm: "none", "ones" (gain 1) or "random" (gain ~ 1 + 0.1 N(0,1))."""
    ws = []
    for which in range(3):  # gate, up, down
        r = rng(cfg, _TAG_W, layer, which)
        ws.append(_store(r.standard_normal((d_ff, d)) * std, wdtype))
    g = None
    if norm == "ones":
        g = np.ones(d, dtype=np.float32)
    elif norm == "random":
        g = (1.0 + 0.1 * rng(cfg, _TAG_GAIN, layer).standard_normal(d)).astype(np.float32)
    elif norm != "none":
        raise ValueError(norm)
    return Layer(ws[0], ws[1], ws[2], g)


def make_x(cfg: int, shape: Sequence[int], *path: int, scale: float = 1.0) -> np.ndarray:
    """float32 N(0, scale^2) activations."""
    return (rng(cfg, _TAG_X, *path).standard_normal(tuple(shape)) * scale).astype(np.float32)


def make_noise(cfg: int, shape: Sequence[int], *path: int, scale: float) -> np.ndarray:
    """float64 N(0, scale^2) perturbation (added to an activation tile, then stored as float32)."""
    return rng(cfg, _TAG_NOISE, *path).standard_normal(tuple(shape)) * scale


def perturb(x: np.ndarray, noise: np.ndarray) -> np.ndarray:
    """x + noise, stored as float32 (input drift between a reference execution and the current one)."""
    return (np.asarray(x, dtype=np.float64) + noise).astype(np.float32)


# ----------------------------------------------------------------------------------------------------------
# Random masks (those that need no activation score)
# ----------------------------------------------------------------------------------------------------------

def uniform_mask(r: np.random.Generator, d_ff: int, k: int) -> np.ndarray:
    """Exactly k distinct active neurons, drawn uniformly without replacement."""
    m = np.zeros(d_ff, dtype=np.uint8)
    m[r.choice(d_ff, size=k, replace=False)] = 1
    return m


def core_plus_random_masks(r: np.random.Generator, d_ff: int, batch: int, k_core: int, k_rest: int) -> np.ndarray:
    """[batch][d_ff] masks sharing one core of k_core neurons, each with k_rest more drawn from the rest."""
    core = r.choice(d_ff, size=k_core, replace=False)
    others = np.setdiff1d(np.arange(d_ff), core)
    out = np.zeros((batch, d_ff), dtype=np.uint8)
    out[:, core] = 1
    for b in range(batch):
        out[b, r.choice(others, size=k_rest, replace=False)] = 1
    return out


def bernoulli_mask(r: np.random.Generator, shape: Sequence[int], p: float) -> np.ndarray:
    return (r.random(tuple(shape)) < p).astype(np.uint8)


# ----------------------------------------------------------------------------------------------------------
# The five workloads (shapes from a pi0-style action expert; see the module docstring)
# ----------------------------------------------------------------------------------------------------------

@dataclass
class Workload:
    """Inputs of one configuration.  Fields unused by a config stay empty.

    layers: per-layer weights.  x: the input the FFN is evaluated on, [B][T][d] float32 (configs 3 uses
    x_steps instead).  x_ref: the reference execution's input that score-based masks are picked on.
    masks: [L][B][d_ff] uint8 when they need no activation score (configs 1 and 5), else None.
    k: active neurons per mask (one value; config 4 uses ks).
    """
    cfg: int
    name: str
    d: int
    d_ff: int
    T: int
    B: int
    wdtype: str
    layers: List[Layer]
    x: Optional[np.ndarray] = None
    x_ref: Optional[np.ndarray] = None
    x_steps: Optional[List[np.ndarray]] = None
    masks: Optional[np.ndarray] = None
    k: int = 0
    ks: List[int] = field(default_factory=list)
    percents: List[int] = field(default_factory=list)
    steps: int = 1
    refresh_steps: List[int] = field(default_factory=list)

    @property
    def L(self) -> int:
        return len(self.layers)


def config1(d: int = 256, d_ff: int = 1024, T: int = 8) -> Workload:
    """Single fp32 SwiGLU layer; mask = uniform-random 25% of the neurons (exactly ceil(0.25 d_ff))."""
    cfg = 1
    k = count_for_percent(25, d_ff)
    layer = make_layer(cfg, 0, d, d_ff, "f32")
    x = make_x(cfg, (1, T, d), 0)
    masks = uniform_mask(rng(cfg, _TAG_MASK, 0), d_ff, k)[None, None, :]
    return Workload(cfg, "single fp32 SwiGLU layer", d, d_ff, T, 1, "f32", [layer], x=x, masks=masks, k=k)


def config2(d: int = 1024, d_ff: int = 4096, T: int = 51) -> Workload:
    """One pi0-style action-expert layer, bf16; mask picked on x_ref, evaluated on x = x_ref + 0.1 N(0,1)."""
    cfg = 2
    layer = make_layer(cfg, 0, d, d_ff, "bf16")
    x_ref = make_x(cfg, (1, T, d), 0)
    x = perturb(x_ref, make_noise(cfg, x_ref.shape, 0, scale=0.1))
    return Workload(cfg, "pi0 action-expert FFN layer", d, d_ff, T, 1, "bf16", [layer], x=x, x_ref=x_ref,
                    k=count_for_percent(30, d_ff))


def config3(L: int = 18, d: int = 1024, d_ff: int = 4096, T: int = 51, steps: int = 10) -> Workload:
    """18-layer stack with RMSNorm; 10 denoising steps with inputs drifting by 0.05 N(0,1) per step.

    Step 0 is dense; the masks are refreshed at steps 1, 3, 5, 7, 9 (from the dense activations of the previous
    step's input) and shared by that step and the next.
    """
    cfg = 3
    layers = [make_layer(cfg, l, d, d_ff, "bf16", norm="ones") for l in range(L)]
    xs = [make_x(cfg, (1, T, d), 0)]
    for s in range(1, steps):
        xs.append(perturb(xs[-1], make_noise(cfg, xs[-1].shape, s, scale=0.05)))
    return Workload(cfg, "action-expert FFN stack", d, d_ff, T, 1, "bf16", layers, x_steps=xs,
                    k=count_for_percent(30, d_ff), steps=steps, refresh_steps=list(range(1, steps, 2)))


def activation_like(cfg: int, shape: Sequence[int], *path: int, quantum: float = 0.0) -> np.ndarray:
    """float32 stand-ins for post-GLU activations h[..][n][t] (neuron-major rows): standard normal values scaled
    per neuron by a lognormal factor (a few neurons carry most of the magnitude, as in section 3.4's coverage
    curve).  quantum > 0 rounds every value to a multiple of it, which makes equal scores (ties) common."""
    r = rng(cfg, _TAG_ACT, *path)
    h = r.standard_normal(tuple(shape))
    scale = np.exp(r.standard_normal(tuple(shape[:-1]) + (1,)))
    h = h * scale
    if quantum > 0:
        h = np.round(h / quantum) * quantum
    return h.astype(np.float32)


def positive_norms(cfg: int, shape: Sequence[int], *path: int) -> np.ndarray:
    """float32 stand-ins for down-projection row norms: 0.5 .. 1.5."""
    return (0.5 + rng(cfg, _TAG_ACT, 1, *path).random(tuple(shape))).astype(np.float32)


@dataclass
class ContextWorkload:
    """One VLM FFN layer of the Context Cache (section 4.1, "Visual-Token Recomputation"): n_tok token rows, the
    visual tokens in rows [v0, v0 + P), the current FFN inputs x and the reference execution's x_ref and y_ref
    (all float32 [n_tok][d]), bf16 weights with the down projection in nn.Linear's [d][d_ff] layout, and k visual
    rows to recompute."""
    d: int
    d_ff: int
    n_tok: int
    v0: int
    P: int
    k: int
    layer: Layer
    w_down_t: np.ndarray
    x: np.ndarray
    x_ref: np.ndarray
    y_ref: np.ndarray


def context_workload(n_tok: int = 850, v0: int = 0, P: int = 768, d: int = 2048, d_ff: int = 16384,
                     rho_num: int = 2, rho_den: int = 5, seed: int = 6) -> ContextWorkload:
    """The VLM prefill FFN of a pi0.5-style model (d = 2048, d_ff = 16384; 3 camera views x 256 visual tokens
    first, then 82 instruction and state rows: 850 rows as in Table 1), rho_p = 0.4 (the paper's default).  x_ref
    is N(0, 1) (a normalized input); x drifts from it by a per-token scale drawn lognormally, so that a minority
    of tokens carries most of the change; y_ref is N(0, 0.1^2)."""
    layer = make_layer(seed, 0, d, d_ff, "bf16")
    x_ref = make_x(seed, (n_tok, d), 1)
    r = rng(seed, _TAG_NOISE, 7)
    scale = 0.05 * np.exp(1.5 * r.standard_normal((n_tok, 1)))
    x = (x_ref + scale * r.standard_normal((n_tok, d))).astype(np.float32)
    y_ref = (0.1 * rng(seed, _TAG_X, 2).standard_normal((n_tok, d))).astype(np.float32)
    k = -(-rho_num * P // rho_den)
    return ContextWorkload(d, d_ff, n_tok, v0, P, k, layer, np.ascontiguousarray(layer.w_down.T), x, x_ref, y_ref)


def group_reference_inputs(w: Workload, anchors: Sequence[int], scale: float = 0.1) -> List[np.ndarray]:
    """For the anchored schedule on a config-3 stack: per group, a similar execution's input (the group's anchor
    input + scale N(0,1)) on which the group's masks are scored (section 4.1 takes them from a reference)."""
    return [perturb(w.x_steps[a], make_noise(w.cfg, w.x_steps[a].shape, 100 + g, scale=scale))
            for g, a in enumerate(anchors)]


def config4(d: int = 2048, d_ff: int = 16384, T: int = 51, percents: Sequence[int] = (10, 30, 50, 100)) -> Workload:
    """Wide FFN density sweep; nested top-k masks of one score vector computed on x_ref."""
    cfg = 4
    layer = make_layer(cfg, 0, d, d_ff, "bf16")
    x_ref = make_x(cfg, (1, T, d), 0)
    x = perturb(x_ref, make_noise(cfg, x_ref.shape, 0, scale=0.1))
    return Workload(cfg, "wide FFN density sweep", d, d_ff, T, 1, "bf16", [layer], x=x, x_ref=x_ref,
                    ks=[count_for_percent(p, d_ff) for p in percents], percents=list(percents))


def config5(B: int = 16, L: int = 18, d: int = 1024, d_ff: int = 4096, T: int = 51,
            core_percent: int = 18, percent: int = 30) -> Workload:
    """B independent sequences, each with its own per-layer mask: a shared core plus a random remainder."""
    cfg = 5
    layers = [make_layer(cfg, l, d, d_ff, "bf16", norm="ones") for l in range(L)]
    x = make_x(cfg, (B, T, d), 0)
    k = count_for_percent(percent, d_ff)
    k_core = count_for_percent(core_percent, d_ff)
    masks = np.stack([core_plus_random_masks(rng(cfg, _TAG_MASK, l), d_ff, B, k_core, k - k_core)
                      for l in range(L)])
    return Workload(cfg, "batched ragged executions", d, d_ff, T, B, "bf16", layers, x=x, masks=masks, k=k)


def ragged_masks(cfg: int, d_ff: int, counts: Sequence[int], *path: int) -> np.ndarray:
    """[len(counts)][d_ff] uniform masks with the given exact counts (for ragged-batch tests)."""
    r = rng(cfg, _TAG_MASK, 99, *path)
    return np.stack([uniform_mask(r, d_ff, int(c)) for c in counts])
