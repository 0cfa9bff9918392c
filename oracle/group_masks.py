"""Plain CPU oracle for building a group's neuron masks from reference activations (paper section 5,
"Constructing Group Neuron Masks", with Eq. 1's contribution score from section 3.4).

TEST INFRASTRUCTURE.  Only the tests, the smoke check and the benchmark's CPU-baseline leg may import this
module.  It shares no code with the GPU library and never calls it.

What is computed, per layer l of a group of S denoising steps:

1. Eq. 1: c[s, n] = (sum over the T actions of |h[s, n, t]|) * ||W_down[n]||_2 for every neuron n and step s.
2. Each step's candidates: the K neurons with the highest c[s, :].
3. The group's mask: among the union of the steps' candidates, the K neurons with the highest summed
   contribution sum_s c[s, n].

Selecting the top K is an integer decision taken on floating-point scores, so this oracle fixes the precision
and the order of every sum to those of the GPU kernels: float32, each sum taken in index order one rounded
addition at a time (|h| over t = 0 .. T-1; w^2 over columns j = 0 .. d-1, each square rounded before it is
added; the steps' scores over s = 0 .. S-1), the norm a correctly rounded float32 square root and the score a
rounded float32 product.  Ties in a ranking go to the lower neuron index.  (The paper leaves the precision
open; it does not affect which neurons are meant, only how ties at the K-th place fall.)
"""
from __future__ import annotations

import numpy as np

F32 = np.float32


def neuron_norms(w_down: np.ndarray) -> np.ndarray:
    """||W_down[n]||_2 for every neuron (the weight factor of Eq. 1), float32, columns summed in order."""
    w = np.asarray(w_down, dtype=F32)
    s = np.zeros(w.shape[0], dtype=F32)
    for j in range(w.shape[1]):
        s = (s + (w[:, j] * w[:, j]).astype(F32)).astype(F32)
    return np.sqrt(s).astype(F32)


def contribution_scores(h: np.ndarray, norms: np.ndarray) -> np.ndarray:
    """Eq. 1 for one step and layer: h float32 [d_ff][T] (neuron-major) -> c float32 [d_ff]."""
    h = np.asarray(h, dtype=F32)
    s = np.zeros(h.shape[0], dtype=F32)
    for t in range(h.shape[1]):
        s = (s + np.abs(h[:, t])).astype(F32)
    return (s * np.asarray(norms, dtype=F32)).astype(F32)


def top_k(score: np.ndarray, k: int, eligible: np.ndarray | None = None) -> np.ndarray:
    """Boolean selection of the k highest scores (among the eligible ones), ties to the lower index."""
    n = score.shape[0]
    idx = np.arange(n) if eligible is None else np.flatnonzero(eligible)
    order = sorted(idx.tolist(), key=lambda i: (-float(score[i]), i))
    sel = np.zeros(n, dtype=bool)
    sel[order[:max(0, k)]] = True
    return sel


def group_mask(h_steps: np.ndarray, norms: np.ndarray, k: int) -> np.ndarray:
    """One layer's group mask (section 5): h_steps float32 [S][d_ff][T] -> uint8 [d_ff]."""
    c = [contribution_scores(h, norms) for h in h_steps]
    union = np.zeros(c[0].shape[0], dtype=bool)
    summed = np.zeros(c[0].shape[0], dtype=F32)
    for cs in c:
        union |= top_k(cs, k)
        summed = (summed + cs).astype(F32)
    return top_k(summed, k, eligible=union).astype(np.uint8)


def group_masks(h: np.ndarray, norms: np.ndarray, k: int) -> np.ndarray:
    """All layers: h float32 [S][L][d_ff][T], norms float32 [L][d_ff] -> uint8 [L][d_ff]."""
    h = np.asarray(h, dtype=F32)
    return np.stack([group_mask(h[:, l], norms[l], k) for l in range(h.shape[1])])


def coverage(score: np.ndarray, mask: np.ndarray) -> float:
    """Share of a step's total contribution captured by a mask (section 3.4's coverage)."""
    score = np.asarray(score, dtype=np.float64)
    tot = float(score.sum())
    return float(score[np.asarray(mask) != 0].sum()) / tot if tot > 0 else 0.0
