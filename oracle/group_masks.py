"""Plain CPU oracle for building a group's neuron masks from reference activations (paper section 5,
"Constructing Group Neuron Masks", with Eq. 1's contribution score from section 3.4).

TEST INFRASTRUCTURE.  Only the tests, the smoke check and the benchmark's CPU-baseline leg may import this
module.  It shares no code with the GPU library and never calls it.

What is computed, per layer l of a group of S denoising steps, in float64 on exact widenings of the inputs:

1. Eq. 1: c[s, n] = (sum over the T actions of |h[s, n, t]|) * ||W_down[n]||_2 for every neuron n and step s.
2. Each step's candidates: the K neurons with the highest c[s, :].
3. The group's mask: among the union of the steps' candidates, the K neurons with the highest summed
   contribution sum_s c[s, n].

Ties in a ranking go to the lower neuron index.  A float32 implementation may order two neurons whose float64
scores lie within its rounding error either way; `score_rel_bound` states that error for any summation order and
`check_group_mask` accepts every mask consistent with it.
"""
from __future__ import annotations

import numpy as np

U32 = 2.0 ** -24  # unit roundoff of float32


def _gamma(n: int) -> float:
    """Higham's gamma_n = n u / (1 - n u): the relative error bound of a float32 sum of n + 1 non-negative terms
    in any order (Accuracy and Stability of Numerical Algorithms, Thm. 4.4)."""
    return n * U32 / (1.0 - n * U32)


def neuron_norms(w_down: np.ndarray) -> np.ndarray:
    """||W_down[n]||_2 for every neuron (the weight factor of Eq. 1): square root of the row's sum of squares."""
    w = np.asarray(w_down, dtype=np.float64)
    return np.sqrt(np.sum(w * w, axis=1))


def norm_rel_bound(d: int) -> float:
    """Relative distance from the float64 norm within which any float32 evaluation lies: the d squares (one
    rounding each) summed in any order, a square root (half the relative error, one rounding); doubled."""
    return 2.0 * ((_gamma(d - 1) + U32) / 2.0 + U32)


def contribution_scores(h: np.ndarray, norms: np.ndarray) -> np.ndarray:
    """Eq. 1 for one step and layer: h [d_ff][T] (neuron-major) -> c float64 [d_ff]."""
    h = np.asarray(h, dtype=np.float64)
    return np.sum(np.abs(h), axis=1) * np.asarray(norms, dtype=np.float64)


def score_rel_bound(T: int, norm_rel: float = 0.0) -> float:
    """Relative distance from the float64 Eq. 1 score within which a float32 score lies, given float32 norms
    within `norm_rel` of their true values (0 when the norms are exact inputs): the sum of T absolute values in
    any order, the product; doubled."""
    return 2.0 * (_gamma(max(T - 1, 0)) + norm_rel + U32)


def top_k(score: np.ndarray, k: int, eligible: np.ndarray | None = None) -> np.ndarray:
    """Boolean selection of the k highest scores (among the eligible ones), ties to the lower index."""
    n = score.shape[0]
    idx = np.arange(n) if eligible is None else np.flatnonzero(eligible)
    order = sorted(idx.tolist(), key=lambda i: (-float(score[i]), i))
    sel = np.zeros(n, dtype=bool)
    sel[order[:max(0, k)]] = True
    return sel


def group_mask(h_steps: np.ndarray, norms: np.ndarray, k: int) -> np.ndarray:
    """One layer's group mask (section 5): h_steps [S][d_ff][T] -> uint8 [d_ff]."""
    c = [contribution_scores(h, norms) for h in h_steps]
    union = np.zeros(c[0].shape[0], dtype=bool)
    for cs in c:
        union |= top_k(cs, k)
    summed = np.sum(np.stack(c), axis=0)
    return top_k(summed, k, eligible=union).astype(np.uint8)


def group_masks(h: np.ndarray, norms: np.ndarray, k: int) -> np.ndarray:
    """All layers: h [S][L][d_ff][T], norms [L][d_ff] -> uint8 [L][d_ff]."""
    h = np.asarray(h, dtype=np.float64)
    return np.stack([group_mask(h[:, l], norms[l], k) for l in range(h.shape[1])])


def check_group_mask(mask: np.ndarray, c_steps: np.ndarray, k: int, rel: float) -> None:
    """Raises AssertionError unless `mask` is a valid section-5 group mask for float64 step scores c_steps
    [S][d_ff] known to within relative `rel` (the summed score then within rel as well, plus the float32 sum over
    the S steps):

    - exactly k neurons;
    - each one is a possible candidate: in some step its score is not below that step's k-th best by more than
      the two values' allowance;
    - no neuron that is certainly some step's candidate (above that step's (k+1)-th best by more than the
      allowance) and was left out has a summed score above a chosen neuron's by more than the allowance."""
    mask = np.asarray(mask) != 0
    c = np.asarray(c_steps, dtype=np.float64)
    S, n = c.shape
    assert int(mask.sum()) == k, (int(mask.sum()), k)
    if k == 0 or k == n:
        return
    lo, hi = 1.0 - rel, 1.0 + rel
    possible = np.zeros(n, dtype=bool)
    certain = np.zeros(n, dtype=bool)
    for s in range(S):
        srt = np.sort(c[s])[::-1]
        kth, next_ = srt[k - 1], srt[k]
        possible |= c[s] * hi >= kth * lo
        certain |= c[s] * lo > next_ * hi
    assert np.all(possible[mask]), np.flatnonzero(mask & ~possible)[:8]
    rel_sum = rel + _gamma(max(S - 1, 0))
    summed = c.sum(axis=0)
    out = certain & ~mask
    if np.any(out):
        assert float(np.min(summed[mask])) * (1.0 + rel_sum) >= float(np.max(summed[out])) * (1.0 - rel_sum)


def coverage(score: np.ndarray, mask: np.ndarray) -> float:
    """Share of a step's total contribution captured by a mask (section 3.4's coverage)."""
    score = np.asarray(score, dtype=np.float64)
    tot = float(score.sum())
    return float(score[np.asarray(mask) != 0].sum()) / tot if tot > 0 else 0.0
