"""Plain CPU oracle for the Context Cache's visual-token recomputation (paper section 4.1, "Visual-Token
Recomputation": Eq. 2 and Eq. 3).

TEST INFRASTRUCTURE.  Only the tests, the smoke check and the benchmark's CPU-baseline leg may import this
module.  It shares no code with the GPU library and never calls it.

What is computed for one VLM FFN layer over a sequence of N tokens whose visual tokens are rows [v0, v0 + P):

1. Eq. 2, per visual token p: d_p = RMS(x_p - xbar_p) / max(RMS(x_p), eps), eps = 1e-6, with x the current FFN
   input and xbar the reference execution's input of the same token.  Float64 on exact widenings of the stored
   float32 inputs, with RMS(v) = sqrt(mean(v^2)).
2. The recomputed rows: the ceil(rho_p P) visual tokens with the largest d_p (ties to the lower token), plus all
   rows outside the visual range (the rows of the text instruction and of the robot state, which the method never
   takes from the cache).
3. Eq. 3: y_hat_p = F(x_p) for recomputed rows and the reference output ybar_p for the others, F being the FFN
   (gate, up, activation, down; no norm inside, no residual).  Float64.

The selection is an integer decision on real-valued scores.  A float32 implementation can order two rows whose
float64 drifts lie within its rounding error either way, so `drift_rel_bound` states how far any float32
evaluation of Eq. 2 may lie from the float64 value, whatever its summation order; the tests accept any top-k that
is consistent with that bound.
"""
from __future__ import annotations

import numpy as np

from .ffn import ACTIVATIONS

EPS = 1e-6
U32 = 2.0 ** -24  # unit roundoff of float32


def drift(x: np.ndarray, x_ref: np.ndarray) -> np.ndarray:
    """Eq. 2 for every row of x ([P][d]) against x_ref, float64 [P]."""
    x = np.asarray(x, dtype=np.float64)
    xr = np.asarray(x_ref, dtype=np.float64)
    diff = x - xr
    rms_diff = np.sqrt(np.mean(diff * diff, axis=1))
    rms_x = np.sqrt(np.mean(x * x, axis=1))
    return rms_diff / np.maximum(rms_x, EPS)


def drift_rel_bound(d: int) -> float:
    """Relative distance from the float64 Eq. 2 value within which every float32 evaluation lies, for any order of
    the two sums of d squares.

    Each squared term carries at most 3 roundings (the difference, the square; the plain x^2 only one), and a
    float32 sum of d non-negative terms in any order is within gamma_(d-1) = (d-1)u / (1 - (d-1)u) of the exact
    sum (Higham, Accuracy and Stability of Numerical Algorithms, Thm. 4.4 with non-negative terms), so each sum is
    within gamma_(d+2).  The mean adds one rounding, the square root halves the relative error and adds one, and the
    quotient of the two RMS values adds the two relative errors and one more rounding.  The result is doubled as a
    safety margin and stays far below the spread of distinct drifts in the workloads (about 1e-4 at d = 2048)."""
    n = d + 2
    g = n * U32 / (1.0 - n * U32)
    per_rms = (g + U32) / 2.0 + U32
    return 2.0 * (2.0 * per_rms + U32)


def recomputed_rows(scores: np.ndarray, n_tokens: int, v0: int, k: int) -> np.ndarray:
    """Ascending int32 rows to recompute: every row outside [v0, v0 + P) and the k visual rows with the largest
    scores (P = len(scores)), ties to the lower token."""
    P = len(scores)
    order = sorted(range(P), key=lambda p: (-float(scores[p]), p))
    chosen = set(v0 + p for p in order[:max(0, k)])
    rows = [r for r in range(n_tokens) if r < v0 or r >= v0 + P or r in chosen]
    return np.asarray(rows, dtype=np.int32)


def check_recomputed_rows(rows: np.ndarray, drift64: np.ndarray, n_tokens: int, v0: int, k: int, rel: float) -> None:
    """Raises AssertionError unless `rows` is a valid Eq. 2 selection given drifts known to within relative `rel`:
    ascending and distinct, every non-visual row present, exactly k visual rows, and no dropped visual row whose
    drift exceeds a chosen one's by more than the two values' rounding allowance.  Among rows of exactly equal
    float64 drift that are exactly representable and equal in any evaluation (zero drift), the lower token wins."""
    rows = np.asarray(rows, dtype=np.int64)
    P = len(drift64)
    assert rows.ndim == 1 and len(rows) == n_tokens - P + k, (len(rows), n_tokens - P + k)
    assert np.all(np.diff(rows) > 0), "rows must be ascending and distinct"
    assert rows.size == 0 or (rows[0] >= 0 and rows[-1] < n_tokens)
    non_visual = np.concatenate([np.arange(0, v0), np.arange(v0 + P, n_tokens)])
    assert np.all(np.isin(non_visual, rows)), "every instruction / state row is recomputed"
    vis = rows[(rows >= v0) & (rows < v0 + P)] - v0
    assert len(vis) == k
    chosen = np.zeros(P, dtype=bool)
    chosen[vis] = True
    if 0 < k < P:
        lo_chosen = float(np.min(drift64[chosen] * (1.0 + rel)))
        hi_dropped = float(np.max(drift64[~chosen] * (1.0 - rel)))
        assert lo_chosen >= hi_dropped, (lo_chosen, hi_dropped)
        zero = drift64 == 0.0
        if np.any(zero & chosen) and np.any(zero & ~chosen):
            assert np.max(np.flatnonzero(zero & chosen)) < np.min(np.flatnonzero(zero & ~chosen)), "zero-drift tie"


def ffn_out(x: np.ndarray, w_gate: np.ndarray, w_up: np.ndarray, w_down_t: np.ndarray, act: str = "gelu_tanh"):
    """F(x) = (act(x W_gate^T) * (x W_up^T)) W_down, float64; w_down_t is [d][d_ff] (nn.Linear's down weight)."""
    x = np.asarray(x, dtype=np.float64)
    h = ACTIVATIONS[act](x @ np.asarray(w_gate, np.float64).T) * (x @ np.asarray(w_up, np.float64).T)
    return h @ np.asarray(w_down_t, np.float64).T


def context_update(x: np.ndarray, y_ref: np.ndarray, rows: np.ndarray, w_gate, w_up, w_down_t,
                   act: str = "gelu_tanh") -> np.ndarray:
    """Eq. 3: y_ref with the listed rows replaced by F(x) of those rows."""
    out = np.array(y_ref, dtype=np.float64)
    rows = np.asarray(rows)
    if rows.size:
        out[rows] = ffn_out(np.asarray(x)[rows], w_gate, w_up, w_down_t, act)
    return out
