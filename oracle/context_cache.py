"""Plain CPU oracle for the Context Cache's visual-token recomputation (paper section 4.1, "Visual-Token
Recomputation": Eq. 2 and Eq. 3).

TEST INFRASTRUCTURE.  Only the tests, the smoke check and the benchmark's CPU-baseline leg may import this
module.  It shares no code with the GPU library and never calls it.

What is computed for one VLM FFN layer over a sequence of N tokens whose visual tokens are rows [v0, v0 + P):

1. Eq. 2, per visual token p: d_p = RMS(x_p - xbar_p) / max(RMS(x_p), eps), eps = 1e-6, with x the current FFN
   input (after RMSNorm) and xbar the reference execution's.
2. The recomputed rows: the ceil(rho_p P) visual tokens with the largest d_p (ties to the lower token), and every
   non-visual row (instruction and robot-state rows are always recomputed).
3. Eq. 3: y_hat_p = F(x_p) for recomputed rows and the reference output ybar_p for the others, F being the FFN
   (gate, up, activation, down; no norm inside, no residual).

The selection is an integer decision on floating-point scores, so the drift is computed in float32 in the
GPU's fixed order: per row, lane j of 64 adds (x - xbar)^2 (and x^2) of columns j, j + 64, j + 128, ... one
rounding per operation, the 64 lane sums are then folded in halves (32, 16, 8, 4, 2, 1 apart); RMS = sqrt(sum /
d) with a rounded division and a correctly rounded square root; d_p = RMS_diff / max(RMS_x, 1e-6) rounded once.
The FFN itself is float64 on exact widenings of the stored inputs.
"""
from __future__ import annotations

import numpy as np

from .ffn import ACTIVATIONS

F32 = np.float32
EPS = F32(1e-6)


def _row_sumsq(v: np.ndarray) -> np.ndarray:
    """float32 sum of squares of each row in the fixed order described above.  v: float32 [rows][d]."""
    rows, d = v.shape
    lanes = np.zeros((rows, 64), dtype=F32)
    for c0 in range(0, d, 64):
        blk = v[:, c0:c0 + 64]
        sq = (blk * blk).astype(F32)
        lanes[:, :sq.shape[1]] = (lanes[:, :sq.shape[1]] + sq).astype(F32)
    width = 64
    while width > 1:
        width //= 2
        lanes = (lanes[:, :width] + lanes[:, width:2 * width]).astype(F32)
    return lanes[:, 0]


def drift(x: np.ndarray, x_ref: np.ndarray) -> np.ndarray:
    """Eq. 2 for every row of x (float32 [P][d]) against x_ref, float32 [P]."""
    x = np.asarray(x, dtype=F32)
    xr = np.asarray(x_ref, dtype=F32)
    d = F32(x.shape[1])
    diff = (x - xr).astype(F32)
    rms_diff = np.sqrt((_row_sumsq(diff) / d).astype(F32)).astype(F32)
    rms_x = np.sqrt((_row_sumsq(x) / d).astype(F32)).astype(F32)
    return (rms_diff / np.maximum(rms_x, EPS)).astype(F32)


def recomputed_rows(scores: np.ndarray, n_tokens: int, v0: int, k: int) -> np.ndarray:
    """Ascending int32 rows to recompute: every row outside [v0, v0 + P) and the k visual rows with the largest
    scores (P = len(scores)), ties to the lower token."""
    P = len(scores)
    order = sorted(range(P), key=lambda p: (-float(scores[p]), p))
    chosen = set(v0 + p for p in order[:max(0, k)])
    rows = [r for r in range(n_tokens) if r < v0 or r >= v0 + P or r in chosen]
    return np.asarray(rows, dtype=np.int32)


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
