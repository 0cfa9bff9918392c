"""Helpers of the GPU tests: move seeded inputs to the device and run the library through its binding.

Nothing here computes the FFN: results come from the HIP library and expected values from the oracle."""
from __future__ import annotations

import numpy as np
import torch

import paper_2609_19104_amd as rm
import workloads as wl

DEV = torch.device("cuda:0")
TOL_BF16 = 2e-2
TOL_F32 = 1e-5
STORE_U = 2.0 ** -24  # unit roundoff of the float32 output store


def dev_weights(layer: wl.Layer):
    def w(a):
        if a.dtype == np.uint16:
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(DEV)
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)

    g = None if layer.norm_g is None else torch.from_numpy(layer.norm_g).to(DEV)
    return (w(layer.w_gate), w(layer.w_up), w(layer.w_down), g)


def dev_f32(a) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)


def compact(masks: np.ndarray):
    """masks uint8 [N][d_ff] -> (idx, count) device tensors via rm_mask_compact."""
    m = torch.from_numpy(np.ascontiguousarray(masks, dtype=np.uint8)).to(DEV)
    n, d_ff = m.shape
    idx = torch.full((n, d_ff), 12345, dtype=torch.int32, device=DEV)
    cnt = torch.full((n,), -7, dtype=torch.int32, device=DEV)
    rm.rm_mask_compact(m, idx, cnt)
    return idx, cnt


def run_layer(layer_dev, x: np.ndarray, idx: torch.Tensor, cnt: torch.Tensor, max_count: int,
              in_place: bool = False) -> np.ndarray:
    wg = layer_dev[0]
    d_ff, d = wg.shape
    B, T, _ = x.shape
    xt = dev_f32(x)
    yt = xt if in_place else torch.full_like(xt, float("nan"))
    ws = rm.workspace(d, d_ff, rm.wdtype_of(wg), B, T, max_count, device=DEV)
    ws.fill_(0xFF)  # NaN in every float32 / bf16 slot: stale workspace read into a result shows
    rm.rm_sparse_ffn_layer(xt, yt, layer_dev, idx, cnt, max_count, ws)
    torch.cuda.synchronize()
    return yt.cpu().numpy()


def run_dense(layer_dev, x: np.ndarray) -> np.ndarray:
    wg = layer_dev[0]
    d_ff, d = wg.shape
    B, T, _ = x.shape
    xt = dev_f32(x)
    yt = torch.full_like(xt, float("nan"))
    ws = rm.workspace(d, d_ff, rm.wdtype_of(wg), B, T, d_ff, device=DEV)
    ws.fill_(0x7F)  # about 3.4e38 in every float32 and bf16 slot
    rm.rm_dense_ffn_ref(xt, yt, layer_dev, ws)
    torch.cuda.synchronize()
    return yt.cpu().numpy()


def run_stack(layers_dev, x: np.ndarray, idx: torch.Tensor, cnt: torch.Tensor, max_count: int) -> np.ndarray:
    wg = layers_dev[0][0]
    d_ff, d = wg.shape
    B, T, _ = x.shape
    xt = dev_f32(x)
    yt = torch.full_like(xt, float("nan"))
    ws = rm.workspace(d, d_ff, rm.wdtype_of(wg), B, T, max_count, device=DEV)
    ws.fill_(0xFF)
    rm.rm_sparse_ffn_stack(xt, yt, layers_dev, idx, cnt, max_count, ws)
    torch.cuda.synchronize()
    return yt.cpu().numpy()


def errors(y: np.ndarray, y_ref: np.ndarray, x: np.ndarray):
    """(relative error of y, relative error of the FFN delta y - x), both max-abs / max-abs.

    y is returned in float32, so each element carries up to u |y| of rounding from its final store
    (u = 2^-24), whatever the kernel did.  When the delta is small next to x that store alone exceeds a tight
    relative bound on the delta, so the delta error counts only what lies beyond it.
    """
    import oracle

    y = np.asarray(y, np.float64)
    x = np.asarray(x, np.float64)
    y_ref = np.asarray(y_ref, np.float64)
    d_ref = y_ref - x
    den = float(np.max(np.abs(d_ref))) if d_ref.size else 0.0
    excess = np.maximum(np.abs(y - y_ref) - STORE_U * np.abs(y_ref), 0.0)
    num = float(np.max(excess)) if excess.size else 0.0
    ed = (0.0 if num == 0.0 else float("inf")) if den == 0.0 else num / den
    return oracle.rel_err(y, y_ref), ed


H_SENTINEL = -12345.0  # h_anchor entries past a list's count must keep it


def run_anchor(layers_dev, x: np.ndarray, idx: torch.Tensor, cnt: torch.Tensor, max_count: int):
    """Eq. 4 anchor step through rm_anchor_ffn_stack -> (y, y_anchor [L][B][T][d], h_anchor [L][B][max_count][T])
    as device tensors (the anchor state stays on the device for the delta steps)."""
    wg = layers_dev[0][0]
    d_ff, d = wg.shape
    B, T, _ = x.shape
    L = len(layers_dev)
    xt = dev_f32(x)
    yt = torch.full_like(xt, float("nan"))
    ya = torch.full((L, B, T, d), float("nan"), dtype=torch.float32, device=DEV)
    ha = torch.full((L, B, max_count, T), H_SENTINEL, dtype=torch.float32, device=DEV)
    ws = rm.workspace(d, d_ff, rm.wdtype_of(wg), B, T, d_ff, device=DEV)
    ws.fill_(0x7F)
    rm.rm_anchor_ffn_stack(xt, yt, layers_dev, idx, cnt, max_count, ya, ha, ws)
    torch.cuda.synchronize()
    return yt, ya, ha


def run_delta(layers_dev, x: np.ndarray, idx: torch.Tensor, cnt: torch.Tensor, max_count: int,
              ya: torch.Tensor, ha: torch.Tensor) -> np.ndarray:
    """Eq. 4 non-anchor step through rm_delta_ffn_stack."""
    wg = layers_dev[0][0]
    d_ff, d = wg.shape
    B, T, _ = x.shape
    xt = dev_f32(x)
    yt = torch.full_like(xt, float("nan"))
    ws = rm.workspace(d, d_ff, rm.wdtype_of(wg), B, T, max_count, device=DEV)
    ws.fill_(0xFF)
    rm.rm_delta_ffn_stack(xt, yt, layers_dev, idx, cnt, max_count, ya, ha, ws)
    torch.cuda.synchronize()
    return yt.cpu().numpy()
