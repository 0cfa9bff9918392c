"""GPU parity of the GeGLU activation (GELU-tanh) and the adaptive output gate against the float64 oracle, on
every path that applies them: the split-K epilogue, the fused down projection (one-sample stacks), the epilogue
inside a stack, and Eq. 4's anchor and delta steps (whose gates may differ, y_a being kept before the gate).

Bars: max-abs relative error 2e-2 (bf16 weights) or 1e-5 (float32 weights) on y and the FFN part y - x; an empty
list gives y == x bit for bit whatever the gate; a delta step at the anchor's own input and gates reproduces
the anchor's y bit for bit."""
import numpy as np
import pytest
import torch

import oracle
import workloads as wl

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2609_19104_amd as rm  # noqa: E402
from gpu_helpers import TOL_BF16, TOL_F32, compact, dev_f32, dev_weights, errors  # noqa: E402


def _gates(seed, L, B, d):
    r = np.random.default_rng(seed)
    return [(1.0 + 0.5 * r.standard_normal((B, d))).astype(np.float32) for _ in range(L)]


def _dev_layers(layers, gates):
    return [dev_weights(l) + (dev_f32(g),) for l, g in zip(layers, gates)]


def _oracle_stack(x, layers, masks, gates, act):
    lay = [l.f64() for l in layers]
    return np.stack([oracle.ffn_stack(x[b], lay, [m[b].astype(np.float64) for m in masks], act=act,
                                      gates=[g[b] for g in gates]) for b in range(x.shape[0])])


CASES = [
    # d, d_ff, L, B, T, k, wdtype, act
    (256, 1000, 1, 2, 51, 333, "bf16", "gelu_tanh"),   # one layer: split-K down + epilogue
    (256, 1000, 1, 2, 51, 333, "bf16", "silu"),
    (1024, 4096, 3, 1, 51, 1229, "bf16", "gelu_tanh"),  # one sample: fused down, xn for the next layer
    (160, 512, 2, 3, 17, 200, "bf16", "gelu_tanh"),     # stack with the epilogue emitting xn
    (2048, 8192, 2, 1, 51, 3000, "bf16", "gelu_tanh"),  # one sample's long list: gate/up and down in one launch
    (1024, 4096, 1, 1, 51, 1229, "bf16", "gelu_tanh"),  # a single d = 1024 layer: the one-launch form too
    (128, 300, 2, 2, 9, 150, "f32", "gelu_tanh"),
    (64, 100, 1, 1, 3, 37, "f32", "silu"),
]


@pytest.mark.parametrize("d,d_ff,L,B,T,k,wdtype,act", CASES)
def test_gated_layers_parity(d, d_ff, L, B, T, k, wdtype, act):
    tol = TOL_BF16 if wdtype == "bf16" else TOL_F32
    layers = [wl.make_layer(101, l, d, d_ff, wdtype, norm="random") for l in range(L)]
    gates = _gates(102, L, B, d)
    x = wl.make_x(101, (B, T, d), d_ff, T)
    masks = [np.stack([wl.uniform_mask(wl.rng(101, 4, l, b), d_ff, k - 20 * b) for b in range(B)])
             for l in range(L)]
    idx, cnt = compact(np.concatenate(masks))
    lws = _dev_layers(layers, gates)
    xt = dev_f32(x)
    y = torch.full_like(xt, float("nan"))
    ws = rm.workspace(d, d_ff, rm.wdtype_of(lws[0][0]), B, T, k)
    if L == 1:
        rm.rm_sparse_ffn_layer(xt, y, lws[0], idx, cnt, k, ws, act=act)
    else:
        rm.rm_sparse_ffn_stack(xt, y, lws, idx, cnt, k, ws, act=act)
    torch.cuda.synchronize()
    ey, ed = errors(y.cpu().numpy(), _oracle_stack(x, layers, masks, gates, act), x)
    print(f"{act} {wdtype} {d}x{d_ff} L={L} B={B}: y {ey:.2e} FFN part {ed:.2e}")
    assert ey <= tol and ed <= tol


@pytest.mark.parametrize("B", [1, 2])
def test_gate_with_empty_list_is_identity(B):
    d, d_ff, L, T = 256, 512, 2, 20
    layers = [wl.make_layer(103, l, d, d_ff, "bf16", norm="random") for l in range(L)]
    lws = _dev_layers(layers, _gates(104, L, B, d))
    x = wl.make_x(103, (B, T, d), 0)
    x[0, 0, :5] = -0.0
    idx, cnt = compact(np.zeros((L * B, d_ff), np.uint8))
    xt = dev_f32(x)
    y = torch.full_like(xt, float("nan"))
    rm.rm_sparse_ffn_stack(xt, y, lws, idx, cnt, 64, rm.workspace(d, d_ff, rm.RM_BF16, B, T, 64), act="gelu_tanh")
    torch.cuda.synchronize()
    assert np.array_equal(y.cpu().numpy().view(np.uint32), x.view(np.uint32))


@pytest.mark.parametrize("d,d_ff,L,B,T,k", [(1024, 4096, 2, 1, 51, 1229), (256, 512, 3, 2, 33, 200),
                                             (2048, 8192, 2, 1, 51, 3000)])
def test_gated_geglu_anchor_and_delta(d, d_ff, L, B, T, k):
    layers = [wl.make_layer(105, l, d, d_ff, "bf16", norm="random") for l in range(L)]
    ga, gt = _gates(106, L, B, d), _gates(107, L, B, d)  # the anchor step's and a later step's gates
    xa = wl.make_x(105, (B, T, d), d_ff, T)
    xt = (xa + 0.05 * np.random.default_rng(108).standard_normal(xa.shape)).astype(np.float32)
    masks = np.stack([np.stack([wl.uniform_mask(wl.rng(105, 4, l, b), d_ff, k) for b in range(B)])
                      for l in range(L)])
    idx, cnt = compact(masks.reshape(L * B, d_ff))
    la, lt = _dev_layers(layers, ga), _dev_layers(layers, gt)
    xat, xtt = dev_f32(xa), dev_f32(xt)
    ya_dev = torch.empty((L, B, T, d), device="cuda")
    ha_dev = torch.empty((L, B, k, T), device="cuda")
    y_anchor = torch.empty_like(xat)
    ws_dense = rm.workspace(d, d_ff, rm.RM_BF16, B, T, d_ff)
    rm.rm_anchor_ffn_stack(xat, y_anchor, la, idx, cnt, k, ya_dev, ha_dev, ws_dense, act="gelu_tanh")
    ws = rm.workspace(d, d_ff, rm.RM_BF16, B, T, k)
    y = torch.empty_like(xtt)
    rm.rm_delta_ffn_stack(xtt, y, lt, idx, cnt, k, ya_dev, ha_dev, ws, act="gelu_tanh")
    y_same = torch.empty_like(xat)
    rm.rm_delta_ffn_stack(xat, y_same, la, idx, cnt, k, ya_dev, ha_dev, ws, act="gelu_tanh")
    torch.cuda.synchronize()
    lay = [l.f64() for l in layers]
    ref_a, ref_ya, ref_ha, ref_t = [], [], [], []
    for b in range(B):
        yb, yab, hab = oracle.anchor_stack(xa[b], lay, act="gelu_tanh", gates=[g[b] for g in ga])
        ref_a.append(yb)
        ref_t.append(oracle.delta_stack(xt[b], lay, [m[b].astype(np.float64) for m in masks], yab, hab,
                                        act="gelu_tanh", gates=[g[b] for g in gt]))
    ey, ed = errors(y_anchor.cpu().numpy(), np.stack(ref_a), xa)
    assert ey <= TOL_BF16 and ed <= TOL_BF16, ("anchor", ey, ed)
    ey, ed = errors(y.cpu().numpy(), np.stack(ref_t), xt)
    assert ey <= TOL_BF16 and ed <= TOL_BF16, ("delta", ey, ed)
    assert np.array_equal(y_same.cpu().numpy().view(np.uint32), y_anchor.cpu().numpy().view(np.uint32))
