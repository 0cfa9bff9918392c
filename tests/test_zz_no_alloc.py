"""GPU test of rm_sparse_ffn_layer_noalloc, the layer entry point that allocates nothing (it takes its
workspace from a per-device array inside the library): three calls in a row on one GPU, each with a smaller
input than the one before (the first at d = 2048 with a list long enough for the one-launch layer form), each checked bit for bit against rm_sparse_ffn_layer with a caller workspace (the same kernels) and
against the float64 oracle within the bf16 / float32 tolerances."""
import numpy as np
import pytest
import torch

import oracle
import workloads as wl

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2609_19104_amd as rm  # noqa: E402
from gpu_helpers import TOL_BF16, TOL_F32, dev_f32, dev_weights, errors, run_layer  # noqa: E402

CALLS = [
    # d, d_ff, wdtype, T, counts per sample, max_count
    (2048, 16384, "bf16", 51, [4916], 4916),  # one sample's long list: the one-launch layer form, its XCD copies
    (1024, 4096, "bf16", 51, [1229, 0, 700], 1229),
    (256, 1024, "bf16", 8, [100], 100),
]


def _lists(masks):
    idx, cnt = [], []
    for m in masks:
        ix, c = oracle.compact_mask(m[None])
        idx.append(ix[0])
        cnt.append(c[0])
    return (torch.from_numpy(np.stack(idx)).cuda(), torch.from_numpy(np.asarray(cnt, np.int32)).cuda())


def _case(i, d, d_ff, wdtype, T, counts, max_count):
    layer = wl.make_layer(41, i, d, d_ff, wdtype, norm="random")
    x = wl.make_x(41, (len(counts), T, d), i)
    masks = wl.ragged_masks(41, d_ff, counts, i)
    return layer, x, masks


def _oracle(layer, x, masks):
    wg, wu, wd, g = layer.f64()
    return np.stack([oracle.masked_ffn(x[b].astype(np.float64), wg, wu, wd, masks[b].astype(np.float64), g)
                     for b in range(x.shape[0])])


def test_noalloc_layer_matches_workspace_layer_on_consecutive_calls():
    for i, (d, d_ff, wdtype, T, counts, max_count) in enumerate(CALLS):
        print(f"call {i}: d={d} d_ff={d_ff} {wdtype} T={T} counts={counts}", flush=True)
        layer, x, masks = _case(i, d, d_ff, wdtype, T, counts, max_count)
        lw = dev_weights(layer)
        idx, cnt = _lists(masks)
        xt = dev_f32(x)
        yt = torch.full_like(xt, float("nan"))
        rm.rm_sparse_ffn_layer_noalloc(xt, yt, lw, idx, cnt, max_count)
        torch.cuda.synchronize()
        y = yt.cpu().numpy()
        y_ws = run_layer(lw, x, idx, cnt, max_count)
        assert np.array_equal(y.view(np.uint32), y_ws.view(np.uint32)), i
        e, ed = errors(y, _oracle(layer, x, masks), x)
        print(f"  rel err {e:.2e}, on the FFN delta {ed:.2e}")
        assert ed <= (TOL_BF16 if wdtype == "bf16" else TOL_F32)
        for b, c in enumerate(counts):
            if c == 0:  # an empty list leaves the sample's rows bit for bit
                assert np.array_equal(y[b].view(np.uint32), x[b].view(np.uint32))


def test_noalloc_layer_in_place_and_rejects_oversize():
    d, d_ff, T = 512, 2048, 20
    layer = wl.make_layer(42, 0, d, d_ff, "bf16")
    x = wl.make_x(42, (1, T, d), 0)
    masks = wl.ragged_masks(42, d_ff, [300])
    lw = dev_weights(layer)
    idx, cnt = _lists(masks)
    xt = dev_f32(x)
    rm.rm_sparse_ffn_layer_noalloc(xt, xt, lw, idx, cnt, 300)  # y == x
    torch.cuda.synchronize()
    assert np.array_equal(xt.cpu().numpy().view(np.uint32), run_layer(lw, x, idx, cnt, 300).view(np.uint32))
    big = torch.zeros((64, 64, 4096), device="cuda")
    wbig = torch.zeros((16384, 4096), dtype=torch.bfloat16, device="cuda")
    ibig = torch.zeros((64, 16384), dtype=torch.int32, device="cuda")
    cbig = torch.zeros((64,), dtype=torch.int32, device="cuda")
    with pytest.raises(rm.RmError) as ei:
        rm.rm_sparse_ffn_layer_noalloc(big, big, (wbig, wbig, wbig, None), ibig, cbig, 16384)
    assert ei.value.status == rm.RM_ERR_WORKSPACE
