"""GPU parity of the one-launch layer form: one sample's list of 257 .. 768 groups of 8 slots at d = 2048 (or a
single layer's list of 8 .. 192 chunks of 32 neurons at d = 1024) runs the gate/up and the down projection in one
launch whose workgroups meet per XCD (layer_xcd_kernel), then the epilogue.  Against the float64 oracle on the same seeded inputs, across that range of list lengths (the shortest,
whose last XCD slice holds 2 chunks and leaves half of that XCD's workgroups without gate/up work, up to slices
of 24 chunks), token counts 1 .. 64, with and without a norm, slots past the count, inside stacks (the per-XCD
counters carried from layer to layer), repeated calls, an empty list and an Eq. 4 delta step.

Bars: max-abs relative error 2e-2 (bf16 weights) on y and on the FFN part y - x; repeated and in-place calls
bitwise equal; an empty list y == x bit for bit; a delta step at the anchor's own input the anchor bit for bit."""
import numpy as np
import pytest
import torch

import oracle
import workloads as wl

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

from gpu_helpers import (TOL_BF16, compact, dev_weights, errors, run_anchor, run_delta, run_layer,  # noqa: E402
                         run_stack)

D = 2048


def test_the_one_launch_form_runs():
    # The calls below take the one-launch form on this device (256 compute units).
    import paper_2609_19104_amd as rm
    for d_ff, T, k in ((8192, 51, 2057), (16384, 17, 6144), (16384, 51, 4916), (8192, 1, 4300)):
        assert rm.rm_layer_kernels(D, d_ff, rm.RM_BF16, 1, T, k) == 1 << rm.RM_KERNEL_LAYER
    for d_ff, T, k in ((4096, 51, 1229), (4096, 64, 4096), (8192, 1, 6144)):
        assert rm.rm_layer_kernels(1024, d_ff, rm.RM_BF16, 1, T, k) == 1 << rm.RM_KERNEL_LAYER
    both = (1 << rm.RM_KERNEL_GATEUP) | (1 << rm.RM_KERNEL_DOWN)
    assert rm.rm_layer_kernels(1024, 4096, rm.RM_BF16, 2, 51, 1229) == both  # two samples
    assert rm.rm_layer_kernels(1024, 4096, rm.RM_BF16, 1, 51, 200) == both   # 7 chunks


def _oracle_layer(layer, x, mult):
    wg, wu, wd, g = layer.f64()
    return np.stack([oracle.masked_ffn(x[b], wg, wu, wd, mult[b], g) for b in range(x.shape[0])])


def _check(y, y_ref, x, label):
    ey, ed = errors(y, y_ref, x)
    print(f"{label}: rel err y {ey:.3e} delta {ed:.3e}")
    assert ey <= TOL_BF16 and ed <= TOL_BF16, f"{label}: rel err y {ey:.3e}, delta {ed:.3e}"


@pytest.mark.parametrize("d_ff,T,k,spare,norm", [
    (8192, 51, 2057, 0, "none"),     # 65 chunks: slices of 9, the last XCD's slice 2 chunks
    (8192, 64, 3001, 0, "random"),   # 94 chunks, slices of 12, a ragged last chunk
    (8192, 1, 4100, 200, "ones"),    # one token; slots past the count
    (16384, 17, 6144, 0, "none"),    # 192 chunks: slices of 24 (3 per wave), the range's end
    (16384, 51, 4916, 0, "random"),  # the count of a top-30% mask of 16384 neurons, with a norm
])
def test_layer_parity(d_ff, T, k, spare, norm):
    layer = wl.make_layer(131, d_ff, D, d_ff, "bf16", norm=norm)
    x = wl.make_x(131, (1, T, D), d_ff, T, k)
    mask = wl.uniform_mask(wl.rng(131, 4, d_ff, T, k), d_ff, k)[None]
    idx, cnt = compact(mask)
    y = run_layer(dev_weights(layer), x, idx, cnt, min(d_ff, k + spare))
    _check(y, _oracle_layer(layer, x, mask.astype(np.float64)), x, f"layer d_ff={d_ff} T={T} k={k}")


@pytest.mark.parametrize("d_ff,T,k,spare,norm", [
    (4096, 51, 1229, 0, "random"),   # a top-30% mask of 4096 neurons: 39 chunks, slices of 5
    (4096, 64, 4000, 96, "none"),    # 128 chunks (slices of 16), slots past the count
    (4096, 1, 256, 0, "ones"),       # 8 chunks, one per XCD; one token
    (8192, 17, 6144, 0, "random"),   # 192 chunks: slices of 24, the range's end
])
def test_layer_parity_d1024(d_ff, T, k, spare, norm):
    d = 1024
    layer = wl.make_layer(136, d_ff, d, d_ff, "bf16", norm=norm)
    x = wl.make_x(136, (1, T, d), d_ff, T, k)
    mask = wl.uniform_mask(wl.rng(136, 4, d_ff, T, k), d_ff, k)[None]
    idx, cnt = compact(mask)
    y = run_layer(dev_weights(layer), x, idx, cnt, min(d_ff, k + spare))
    _check(y, _oracle_layer(layer, x, mask.astype(np.float64)), x, f"layer d=1024 d_ff={d_ff} T={T} k={k}")
    y2 = run_layer(dev_weights(layer), x, idx, cnt, min(d_ff, k + spare), in_place=True)
    assert np.array_equal(y.view(np.uint32), y2.view(np.uint32))


def test_stack_repeat_and_in_place():
    # Three layers with ragged counts: each layer's launch finds the counters where the last one left them.
    d_ff, T, L = 8192, 51, 3
    counts = [3000, 2600, 3500]
    layers = [wl.make_layer(132, l, D, d_ff, "bf16", norm="random") for l in range(L)]
    lws = [dev_weights(l) for l in layers]
    x = wl.make_x(132, (1, T, D), 0)
    masks = np.stack([wl.uniform_mask(wl.rng(132, 4, l), d_ff, c) for l, c in enumerate(counts)])
    idx, cnt = compact(masks)
    y = run_stack(lws, x, idx, cnt, max(counts))
    y2 = run_stack(lws, x, idx, cnt, max(counts))
    assert np.array_equal(y.view(np.uint32), y2.view(np.uint32))
    ref = oracle.ffn_stack(x[0], [lay.f64() for lay in layers], [m.astype(np.float64) for m in masks])[None]
    _check(y, ref, x, "stack")
    # Layer by layer (each call with its own prologue): the same kernels, so the same bits.
    yl = x
    for l in range(L):
        yl = run_layer(lws[l], yl, idx[l:l + 1].contiguous(), cnt[l:l + 1].contiguous(), max(counts))
    assert np.array_equal(yl.view(np.uint32), y.view(np.uint32))
    y_in = run_layer(lws[0], x, idx[:1].contiguous(), cnt[:1].contiguous(), max(counts), in_place=True)
    y_out = run_layer(lws[0], x, idx[:1].contiguous(), cnt[:1].contiguous(), max(counts))
    assert np.array_equal(y_in.view(np.uint32), y_out.view(np.uint32))


def test_empty_and_clamped_counts():
    d_ff, T = 8192, 33
    layer = wl.make_layer(133, 0, D, d_ff, "bf16", norm="random")
    lw = dev_weights(layer)
    x = wl.make_x(133, (1, T, D), 0)
    x[0, 0, :5] = -0.0
    idx, cnt = compact(np.zeros((1, d_ff), np.uint8))
    y = run_layer(lw, x, idx, cnt, 3000)  # the plan of a 3000-slot list, no listed neuron
    assert np.array_equal(y.view(np.uint32), x.view(np.uint32))
    # A count above max_count: only the first max_count listed neurons are applied.
    mask = wl.uniform_mask(wl.rng(133, 4), d_ff, 4000)[None]
    idx, cnt = compact(mask)
    y = run_layer(lw, x, idx, cnt, 2500)
    first = np.zeros(d_ff)
    first[oracle.compact_mask(mask)[0][0, :2500]] = 1
    _check(y, _oracle_layer(layer, x, first[None]), x, "clamped count")


def test_delta_step():
    # Eq. 4: the dense anchor keeps y_a and the group list's h_a (captured by the spread gate/up launch); the
    # delta step runs the one-launch form on the same list.
    d_ff, T, L, k = 8192, 51, 2, 3000
    layers = [wl.make_layer(134, l, D, d_ff, "bf16", norm="random") for l in range(L)]
    lws = [dev_weights(l) for l in layers]
    xa = wl.make_x(134, (1, T, D), 0)
    xt = (xa + 0.05 * np.random.default_rng(135).standard_normal(xa.shape)).astype(np.float32)
    masks = np.stack([wl.uniform_mask(wl.rng(134, 4, l), d_ff, k - 100 * l) for l in range(L)])
    idx, cnt = compact(masks)
    y, ya, ha = run_anchor(lws, xa, idx, cnt, k)
    yd = run_delta(lws, xt, idx, cnt, k, ya, ha)
    lay = [l.f64() for l in layers]
    _, ya_ref, ha_ref = oracle.anchor_stack(xa[0], lay)
    ref = oracle.delta_stack(xt[0], lay, [m.astype(np.float64) for m in masks], ya_ref, ha_ref)[None]
    _check(yd, ref, xt, "delta step")
    y_same = run_delta(lws, xa, idx, cnt, k, ya, ha)
    assert np.array_equal(y_same.view(np.uint32), y.cpu().numpy().view(np.uint32))


def _masked(lws, x, masks, max_count, mask_dev=None):
    """rm_masked_ffn_layer (one mask) or rm_masked_ffn_stack -> (y, idx, count) as numpy arrays."""
    import paper_2609_19104_amd as rm
    d_ff, d = lws[0][0].shape
    n = masks.shape[0]
    xt = torch.from_numpy(np.ascontiguousarray(x)).cuda()
    mt = torch.from_numpy(masks).cuda() if mask_dev is None else mask_dev
    idx = torch.full((n, d_ff), 777, dtype=torch.int32, device="cuda")
    cnt = torch.full((n,), -3, dtype=torch.int32, device="cuda")
    y = torch.full_like(xt, float("nan"))
    ws = rm.workspace(d, d_ff, rm.RM_BF16, 1, x.shape[1], max_count)
    ws.fill_(0xFF)
    if n == 1:
        rm.rm_masked_ffn_layer(xt, y, lws[0], mt, idx, cnt, max_count, ws)
    else:
        rm.rm_masked_ffn_stack(xt, y, lws, mt, idx, cnt, max_count, ws)
    torch.cuda.synchronize()
    return y.cpu().numpy(), idx.cpu().numpy(), cnt.cpu().numpy()


@pytest.mark.parametrize("d,d_ff,L,T,counts,max_count", [
    (2048, 8192, 2, 51, [3000, 2600], 3000),  # a masked stack: each layer's launch compacts its own mask
    (2048, 16384, 1, 51, [4000], 2500),       # count above max_count: the whole list out, 2500 applied
    (2048, 16384, 1, 17, [0], 3000),          # an empty mask
    (1024, 4096, 1, 64, [4096], 4096),        # every neuron
    (1024, 4112, 1, 5, [4100], 4112),         # d_ff = 257 x 16: the last chunk past d_ff, slots past the count
])
def test_masked_calls_in_the_one_launch_range(d, d_ff, L, T, counts, max_count):
    # Masked calls whose lists the one-launch form takes: idx / count bit for bit the oracle's compaction (the -1
    # tail included); y bit for bit the same call on those lists at d = 2048 (the compaction launch ahead of the
    # same kernels), within the bar of the oracle at d = 1024 (a masked single layer there keeps the compaction in
    # the prologue's launch and the gate/up and fused down kernels).
    import paper_2609_19104_amd as rm
    assert rm.rm_layer_kernels(d, d_ff, rm.RM_BF16, 1, T, max_count) == 1 << rm.RM_KERNEL_LAYER
    layers = [wl.make_layer(137, l, d, d_ff, "bf16", norm="random") for l in range(L)]
    lws = [dev_weights(l) for l in layers]
    x = wl.make_x(137, (1, T, d), d_ff, T)
    masks = np.stack([wl.uniform_mask(wl.rng(137, 4, l, d_ff), d_ff, c) for l, c in enumerate(counts)])
    y, idx, cnt = _masked(lws, x, masks, max_count)
    idx_ref, cnt_ref = oracle.compact_mask(masks)
    assert np.array_equal(cnt, cnt_ref) and np.array_equal(idx, idx_ref)
    i2, c2 = compact(masks)
    y2 = run_layer(lws[0], x, i2, c2, max_count) if L == 1 else run_stack(lws, x, i2, c2, max_count)
    if counts == [0]:
        assert np.array_equal(y.view(np.uint32), x.view(np.uint32))
    if d == 2048:
        assert np.array_equal(y.view(np.uint32), y2.view(np.uint32))
    else:
        applied = np.zeros((L, d_ff))
        for l in range(L):
            applied[l, idx_ref[l, :min(cnt_ref[l], max_count)]] = 1
        ref = oracle.ffn_stack(x[0], [lay.f64() for lay in layers], list(applied))[None]
        _check(y, ref, x, "masked call")
        _check(y2, ref, x, "call on the lists")



def test_form_switched_off_by_the_environment(tmp_path):
    # RM_NO_LAYER_FORM=1 (read at the process's first call): the same layer takes the other kernels, in a child
    # process; both results within the bar of the oracle.
    import os
    import subprocess
    import sys
    import paper_2609_19104_amd as rm
    d_ff, T, k = 8192, 17, 3000
    assert rm.rm_layer_kernels(D, d_ff, rm.RM_BF16, 1, T, k) == 1 << rm.RM_KERNEL_LAYER
    here = os.path.dirname(os.path.abspath(__file__))
    out = tmp_path / "y.npy"
    child = f"""
import sys
sys.path[:0] = [{here!r}, {os.path.dirname(here)!r}]
import numpy as np, torch
import paper_2609_19104_amd as rm, workloads as wl
from gpu_helpers import compact, dev_weights, run_layer
both = (1 << rm.RM_KERNEL_GATEUP) | (1 << rm.RM_KERNEL_DOWN)
assert rm.rm_layer_kernels({D}, {d_ff}, rm.RM_BF16, 1, {T}, {k}) == both
layer = wl.make_layer(139, 0, {D}, {d_ff}, "bf16", norm="random")
x = wl.make_x(139, (1, {T}, {D}), 0)
idx, cnt = compact(wl.uniform_mask(wl.rng(139, 4), {d_ff}, {k})[None])
np.save({str(out)!r}, run_layer(dev_weights(layer), x, idx, cnt, {k}))
"""
    env = dict(os.environ, RM_NO_LAYER_FORM="1")
    r = subprocess.run([sys.executable, "-c", child], env=env, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-2000:]
    y_off = np.load(out)
    layer = wl.make_layer(139, 0, D, d_ff, "bf16", norm="random")
    x = wl.make_x(139, (1, T, D), 0)
    mask = wl.uniform_mask(wl.rng(139, 4), d_ff, k)[None]
    idx, cnt = compact(mask)
    y_on = run_layer(dev_weights(layer), x, idx, cnt, k)
    ref = _oracle_layer(layer, x, mask.astype(np.float64))
    _check(y_on, ref, x, "one-launch form")
    _check(y_off, ref, x, "form switched off")
    assert not np.array_equal(y_on.view(np.uint32), y_off.view(np.uint32))  # the other kernels did run
