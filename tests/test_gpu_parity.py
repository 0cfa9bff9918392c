"""GPU parity: the HIP library through its C ABI against the float64 CPU oracle, on the same seeded inputs.

Bars: compaction bit-exact (idx including its -1 tail, and count); FFN outputs within max-abs relative error
2e-2 (bf16 weights) or 1e-5 (float32 weights) of the oracle, on both y and the FFN delta y - x; the empty list
gives y == x bit for bit."""
import numpy as np
import pytest
import torch

import oracle
import workloads as wl

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2609_19104_amd as rm  # noqa: E402
from gpu_helpers import (TOL_BF16, TOL_F32, compact, dev_f32, dev_weights, errors, run_dense,  # noqa: E402
                         run_layer, run_stack)


def _oracle_layer(layer, x, mult):
    wg, wu, wd, g = layer.f64()
    return np.stack([oracle.masked_ffn(x[b], wg, wu, wd, mult[b], g) for b in range(x.shape[0])])


def _masks_to_lists(masks):
    idx, cnt = compact(masks)
    torch.cuda.synchronize()
    ref_idx, ref_cnt = oracle.compact_mask(masks)
    assert np.array_equal(cnt.cpu().numpy(), ref_cnt)
    assert np.array_equal(idx.cpu().numpy(), ref_idx)
    return idx, cnt


def _check(y, y_ref, x, tol, label=""):
    ey, ed = errors(y, y_ref, x)
    print(f"{label} rel err y {ey:.3e} delta {ed:.3e}")
    assert ey <= tol and ed <= tol, f"{label}: rel err y {ey:.3e}, delta {ed:.3e} > {tol}"


# ------------------------------------------------------------------------------------------------ compaction

@pytest.mark.parametrize("d_ff", [1, 3, 63, 64, 65, 1000, 1001, 1024, 4095, 4096, 16384])
@pytest.mark.parametrize("p", [0.0, 0.02, 0.3, 0.97, 1.0])
def test_compact_random_bit_exact(d_ff, p):
    masks = wl.bernoulli_mask(np.random.default_rng(d_ff * 7 + int(p * 100)), (5, d_ff), p)
    masks[masks == 1] = np.random.default_rng(1).integers(1, 256, size=int(masks.sum()), dtype=np.uint8)
    _masks_to_lists(masks)


def test_compact_edge_masks_bit_exact():
    for d_ff in (1, 2, 255, 256, 257, 1023, 1025, 4096):
        rows = [np.zeros(d_ff), np.ones(d_ff), np.eye(1, d_ff, 0)[0], np.eye(1, d_ff, d_ff - 1)[0],
                (np.arange(d_ff) % 2 == 1), (np.arange(d_ff) % 64 == 63)]
        _masks_to_lists(np.stack(rows).astype(np.uint8))


def test_compact_bool_tensor_storage():
    m = torch.from_numpy(wl.bernoulli_mask(np.random.default_rng(3), (4, 300), 0.4).astype(bool)).cuda()
    idx = torch.empty((4, 300), dtype=torch.int32, device="cuda")
    cnt = torch.empty(4, dtype=torch.int32, device="cuda")
    rm.rm_mask_compact(m, idx, cnt)
    ref_idx, ref_cnt = oracle.compact_mask(m.cpu().numpy().astype(np.uint8))
    assert np.array_equal(idx.cpu().numpy(), ref_idx) and np.array_equal(cnt.cpu().numpy(), ref_cnt)


def test_compact_config5_masks():
    w = wl.config5()
    _masks_to_lists(w.masks.reshape(-1, w.d_ff))


# ------------------------------------------------------------------------------------------------ small layers

BF16_CASES = [
    # d, d_ff, T, k, norm
    (256, 1000, 51, 333, "none"),
    (256, 1000, 1, 1000, "random"),
    (512, 777, 65, 500, "random"),
    (128, 300, 130, 64, "none"),
    (96, 64, 17, 1, "none"),
    (160, 200, 64, 199, "ones"),
    (1024, 4096, 51, 1229, "none"),
    # long lists: the pipelined gate/up kernel with 2, 4 and 8 neuron groups per workgroup and 1 or 2 column
    # chunks; the staged kernel for a chunk count it does not cover and for T > 64
    (256, 8192, 40, 4096, "random"),
    (512, 8192, 51, 8192, "none"),
    (512, 16384, 64, 16384, "ones"),
    (768, 4096, 33, 2048, "none"),
    (256, 8192, 100, 4096, "none"),
    # T > 64 at d = 2048 and d = 768: the staged kernel with eight and three column chunks
    (2048, 4096, 100, 1500, "random"),
    (768, 2048, 90, 700, "ones"),
    # one sample with 256 .. 1024 groups of 8 slots: the spread gate/up kernel with 2, 3 and 4 groups per
    # workgroup, 1 to 8 column chunks; a grid with only four workgroups of two groups
    (2048, 8192, 51, 6000, "random"),
    (1024, 8192, 64, 8192, "ones"),
    (256, 4096, 17, 2056, "none"),
    (512, 4096, 51, 2500, "random"),
    # the split down projection's K-slices of 12, 24 and 28 chunks (3, 6 and 7 per wave), 256 workgroups or fewer
    (1024, 8192, 51, 5000, "none"),
    (1024, 16384, 51, 11000, "random"),
    (1024, 16384, 33, 13500, "none"),
]


@pytest.mark.parametrize("d,d_ff,T,k,norm", BF16_CASES)
def test_bf16_layer_parity(d, d_ff, T, k, norm):
    layer = wl.make_layer(11, d, d, d_ff, "bf16", norm=norm)
    x = wl.make_x(11, (1, T, d), d_ff, T)
    mask = wl.uniform_mask(wl.rng(11, 4, d, d_ff, T), d_ff, k)[None]
    idx, cnt = _masks_to_lists(mask)
    y = run_layer(dev_weights(layer), x, idx, cnt, k)
    _check(y, _oracle_layer(layer, x, mask.astype(np.float64)), x, TOL_BF16, f"bf16 {d}x{d_ff} T={T} k={k}")


F32_CASES = [
    (256, 1024, 8, 256, "none"),
    (64, 100, 3, 37, "random"),
    (288, 513, 17, 200, "none"),
    (32, 16, 1, 16, "ones"),
]


@pytest.mark.parametrize("d,d_ff,T,k,norm", F32_CASES)
def test_f32_layer_parity(d, d_ff, T, k, norm):
    layer = wl.make_layer(12, d, d, d_ff, "f32", norm=norm)
    x = wl.make_x(12, (1, T, d), d_ff, T)
    mask = wl.uniform_mask(wl.rng(12, 4, d, d_ff, T), d_ff, k)[None]
    idx, cnt = _masks_to_lists(mask)
    y = run_layer(dev_weights(layer), x, idx, cnt, k)
    _check(y, _oracle_layer(layer, x, mask.astype(np.float64)), x, TOL_F32, f"f32 {d}x{d_ff} T={T} k={k}")


# ------------------------------------------------------------------------------------------------ invariants

@pytest.mark.parametrize("wdtype", ["bf16", "f32"])
def test_empty_list_is_bitwise_identity(wdtype):
    layer = wl.make_layer(13, 0, 256, 512, wdtype, norm="random")
    x = wl.make_x(13, (3, 20, 256), 0)
    x[0, 0, :5] = -0.0
    mask = np.zeros((3, 512), np.uint8)
    idx, cnt = _masks_to_lists(mask)
    y = run_layer(dev_weights(layer), x, idx, cnt, 100)
    assert np.array_equal(y.view(np.uint32), x.view(np.uint32))
    y0 = run_layer(dev_weights(layer), x, idx, cnt, 0)
    assert np.array_equal(y0.view(np.uint32), x.view(np.uint32))


@pytest.mark.parametrize("wdtype", ["bf16", "f32"])
def test_all_ones_equals_dense_and_oracle(wdtype):
    layer = wl.make_layer(14, 0, 256, 640, wdtype, norm="random")
    x = wl.make_x(14, (2, 51, 256), 0)
    mask = np.ones((2, 640), np.uint8)
    idx, cnt = _masks_to_lists(mask)
    lw = dev_weights(layer)
    y_sparse = run_layer(lw, x, idx, cnt, 640)
    y_dense = run_dense(lw, x)
    assert np.array_equal(y_sparse, y_dense)
    wg, wu, wd, g = layer.f64()
    y_ref = np.stack([oracle.dense_ffn(x[b], wg, wu, wd, g) for b in range(2)])
    _check(y_dense, y_ref, x, TOL_BF16 if wdtype == "bf16" else TOL_F32, f"dense {wdtype}")


@pytest.mark.parametrize("wdtype", ["bf16", "f32"])
def test_permuted_and_duplicated_lists(wdtype):
    d, d_ff, T = 256, 700, 33
    layer = wl.make_layer(15, 0, d, d_ff, wdtype)
    x = wl.make_x(15, (1, T, d), 0)
    r = np.random.default_rng(15)
    lst = r.choice(d_ff, size=300, replace=False).astype(np.int32)  # not sorted
    lst = np.concatenate([lst, lst[:40]])                             # 40 repeats: a multiset
    idx = np.full((1, d_ff), -1, np.int32)
    idx[0, : lst.size] = lst
    idx_t = torch.from_numpy(idx).cuda()
    cnt_t = torch.tensor([lst.size], dtype=torch.int32, device="cuda")
    lw = dev_weights(layer)
    y = run_layer(lw, x, idx_t, cnt_t, lst.size)
    mult = oracle.multiplicity(lst, lst.size, d_ff)
    tol = TOL_BF16 if wdtype == "bf16" else TOL_F32
    _check(y, _oracle_layer(layer, x, mult[None]), x, tol, f"multiset {wdtype}")
    idx_rev = idx.copy()
    idx_rev[0, : lst.size] = lst[::-1]
    y_rev = run_layer(lw, x, torch.from_numpy(idx_rev).cuda(), cnt_t, lst.size)
    _check(y_rev, _oracle_layer(layer, x, mult[None]), x, tol, f"reversed {wdtype}")


@pytest.mark.parametrize("wdtype", ["bf16", "f32"])
def test_in_place_and_deterministic(wdtype):
    layer = wl.make_layer(16, 0, 512, 1024, wdtype, norm="ones")
    x = wl.make_x(16, (2, 51, 512), 0)
    masks = np.stack([wl.uniform_mask(wl.rng(16, 4, b), 1024, 300) for b in range(2)])
    idx, cnt = _masks_to_lists(masks)
    lw = dev_weights(layer)
    y1 = run_layer(lw, x, idx, cnt, 300)
    y2 = run_layer(lw, x, idx, cnt, 300)
    y3 = run_layer(lw, x, idx, cnt, 300, in_place=True)
    assert np.array_equal(y1, y2) and np.array_equal(y1, y3)


def test_ragged_batch_counts():
    d, d_ff, T = 1024, 4096, 51
    counts = [0, 1, 63, 64, 65, 1229, 4096]
    layer = wl.make_layer(17, 0, d, d_ff, "bf16", norm="ones")
    x = wl.make_x(17, (len(counts), T, d), 0)
    masks = wl.ragged_masks(17, d_ff, counts)
    idx, cnt = _masks_to_lists(masks)
    y = run_layer(dev_weights(layer), x, idx, cnt, max(counts))
    y_ref = _oracle_layer(layer, x, masks.astype(np.float64))
    assert np.array_equal(y[0].view(np.uint32), x[0].view(np.uint32))
    for b, c in enumerate(counts[1:], start=1):
        _check(y[b], y_ref[b], x[b], TOL_BF16, f"ragged count {c}")


def test_ragged_batch_counts_f32():
    # The float32 path at config 1's shape with a host bound of d_ff: most samples use far fewer K-slices than the
    # launch has, and the slices past a sample's count hold stale workspace (NaN from run_layer's poison), which the
    # epilogue must not add.
    d, d_ff, T = 256, 1024, 8
    counts = [0, 1, 7, 8, 9, 100, 256, 1024]
    layer = wl.make_layer(27, 0, d, d_ff, "f32")
    x = wl.make_x(27, (len(counts), T, d), 0)
    masks = wl.ragged_masks(27, d_ff, counts)
    idx, cnt = _masks_to_lists(masks)
    y = run_layer(dev_weights(layer), x, idx, cnt, d_ff)
    y_ref = _oracle_layer(layer, x, masks.astype(np.float64))
    assert np.array_equal(y[0].view(np.uint32), x[0].view(np.uint32))
    for b, c in enumerate(counts[1:], start=1):
        _check(y[b], y_ref[b], x[b], TOL_F32, f"f32 ragged count {c}")


def test_counts_above_max_count_are_clamped_not_read_past():
    # count[b] larger than the host bound: only the first max_count listed neurons are applied.
    d, d_ff, T = 256, 512, 16
    layer = wl.make_layer(18, 0, d, d_ff, "bf16")
    x = wl.make_x(18, (1, T, d), 0)
    mask = wl.uniform_mask(wl.rng(18, 4), d_ff, 200)[None]
    idx, cnt = _masks_to_lists(mask)
    y = run_layer(dev_weights(layer), x, idx, cnt, 96)
    first = np.zeros(d_ff)
    first[oracle.compact_mask(mask)[0][0, :96]] = 1
    _check(y, _oracle_layer(layer, x, first[None]), x, TOL_BF16, "clamped")


def test_stack_equals_layer_sequence():
    d, d_ff, T, L, B = 256, 512, 51, 3, 2
    layers = [wl.make_layer(19, l, d, d_ff, "bf16", norm="random") for l in range(L)]
    x = wl.make_x(19, (B, T, d), 0)
    masks = np.stack([np.stack([wl.uniform_mask(wl.rng(19, 4, l, b), d_ff, 100 + 50 * l) for b in range(B)])
                      for l in range(L)])
    idx, cnt = compact(masks.reshape(L * B, d_ff))
    lws = [dev_weights(l) for l in layers]
    y_stack = run_stack(lws, x, idx, cnt, 200)
    y = x
    for l in range(L):
        y = run_layer(lws[l], y, idx[l * B:(l + 1) * B].contiguous(), cnt[l * B:(l + 1) * B].contiguous(), 200)
    # Inside a stack the down projection runs fused (one workgroup sums the whole list in wave order), a single
    # layer splits it over K-slices: the same terms, added in another order, so the two agree to rounding.
    ey, ed = errors(y_stack, y, x)
    assert ey <= 1e-5 and ed <= 1e-5, (ey, ed)
    ref = np.stack([oracle.ffn_stack(x[b], [lay.f64() for lay in layers],
                                     [masks[l, b].astype(np.float64) for l in range(L)]) for b in range(B)])
    _check(y_stack, ref, x, TOL_BF16, "stack")


@pytest.mark.parametrize("k", [1700, 2048, 2100, 64])
def test_batched_stack_list_lengths(k):
    # Several samples inside a stack: lists of up to 64 chunks run the fused down projection with one 64-token
    # workgroup per (sample, column tile), its chunks in stages of 3 (1700 neurons: 54 chunks, 7 per wave, three
    # stages; 2048: 8 per wave), longer ones the split projection and the epilogue (2100: 66 chunks), short ones
    # one chunk per wave.  T = 40 leaves rows 40-63 of the token block padding.
    d, d_ff, T, L, B = 512, 4096, 40, 2, 3
    layers = [wl.make_layer(23, l, d, d_ff, "bf16", norm="random") for l in range(L)]
    x = wl.make_x(23, (B, T, d), k)
    step = 40 if k > 100 else 8  # the samples' counts differ: ragged lists within the batch
    masks = np.stack([np.stack([wl.uniform_mask(wl.rng(23, 4, k, l, b), d_ff, k - step * b) for b in range(B)])
                      for l in range(L)])
    idx, cnt = compact(masks.reshape(L * B, d_ff))
    y = run_stack([dev_weights(l) for l in layers], x, idx, cnt, k)
    ref = np.stack([oracle.ffn_stack(x[b], [lay.f64() for lay in layers],
                                     [masks[l, b].astype(np.float64) for l in range(L)]) for b in range(B)])
    _check(y, ref, x, TOL_BF16, f"batched stack k={k}")


def test_batched_stack_partial_column_tile():
    # Several samples run 64-column fused-down tiles (4 columns per lane): at d = 160 the last tile's second
    # 32-column block lies past the row, so its lanes store nothing, not even a norm partial.
    d, d_ff, T, L, B, k = 160, 1024, 40, 3, 2, 300
    layers = [wl.make_layer(24, l, d, d_ff, "bf16", norm="random") for l in range(L)]
    x = wl.make_x(24, (B, T, d), k)
    masks = np.stack([np.stack([wl.uniform_mask(wl.rng(24, 4, l, b), d_ff, k - 20 * b) for b in range(B)])
                      for l in range(L)])
    idx, cnt = compact(masks.reshape(L * B, d_ff))
    y = run_stack([dev_weights(l) for l in layers], x, idx, cnt, k)
    ref = np.stack([oracle.ffn_stack(x[b], [lay.f64() for lay in layers],
                                     [masks[l, b].astype(np.float64) for l in range(L)]) for b in range(B)])
    _check(y, ref, x, TOL_BF16, "batched stack, partial column tile")


# ------------------------------------------------------------------------------------------------ masks in

MASKED_CASES = [
    # d, d_ff, L, B, T, p (mask density), wdtype, norm
    (256, 1000, 1, 3, 51, 0.3, "bf16", "random"),
    (1024, 4096, 1, 1, 51, 0.3, "bf16", "none"),
    (512, 4095, 2, 2, 17, 0.5, "bf16", "ones"),
    (256, 16384, 1, 2, 8, 0.1, "bf16", "none"),
    (128, 300, 3, 2, 9, 0.6, "f32", "random"),
    # one sample, 257 .. 768 groups of 8 slots: the spread gate/up kernel behind the masked calls
    (2048, 16384, 1, 1, 51, 0.3, "bf16", "none"),
    (256, 8192, 1, 1, 40, 0.3, "bf16", "none"),
    (1024, 4096, 1, 1, 64, 0.6, "bf16", "random"),
    (512, 6000, 1, 1, 33, 0.4, "bf16", "none"),
]


@pytest.mark.parametrize("d,d_ff,L,B,T,p,wdtype,norm", MASKED_CASES)
@pytest.mark.parametrize("spare", [0, 1], ids=["tight", "max_count_above_count"])
def test_masked_calls_equal_compaction_then_lists(d, d_ff, L, B, T, p, wdtype, norm, spare):
    # rm_masked_ffn_layer / _stack = rm_mask_compact + rm_sparse_ffn_layer / _stack, bit for bit where the two
    # take the same kernels, and their lists are the oracle's; with max_count at the masks' largest count, or
    # well above it (slots past the count).
    layers = [wl.make_layer(71, l, d, d_ff, wdtype, norm=norm) for l in range(L)]
    lws = [dev_weights(l) for l in layers]
    x = wl.make_x(71, (B, T, d), d_ff, T)
    masks = wl.bernoulli_mask(wl.rng(71, 4, d_ff, L), (L * B, d_ff), p)
    max_count = int(masks.sum(axis=1).max())
    if spare:
        max_count = min(d_ff, max_count + max_count // 3)
    idx_ref, cnt_ref = oracle.compact_mask(masks)
    xt = torch.from_numpy(x).cuda()
    mt = torch.from_numpy(masks).cuda()
    idx = torch.full((L * B, d_ff), 777, dtype=torch.int32, device="cuda")
    cnt = torch.full((L * B,), -3, dtype=torch.int32, device="cuda")
    y = torch.full_like(xt, float("nan"))
    ws = rm.workspace(d, d_ff, rm.wdtype_of(lws[0][0]), B, T, max_count)
    ws.fill_(0xFF)  # NaN in every float32 and bf16 slot
    if L == 1:
        rm.rm_masked_ffn_layer(xt, y, lws[0], mt, idx, cnt, max_count, ws)
    else:
        rm.rm_masked_ffn_stack(xt, y, lws, mt, idx, cnt, max_count, ws)
    torch.cuda.synchronize()
    assert np.array_equal(idx.cpu().numpy(), idx_ref) and np.array_equal(cnt.cpu().numpy(), cnt_ref)
    i2, c2 = _masks_to_lists(masks)
    y2 = run_layer(lws[0], x, i2, c2, max_count) if L == 1 else run_stack(lws, x, i2, c2, max_count)
    one_launch = rm.rm_layer_kernels(d, d_ff, rm.wdtype_of(lws[0][0]), B, T, max_count) == 1 << rm.RM_KERNEL_LAYER
    if L == 1 and d == 1024 and one_launch:
        # rm_sparse_ffn_layer takes the one-launch layer kernel, the masked call the prologue (with the
        # compaction), gate/up and fused down kernels: both within the bar of the oracle.
        tol = TOL_BF16 if wdtype == "bf16" else TOL_F32
        applied = np.zeros((L * B, d_ff))
        for i in range(L * B):
            applied[i, idx_ref[i, :min(cnt_ref[i], max_count)]] = 1
        ref = _oracle_layer(layers[0], x, applied)
        _check(y.cpu().numpy(), ref, x, tol, "masked call")
        _check(y2, ref, x, tol, "call on the lists")
    else:
        assert np.array_equal(y.cpu().numpy().view(np.uint32), y2.view(np.uint32))


# ------------------------------------------------------------------------------------------------ one-sample stacks
# A single sample's layer or stack with a list of at most 2048 neurons runs the down projection fused with the
# epilogue: one workgroup per (32-column tile, 16-token tile) sums the whole list and
# writes the next layer's input with its 32-column norm partials (2 columns per lane).

FUSED_CASES = [
    # d, d_ff, L, T, k, norm
    (96, 200, 3, 17, 150, "random"),    # three 32-column tiles, a norm over a short last span, 5 chunks
    (160, 512, 2, 70, 300, "none"),     # five token tiles (T > 64)
    (2048, 4096, 1, 51, 1500, "random"),  # one layer at d = 2048
    (1024, 4096, 2, 1, 2048, "ones"),   # T = 1, 64 chunks (8 per wave)
    (256, 2048, 3, 64, 1999, "random"),
    (2048, 8192, 2, 51, 1600, "random"),  # d = 2048 inside a stack: 8 spans of norm partials per token
]


@pytest.mark.parametrize("d,d_ff,L,T,k,norm", FUSED_CASES)
def test_single_sample_stack_parity(d, d_ff, L, T, k, norm):
    layers = [wl.make_layer(81, l, d, d_ff, "bf16", norm=norm) for l in range(L)]
    x = wl.make_x(81, (1, T, d), d_ff, T)
    masks = np.stack([wl.uniform_mask(wl.rng(81, 4, l, d_ff), d_ff, k - 37 * l) for l in range(L)])
    idx, cnt = _masks_to_lists(masks)
    lws = [dev_weights(l) for l in layers]
    y = run_stack(lws, x, idx, cnt, k)
    ref = oracle.ffn_stack(x[0], [lay.f64() for lay in layers], [m.astype(np.float64) for m in masks])
    _check(y[0], ref, x[0], TOL_BF16, f"one-sample stack {d}x{d_ff} L={L} T={T} k={k}")


def test_single_sample_stack_empty_lists_are_identity():
    d, d_ff, L, T = 256, 512, 3, 20
    layers = [wl.make_layer(82, l, d, d_ff, "bf16", norm="random") for l in range(L)]
    x = wl.make_x(82, (1, T, d), 0)
    x[0, 0, :7] = -0.0
    idx, cnt = _masks_to_lists(np.zeros((L, d_ff), np.uint8))
    y = run_stack([dev_weights(l) for l in layers], x, idx, cnt, 64)
    assert np.array_equal(y.view(np.uint32), x.view(np.uint32))
