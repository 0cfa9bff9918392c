"""Pins for the CPU oracle: closed forms, library special cases, invariants and brute force.

None of these re-type the oracle's own formula: each one checks it against something the mathematics or a
different implementation fixes, so that a dropped term, a wrong sign or index or a transposed operand in the
oracle fails at least one of them.
"""
import itertools
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import workloads as wl


def _rand_layer(seed, d, d_ff, norm=False):
    r = np.random.default_rng(seed)
    wg = r.standard_normal((d_ff, d)) * 0.3
    wu = r.standard_normal((d_ff, d)) * 0.3
    wd = r.standard_normal((d_ff, d)) * 0.3
    g = (1.0 + 0.2 * r.standard_normal(d)) if norm else None
    return wg, wu, wd, g


def _torch_swiglu(x, wg, wu, wd, g=None, eps=1e-6, zero_down_rows=None, zero_up_rows=None, act="silu", gate=None):
    """Textbook SwiGLU (or GeGLU) FFN + residual through torch's float64 library ops (an independent
    implementation); gate multiplies the FFN output before the residual."""
    xt = torch.tensor(x, dtype=torch.float64)
    wg_t = torch.tensor(wg, dtype=torch.float64)
    wu_t = torch.tensor(wu, dtype=torch.float64)
    wd_t = torch.tensor(wd, dtype=torch.float64)
    if zero_down_rows is not None:
        wd_t[torch.tensor(zero_down_rows, dtype=torch.long)] = 0.0
    if zero_up_rows is not None:
        wu_t[torch.tensor(zero_up_rows, dtype=torch.long)] = 0.0
    xn = xt
    if g is not None:
        xn = F.rms_norm(xt, (xt.shape[-1],), weight=torch.tensor(g, dtype=torch.float64), eps=eps)
    a = F.linear(xn, wg_t)
    h = (F.silu(a) if act == "silu" else F.gelu(a, approximate="tanh")) * F.linear(xn, wu_t)
    # nn.Linear convention: down_proj.weight is [d][d_ff] = transpose of the neuron-major rows.
    f = F.linear(h, wd_t.T.contiguous())
    if gate is not None:
        f = f * torch.tensor(gate, dtype=torch.float64)
    return (xt + f).numpy()


# ------------------------------------------------------------------------------------------------ GeGLU, gate

def test_gelu_tanh_matches_library_and_closed_forms():
    z = np.concatenate([np.linspace(-12, 12, 2001), [-80.0, 80.0, 0.0, 1e-9]])
    ref = F.gelu(torch.tensor(z, dtype=torch.float64), approximate="tanh").numpy()
    assert np.max(np.abs(oracle.gelu_tanh(z) - ref)) < 1e-14
    assert oracle.gelu_tanh(np.array([0.0]))[0] == 0.0
    # tanh is odd, so gelu(z) - gelu(-z) = z.
    assert np.max(np.abs(oracle.gelu_tanh(z) - oracle.gelu_tanh(-z) - z)) < 1e-12


@pytest.mark.parametrize("norm", [False, True])
def test_geglu_and_gate_match_torch(norm):
    wg, wu, wd, g = _rand_layer(50, 16, 40, norm)
    r = np.random.default_rng(51)
    x = r.standard_normal((5, 16))
    gate = 1.0 + 0.5 * r.standard_normal(16)
    m = wl.bernoulli_mask(r, (40,), 0.5)
    off = np.flatnonzero(m == 0)
    got = oracle.masked_ffn(x, wg, wu, wd, m.astype(float), g, act="gelu_tanh", gate=gate)
    ref = _torch_swiglu(x, wg, wu, wd, g, zero_down_rows=off, act="gelu_tanh", gate=gate)
    assert np.max(np.abs(got - ref)) < 1e-13
    # The gate scales the FFN part only: all ones is no gate, zeros leave the residual, and it is linear.
    plain = oracle.masked_ffn(x, wg, wu, wd, m.astype(float), g)
    assert np.array_equal(oracle.masked_ffn(x, wg, wu, wd, m.astype(float), g, gate=np.ones(16)), plain)
    assert np.array_equal(oracle.masked_ffn(x, wg, wu, wd, m.astype(float), g, gate=np.zeros(16)), x)
    twice = oracle.masked_ffn(x, wg, wu, wd, m.astype(float), g, gate=2 * np.ones(16))
    assert np.max(np.abs((twice - x) - 2 * (plain - x))) < 1e-13


def test_gated_geglu_anchor_and_delta_stacks():
    layers = [_rand_layer(52 + l, 8, 12, True) for l in range(3)]
    r = np.random.default_rng(55)
    xa = r.standard_normal((4, 8))
    xt = xa + 0.05 * r.standard_normal((4, 8))
    ga = [1.0 + 0.3 * r.standard_normal(8) for _ in range(3)]  # the anchor step's gates
    gt = [1.0 + 0.3 * r.standard_normal(8) for _ in range(3)]  # a later step's gates (another timestep)
    y_anchor, ya, ha = oracle.anchor_stack(xa, layers, act="gelu_tanh", gates=ga)
    ref = xa
    for (wg, wu, wd, g), gg in zip(layers, ga):
        ref = _torch_swiglu(ref, wg, wu, wd, g, act="gelu_tanh", gate=gg)
    assert np.max(np.abs(y_anchor - ref)) < 1e-12
    # Every neuron selected: the dense gated stack at the current input with the current gates, since y_a is
    # kept before the gate.
    full = oracle.delta_stack(xt, layers, [np.ones(12)] * 3, ya, ha, act="gelu_tanh", gates=gt)
    ref = xt
    for (wg, wu, wd, g), gg in zip(layers, gt):
        ref = _torch_swiglu(ref, wg, wu, wd, g, act="gelu_tanh", gate=gg)
    assert np.max(np.abs(full - ref)) < 1e-12
    # No neuron selected: each layer adds its gated anchor output.
    empty = oracle.delta_stack(xt, layers, [np.zeros(12)] * 3, ya, ha, act="gelu_tanh", gates=gt)
    assert np.array_equal(empty, ((xt + ya[0] * gt[0]) + ya[1] * gt[1]) + ya[2] * gt[2])


# ------------------------------------------------------------------------------------------------ SiLU

def test_silu_closed_forms():
    # sigmoid(ln 3) = 3/4, so SiLU(ln 3) = 0.75 ln 3; sigmoid(-ln 3) = 1/4.
    assert oracle.silu(np.array([math.log(3.0)]))[0] == pytest.approx(0.75 * math.log(3.0), rel=1e-15)
    assert oracle.silu(np.array([-math.log(3.0)]))[0] == pytest.approx(-0.25 * math.log(3.0), rel=1e-15)
    assert oracle.silu(np.array([0.0]))[0] == 0.0
    # Far tails: SiLU(z) -> z for z -> +inf, -> z e^z for z -> -inf (no overflow).
    assert oracle.silu(np.array([60.0]))[0] == pytest.approx(60.0, rel=1e-15)
    assert oracle.silu(np.array([-800.0]))[0] == 0.0
    assert oracle.silu(np.array([-40.0]))[0] == pytest.approx(-40.0 * math.exp(-40.0), rel=1e-12)


def test_silu_odd_part_identity():
    # z*s(z) - (-z)*s(-z) = z (s(z) + s(-z)) = z for every z: catches a wrong sign in either branch.
    z = np.linspace(-30, 30, 2001)
    assert np.max(np.abs(oracle.silu(z) - oracle.silu(-z) - z)) < 1e-13


def test_silu_minimum():
    # The global minimum of z*sigmoid(z) is at z* = -(1 + W(1/e)) = -1.2784645427610738 (W = Lambert W),
    # with value -0.27846454276107380 (z* sigmoid(z*) = z* + 1).
    zs = -1.2784645427610738
    assert oracle.silu(np.array([zs]))[0] == pytest.approx(zs + 1.0, abs=1e-15)
    grid = np.linspace(-3, 1, 400001)
    assert float(np.min(oracle.silu(grid))) == pytest.approx(zs + 1.0, abs=1e-11)


def test_silu_matches_library():
    z = np.random.default_rng(0).standard_normal(10000) * 8
    ref = F.silu(torch.tensor(z, dtype=torch.float64)).numpy()
    assert np.max(np.abs(oracle.silu(z) - ref)) < 1e-14


# ------------------------------------------------------------------------------------------------ RMSNorm

def test_rms_norm_closed_form():
    x = np.array([3.0, 4.0])  # mean square 12.5
    out = oracle.rms_norm(x, np.array([1.0, 2.0]), eps=0.0)
    assert out == pytest.approx([3.0 / math.sqrt(12.5), 8.0 / math.sqrt(12.5)], rel=1e-15)
    out = oracle.rms_norm(x, np.ones(2), eps=1e-6)
    assert out == pytest.approx(x / math.sqrt(12.5 + 1e-6), rel=1e-15)


def test_rms_norm_matches_library_and_scale_invariance():
    r = np.random.default_rng(1)
    x = r.standard_normal((7, 33))
    g = 1 + 0.1 * r.standard_normal(33)
    ref = F.rms_norm(torch.tensor(x), (33,), weight=torch.tensor(g), eps=1e-6).numpy()
    assert np.max(np.abs(oracle.rms_norm(x, g) - ref)) < 1e-14
    # Scaling a row by c > 0 leaves it unchanged once eps is negligible.
    assert np.allclose(oracle.rms_norm(5.0 * x, g, eps=0.0), oracle.rms_norm(x, g, eps=0.0), rtol=1e-14, atol=0)


# ------------------------------------------------------------------------------------------------ compaction

def test_compact_fixtures():
    idx, cnt = oracle.compact_mask(np.array([0, 1, 1, 0, 1], dtype=np.uint8))
    assert cnt == 3 and idx.tolist() == [1, 2, 4, -1, -1]
    idx, cnt = oracle.compact_mask(np.zeros(6, np.uint8))
    assert cnt == 0 and idx.tolist() == [-1] * 6
    idx, cnt = oracle.compact_mask(np.array([7, 255, 1], dtype=np.uint8))  # any nonzero byte is active
    assert cnt == 3 and idx.tolist() == [0, 1, 2]
    idx, cnt = oracle.compact_mask(np.array([[1, 0, 0, 1], [0, 0, 0, 0], [0, 0, 2, 0]], np.uint8))
    assert cnt.tolist() == [2, 0, 1]
    assert idx.tolist() == [[0, 3, -1, -1], [-1] * 4, [2, -1, -1, -1]]


def test_compact_exhaustive_small():
    # Every mask of length <= 10: the list is strictly ascending, has popcount entries, scatters back to the mask,
    # and its tail is -1.
    for n in range(1, 11):
        for bits in itertools.product([0, 1], repeat=n):
            m = np.array(bits, dtype=np.uint8)
            idx, cnt = oracle.compact_mask(m)
            assert cnt == sum(bits)
            assert all(idx[i] < idx[i + 1] for i in range(cnt - 1))
            back = np.zeros(n, np.uint8)
            back[idx[:cnt]] = 1
            assert back.tolist() == list(bits)
            assert (idx[cnt:] == -1).all()


def test_compact_edge_masks():
    for d_ff in (1, 63, 64, 65, 255, 256, 257, 1000, 4096):
        for m in (np.zeros(d_ff), np.ones(d_ff), np.eye(1, d_ff, 0)[0], np.eye(1, d_ff, d_ff - 1)[0],
                  (np.arange(d_ff) % 2 == 1)):
            m = m.astype(np.uint8)
            idx, cnt = oracle.compact_mask(m)
            assert cnt == int(m.sum())
            assert (np.diff(idx[:cnt]) > 0).all()
            assert (m[idx[:cnt]] == 1).all() and (idx[cnt:] == -1).all()


# ------------------------------------------------------------------------------------------------ masked FFN

def test_scalar_closed_form():
    # d = 1, d_ff = 1: y = x + wd * SiLU(wg x) * (wu x).  With x = 2, wg = 0.5, wu = 3, wd = 0.25:
    # SiLU(1) = 1 / (1 + e^-1), y = 2 + 0.25 * 6 / (1 + e^-1).
    y = oracle.masked_ffn(np.array([[2.0]]), np.array([[0.5]]), np.array([[3.0]]), np.array([[0.25]]),
                          np.array([1.0]))
    assert y[0, 0] == pytest.approx(2.0 + 1.5 / (1.0 + math.exp(-1.0)), rel=1e-15)
    y0 = oracle.masked_ffn(np.array([[2.0]]), np.array([[0.5]]), np.array([[3.0]]), np.array([[0.25]]),
                           np.array([0.0]))
    assert y0[0, 0] == 2.0


def test_two_neuron_hand_example():
    # d = 2, d_ff = 2, one token x = (1, -1).  Neuron 0: gate (1, 0) -> 1, up (0, -2) -> 2, down (1, 2).
    # Neuron 1: gate (0, 1) -> -1, up (1, 1) -> 0, down (5, 5) -> contributes 0 whatever the gate.
    # y = x + SiLU(1) * 2 * (1, 2).
    wg = np.array([[1.0, 0.0], [0.0, 1.0]])
    wu = np.array([[0.0, -2.0], [1.0, 1.0]])
    wd = np.array([[1.0, 2.0], [5.0, 5.0]])
    s1 = 1.0 / (1.0 + math.exp(-1.0))
    y = oracle.masked_ffn(np.array([[1.0, -1.0]]), wg, wu, wd, np.array([1.0, 1.0]))
    assert y[0] == pytest.approx([1.0 + 2 * s1, -1.0 + 4 * s1], rel=1e-15)
    y = oracle.masked_ffn(np.array([[1.0, -1.0]]), wg, wu, wd, np.array([0.0, 1.0]))
    assert y[0].tolist() == [1.0, -1.0]


@pytest.mark.parametrize("norm", [False, True])
def test_dense_equals_torch_swiglu(norm):
    wg, wu, wd, g = _rand_layer(2, 24, 40, norm)
    x = np.random.default_rng(3).standard_normal((5, 24))
    ref = _torch_swiglu(x, wg, wu, wd, g)
    assert np.max(np.abs(oracle.dense_ffn(x, wg, wu, wd, g) - ref)) < 1e-13


@pytest.mark.parametrize("norm", [False, True])
def test_masked_equals_dense_with_zeroed_rows(norm):
    # A masked FFN is the dense FFN whose inactive neurons have their down rows (equally, their up rows) zeroed.
    wg, wu, wd, g = _rand_layer(4, 16, 48, norm)
    x = np.random.default_rng(5).standard_normal((3, 16))
    m = wl.bernoulli_mask(np.random.default_rng(6), (48,), 0.4)
    off = np.flatnonzero(m == 0)
    got = oracle.masked_ffn(x, wg, wu, wd, oracle.mask_multiplicity(m), g)
    assert np.max(np.abs(got - _torch_swiglu(x, wg, wu, wd, g, zero_down_rows=off))) < 1e-13
    assert np.max(np.abs(got - _torch_swiglu(x, wg, wu, wd, g, zero_up_rows=off))) < 1e-13


def test_empty_mask_is_identity():
    wg, wu, wd, g = _rand_layer(7, 8, 12, True)
    x = np.random.default_rng(8).standard_normal((4, 8))
    assert np.array_equal(oracle.masked_ffn(x, wg, wu, wd, np.zeros(12), g), x)


def test_neuron_permutation_invariance():
    wg, wu, wd, _ = _rand_layer(9, 10, 20)
    x = np.random.default_rng(10).standard_normal((3, 10))
    m = wl.bernoulli_mask(np.random.default_rng(11), (20,), 0.5).astype(np.float64)
    p = np.random.default_rng(12).permutation(20)
    a = oracle.masked_ffn(x, wg, wu, wd, m)
    b = oracle.masked_ffn(x, wg[p], wu[p], wd[p], m[p])
    assert np.max(np.abs(a - b)) < 1e-13


def test_disjoint_mask_additivity():
    wg, wu, wd, g = _rand_layer(13, 12, 30, True)
    x = np.random.default_rng(14).standard_normal((4, 12))
    r = np.random.default_rng(15)
    m1 = wl.bernoulli_mask(r, (30,), 0.5).astype(np.float64)
    m2 = (1 - m1) * wl.bernoulli_mask(r, (30,), 0.5)
    d1 = oracle.masked_ffn(x, wg, wu, wd, m1, g) - x
    d2 = oracle.masked_ffn(x, wg, wu, wd, m2, g) - x
    d12 = oracle.masked_ffn(x, wg, wu, wd, m1 + m2, g) - x
    assert np.max(np.abs(d12 - d1 - d2)) < 1e-13


def test_dyadic_scaling_of_down_rows():
    wg, wu, wd, _ = _rand_layer(16, 8, 16)
    x = np.random.default_rng(17).standard_normal((2, 8))
    m = np.ones(16)
    d1 = oracle.masked_ffn(x, wg, wu, wd, m) - x
    d2 = oracle.masked_ffn(x, wg, wu, 2.0 * wd, m) - x
    # Exact up to the rounding of the residual add and its subtraction here.
    assert np.max(np.abs(d2 - 2.0 * d1)) < 1e-14
    # Doubling the up rows doubles h and so the delta too; doubling the gate rows does not.
    d3 = oracle.masked_ffn(x, wg, 2.0 * wu, wd, m) - x
    d4 = oracle.masked_ffn(x, 2.0 * wg, wu, wd, m) - x
    assert np.max(np.abs(d3 - 2.0 * d1)) < 1e-14
    assert np.max(np.abs(d4 - 2.0 * d1)) > 1e-3


def test_multiset_duplicates_count_twice():
    wg, wu, wd, _ = _rand_layer(18, 6, 10)
    x = np.random.default_rng(19).standard_normal((2, 6))
    idx = np.array([3, 7, 3, 1], dtype=np.int32)
    mult = oracle.multiplicity(idx, 4, 10)
    assert mult.tolist() == [0, 1, 0, 2, 0, 0, 0, 1, 0, 0]
    wd2 = wd.copy()
    wd2[3] *= 2.0
    ref = oracle.masked_ffn(x, wg, wu, wd2, (mult > 0).astype(float))
    assert np.max(np.abs(oracle.masked_ffn(x, wg, wu, wd, mult) - ref)) < 1e-14


def test_residual_uses_unnormalized_input():
    wg, wu, wd, g = _rand_layer(20, 8, 12, True)
    x = np.random.default_rng(21).standard_normal((3, 8)) * 4
    y = oracle.masked_ffn(x, wg, wu, wd, np.ones(12), g)
    xn = oracle.rms_norm(x, g)
    y_from_xn = oracle.masked_ffn(xn, wg, wu, wd, np.ones(12), None)
    assert np.max(np.abs((y - x) - (y_from_xn - xn))) < 1e-13


def _brute_force_gathered(x, wg, wu, wd, idx, count):
    """Scalar loops over the active list only (the gathered form), with math.exp."""
    T, d = len(x), len(x[0])
    y = [[float(x[t][c]) for c in range(d)] for t in range(T)]
    for t in range(T):
        for i in range(count):
            n = int(idx[i])
            gsum = sum(float(wg[n][j]) * float(x[t][j]) for j in range(d))
            usum = sum(float(wu[n][j]) * float(x[t][j]) for j in range(d))
            h = gsum / (1.0 + math.exp(-gsum)) * usum
            for c in range(d):
                y[t][c] += h * float(wd[n][c])
    return np.array(y)


def test_brute_force_tiny_all_masks():
    # d_ff = 6: all 64 masks, d = 5, T = 2.
    wg, wu, wd, _ = _rand_layer(22, 5, 6)
    x = np.random.default_rng(23).standard_normal((2, 5))
    for bits in itertools.product([0, 1], repeat=6):
        m = np.array(bits, np.uint8)
        idx, cnt = oracle.compact_mask(m)
        got = oracle.masked_ffn(x, wg, wu, wd, oracle.mask_multiplicity(m))
        assert np.max(np.abs(got - _brute_force_gathered(x, wg, wu, wd, idx, int(cnt)))) < 1e-12


def test_brute_force_tiny_random_lists():
    for seed in range(5):
        r = np.random.default_rng(100 + seed)
        d, d_ff, T = int(r.integers(1, 17)), int(r.integers(1, 33)), int(r.integers(1, 4))
        wg, wu, wd, _ = _rand_layer(seed, d, d_ff)
        x = r.standard_normal((T, d))
        cnt = int(r.integers(0, 2 * d_ff))
        idx = r.integers(0, d_ff, size=cnt).astype(np.int32)  # a multiset, possibly with repeats
        got = oracle.masked_ffn(x, wg, wu, wd, oracle.multiplicity(idx, cnt, d_ff))
        assert np.max(np.abs(got - _brute_force_gathered(x, wg, wu, wd, idx, cnt))) < 1e-12


def test_bf16_weights_are_exact_widenings():
    layer = wl.make_layer(99, 0, 16, 8, "bf16")
    wg, _, _, _ = layer.f64()
    # Every value is a bf16: at most 8 significant bits.
    m, _ = np.frexp(wg)
    assert np.array_equal(m * 256, np.round(m * 256))
    t = torch.tensor(wg, dtype=torch.float64)
    assert np.array_equal(t.to(torch.bfloat16).to(torch.float64).numpy(), wg)


def test_bf16_rounding_matches_torch():
    a = np.random.default_rng(24).standard_normal(20000) * 3
    ours = wl.bf16_bits_to_f64(wl.bf16_bits(a))
    ref = torch.tensor(a.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(ours, ref)


# ------------------------------------------------------------------------------------------------ Eq. 4

def test_local_update_full_mask_gives_current_dense_output():
    # With every neuron selected, y_a + (h_t - h_a) W = h_t W: the dense FFN output at the current input,
    # whatever the anchor.
    wg, wu, wd, g = _rand_layer(25, 10, 14, True)
    r = np.random.default_rng(26)
    xa, xt = r.standard_normal((3, 10)), r.standard_normal((3, 10))
    ha, ht = oracle.hidden(xa, wg, wu, g), oracle.hidden(xt, wg, wu, g)
    ya = ha @ wd
    got = oracle.local_update(ya, ht, ha, np.ones(14), wd)
    ref = _torch_swiglu(xt, wg, wu, wd, g) - xt
    assert np.max(np.abs(got - ref)) < 1e-13


def test_local_update_special_cases():
    wg, wu, wd, _ = _rand_layer(27, 6, 9)
    r = np.random.default_rng(28)
    xa, xt = r.standard_normal((2, 6)), r.standard_normal((2, 6))
    ha, ht = oracle.hidden(xa, wg, wu), oracle.hidden(xt, wg, wu)
    ya = ha @ wd
    # Empty mask: the anchor output is reused unchanged.
    assert np.array_equal(oracle.local_update(ya, ht, ha, np.zeros(9), wd), ya)
    # Zero anchor: the masked FFN's delta.
    m = wl.bernoulli_mask(r, (9,), 0.5).astype(float)
    got = oracle.local_update(np.zeros_like(ya), ht, np.zeros_like(ht), m, wd)
    assert np.max(np.abs(got - (oracle.masked_ffn(xt, wg, wu, wd, m) - xt))) < 1e-14


def _torch_dense_chain(x, layers):
    outs = [np.asarray(x, np.float64)]
    for wg, wu, wd, g in layers:
        outs.append(_torch_swiglu(outs[-1], wg, wu, wd, g))
    return outs


def test_anchor_stack_keeps_dense_outputs_and_activations():
    layers = [_rand_layer(40 + l, 8, 12, True) for l in range(3)]
    x = np.random.default_rng(43).standard_normal((2, 5, 8))
    y, ya, ha = oracle.anchor_stack(x, layers)
    outs = _torch_dense_chain(x, layers)
    assert np.max(np.abs(y - outs[-1])) < 1e-12
    for l, (wg, wu, wd, g) in enumerate(layers):
        # y_a is the layer's FFN output before the residual; h_a its activations at the layer's input.
        assert np.max(np.abs(ya[l] - (outs[l + 1] - outs[l]))) < 1e-12
        xn = F.rms_norm(torch.tensor(outs[l]), (8,), weight=torch.tensor(g), eps=1e-6)
        h = (F.silu(F.linear(xn, torch.tensor(wg))) * F.linear(xn, torch.tensor(wu))).numpy()
        assert np.max(np.abs(ha[l] - h)) < 1e-12


def _brute_eq4_layer(x, layer, mask, ya, ha, eps=1e-6):
    """Eq. 4 for one layer by scalar loops: x + y_a + sum over masked n of (h_t[n] - h_a[n]) W_down[n]."""
    wg, wu, wd, g = layer
    T, d = len(x), len(x[0])
    out = []
    for t in range(T):
        ms = sum(x[t][j] * x[t][j] for j in range(d)) / d
        xn = [x[t][j] / math.sqrt(ms + eps) * g[j] for j in range(d)]
        row = []
        for c in range(d):
            acc = ya[t][c]
            for n in range(len(wg)):
                if mask[n]:
                    a = sum(wg[n][j] * xn[j] for j in range(d))
                    u = sum(wu[n][j] * xn[j] for j in range(d))
                    h = a / (1.0 + math.exp(-a)) * u
                    acc += (h - ha[t][n]) * wd[n][c]
            row.append(x[t][c] + acc)
        out.append(row)
    return np.array(out)


def test_delta_stack_matches_brute_force_eq4():
    layer = _rand_layer(44, 3, 5, True)
    r = np.random.default_rng(45)
    xa, xt = r.standard_normal((2, 3)), r.standard_normal((2, 3))
    _, ya, ha = oracle.anchor_stack(xa, [layer])
    mask = np.array([1, 0, 1, 1, 0])
    got = oracle.delta_stack(xt, [layer], [mask.astype(float)], ya, ha)
    ref = _brute_eq4_layer(xt.tolist(), layer, mask, ya[0].tolist(), ha[0].tolist())
    assert np.max(np.abs(got - ref)) < 1e-13


def test_delta_stack_special_cases():
    layers = [_rand_layer(46 + l, 8, 12, True) for l in range(3)]
    r = np.random.default_rng(49)
    xa = r.standard_normal((4, 8))
    xt = xa + 0.05 * r.standard_normal((4, 8))
    y_anchor, ya, ha = oracle.anchor_stack(xa, layers)
    masks = [wl.bernoulli_mask(r, (12,), 0.4).astype(float) for _ in range(3)]
    # At the anchor's own input every layer reproduces the anchor, whatever the masks.
    assert np.array_equal(oracle.delta_stack(xa, layers, masks, ya, ha), y_anchor)
    # Every neuron selected: the dense stack at the current input.
    full = oracle.delta_stack(xt, layers, [np.ones(12)] * 3, ya, ha)
    assert np.max(np.abs(full - _torch_dense_chain(xt, layers)[-1])) < 1e-12
    # No neuron selected: each layer adds its anchor output to its own input.
    empty = oracle.delta_stack(xt, layers, [np.zeros(12)] * 3, ya, ha)
    assert np.array_equal(empty, ((xt + ya[0]) + ya[1]) + ya[2])
    # Zero anchor: the masked stack.
    zero = oracle.delta_stack(xt, layers, masks, np.zeros_like(ya), np.zeros_like(ha))
    assert np.max(np.abs(zero - oracle.ffn_stack(xt, layers, masks))) < 1e-12


# ------------------------------------------------------------------------------------------------ stacks

def test_stack_reduces_to_layers_and_identity():
    layers = [_rand_layer(30 + l, 8, 12, True) for l in range(3)]
    x = np.random.default_rng(33).standard_normal((4, 8))
    r = np.random.default_rng(34)
    mults = [wl.bernoulli_mask(r, (12,), 0.5).astype(float) for _ in range(3)]
    ref = x
    for (wg, wu, wd, g), m in zip(layers, mults):
        ref = _torch_swiglu(ref, wg, wu, wd, g, zero_down_rows=np.flatnonzero(m == 0))
    assert np.max(np.abs(oracle.ffn_stack(x, layers, mults) - ref)) < 1e-12
    assert np.array_equal(oracle.ffn_stack(x, layers, [np.zeros(12)] * 3), x)


# ------------------------------------------------------------------------------------------------ masks

def test_topk_mask_ties_and_nesting():
    s = np.array([0.5, 2.0, 0.5, 2.0, 1.0, 0.5])
    assert oracle.topk_mask(s, 1).tolist() == [0, 1, 0, 0, 0, 0]
    assert oracle.topk_mask(s, 3).tolist() == [0, 1, 0, 1, 1, 0]
    assert oracle.topk_mask(s, 4).tolist() == [1, 1, 0, 1, 1, 0]  # tie at 0.5 -> lowest index
    ms = oracle.nested_topk_masks(np.random.default_rng(35).standard_normal(100), [10, 30, 50, 100])
    assert ms.sum(axis=1).tolist() == [10, 30, 50, 100]
    assert all(((ms[i] == 1) <= (ms[i + 1] == 1)).all() for i in range(3))


def test_contribution_score_hand_example():
    # Eq. 1: neuron 0 has |h| summing to 3 and a down row of norm 5; neuron 1 sums to 1 with norm 1.
    h = np.array([[1.0, -0.5], [-2.0, 0.5]])
    wd = np.array([[3.0, 4.0], [0.0, -1.0]])
    assert oracle.contribution_score(h, wd).tolist() == [15.0, 1.0]


def test_mean_abs_activation_matches_torch():
    wg, wu, wd, g = _rand_layer(36, 8, 10, True)
    x = np.random.default_rng(37).standard_normal((5, 8))
    xt = torch.tensor(x)
    xn = F.rms_norm(xt, (8,), weight=torch.tensor(g), eps=1e-6)
    h = F.silu(F.linear(xn, torch.tensor(wg))) * F.linear(xn, torch.tensor(wu))
    assert np.max(np.abs(oracle.mean_abs_activation(x, wg, wu, g) - h.abs().mean(0).numpy())) < 1e-14


def test_budget_rule():
    # K = ceil(rho * H): the paper's top-k of 2048 at rho = 0.5 and H = 4096, and the workload counts.
    assert oracle.ceil_budget(1, 2, 4096) == 2048
    assert oracle.ceil_budget(3, 10, 4096) == 1229
    assert oracle.ceil_budget(1, 4, 1024) == 256
    assert [oracle.ceil_budget(p, 100, 16384) for p in (10, 30, 50, 100)] == [1639, 4916, 8192, 16384]
    assert oracle.ceil_budget(18, 100, 4096) == 738
    assert [wl.count_for_percent(p, 16384) for p in (10, 30, 50, 100)] == [1639, 4916, 8192, 16384]


def test_rel_err():
    assert oracle.rel_err(np.array([1.0, 2.0]), np.array([1.0, 2.0])) == 0.0
    assert oracle.rel_err(np.array([1.0, 2.5]), np.array([1.0, 2.0])) == 0.25
    assert oracle.rel_err(np.zeros(3), np.zeros(3)) == 0.0
