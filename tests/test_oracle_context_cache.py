"""Pins for the Context Cache oracle (section 4.1, "Visual-Token Recomputation": Eq. 2 drift, Eq. 3 update).

Each pin checks the oracle against something fixed independently of it: the float64 formula, exact special
cases of float32 arithmetic, a stable sort, a hand example, or torch's library FFN."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import context_cache as cc


def _drift64(x, xr):
    x, xr = np.asarray(x, np.float64), np.asarray(xr, np.float64)
    rms = lambda v: np.sqrt(np.mean(v * v, axis=1))  # noqa: E731
    return rms(x - xr) / np.maximum(rms(x), 1e-6)


@pytest.mark.parametrize("d", [32, 96, 2048])
def test_drift_matches_float64_formula(d):
    r = np.random.default_rng(d)
    x = r.standard_normal((40, d)).astype(np.float32)
    xr = (x + r.standard_normal((40, d)) * r.random((40, 1))).astype(np.float32)
    got = cc.drift(x, xr).astype(np.float64)
    assert np.max(np.abs(got - _drift64(x, xr)) / _drift64(x, xr)) < 2e-6


def test_drift_exact_special_cases():
    r = np.random.default_rng(1)
    x = r.standard_normal((8, 128)).astype(np.float32)
    xr = r.standard_normal((8, 128)).astype(np.float32)
    assert np.all(cc.drift(x, x) == 0)                  # no drift
    assert np.all(cc.drift(x, np.zeros_like(x)) == 1)   # x - 0 and x take the same float32 path
    assert np.array_equal(cc.drift(2 * x, 2 * xr), cc.drift(x, xr))  # scaling by 2 is exact throughout
    z = np.zeros((1, 128), np.float32)
    rms_ref = np.sqrt(np.float32(np.sum(xr[:1].astype(np.float64) ** 2) / 128))
    assert abs(float(cc.drift(z, xr[:1])[0]) - rms_ref / 1e-6) / (rms_ref / 1e-6) < 1e-5  # the eps floor


def test_recomputed_rows_hand_example_and_sort():
    # Tokens 0-1 are text, 2-6 visual (P = 5), 7 is state; k = 2 of the visual ones: scores 0.5, 0.9, 0.1, 0.9,
    # 0.2 -> the two 0.9s (visual 1 and 3 -> rows 3 and 5), the tie broken to the lower token.
    s = np.array([0.5, 0.9, 0.1, 0.9, 0.2], np.float32)
    assert cc.recomputed_rows(s, 8, 2, 2).tolist() == [0, 1, 3, 5, 7]
    assert cc.recomputed_rows(s, 8, 2, 0).tolist() == [0, 1, 7]
    assert cc.recomputed_rows(s, 8, 2, 5).tolist() == list(range(8))
    r = np.random.default_rng(2)
    for _ in range(20):
        P, v0, n, k = 30, int(r.integers(0, 5)), 40, int(r.integers(0, 31))
        sc = r.integers(0, 6, size=P).astype(np.float32)
        ref = set(range(n)) - set(range(v0, v0 + P)) | set((v0 + np.argsort(-sc, kind="stable")[:k]).tolist())
        assert cc.recomputed_rows(sc, n, v0, k).tolist() == sorted(ref)


def test_context_update_matches_torch_ffn():
    r = np.random.default_rng(3)
    d, d_ff, n = 32, 64, 12
    wg, wu = r.standard_normal((d_ff, d)) * 0.2, r.standard_normal((d_ff, d)) * 0.2
    wdt = r.standard_normal((d, d_ff)) * 0.2  # nn.Linear down weight [d][d_ff]
    x, y_ref = r.standard_normal((n, d)), r.standard_normal((n, d))
    rows = np.array([1, 4, 5, 11])
    got = cc.context_update(x, y_ref, rows, wg, wu, wdt)
    xt = torch.tensor(x[rows])
    ref = F.linear(F.gelu(F.linear(xt, torch.tensor(wg)), approximate="tanh") * F.linear(xt, torch.tensor(wu)),
                   torch.tensor(wdt)).numpy()
    assert np.max(np.abs(got[rows] - ref)) < 1e-12
    keep = np.setdiff1d(np.arange(n), rows)
    assert np.array_equal(got[keep], y_ref[keep])
    assert np.array_equal(cc.context_update(x, y_ref, np.array([], int), wg, wu, wdt), y_ref)
