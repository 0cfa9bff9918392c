"""Pins for the Context Cache oracle (section 4.1, "Visual-Token Recomputation": Eq. 2 drift, Eq. 3 update).

Each pin checks the oracle against something fixed independently of it: a value worked out by hand, exact special
cases, torch's library vector norm, float32 evaluations in several summation orders (for the rounding bound), a
stable sort, or torch's library FFN.  The selection checker is pinned by planting mistakes in valid selections."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import context_cache as cc


def test_drift_hand_example():
    # x = (3, 4), xbar = (3, 0): RMS(x - xbar) = sqrt(16 / 2), RMS(x) = sqrt(25 / 2), d = sqrt(16 / 25) = 0.8.
    assert cc.drift(np.array([[3.0, 4.0]]), np.array([[3.0, 0.0]]))[0] == pytest.approx(0.8, rel=1e-15)
    # x = (1, 1, 1, 1), xbar = (1, -1, 1, -1): diff (0, 2, 0, 2) -> RMS sqrt(2); RMS(x) = 1.
    assert cc.drift(np.ones((1, 4)), np.array([[1.0, -1, 1, -1]]))[0] == pytest.approx(np.sqrt(2.0), rel=1e-15)


@pytest.mark.parametrize("d", [32, 96, 2048])
def test_drift_matches_torch_vector_norms(d):
    # RMS(v) = ||v||_2 / sqrt(d): torch's library 2-norm, a routine the oracle does not use.
    r = np.random.default_rng(d)
    x = r.standard_normal((40, d)).astype(np.float32)
    xr = (x + r.standard_normal((40, d)) * r.random((40, 1))).astype(np.float32)
    xt, xrt = torch.tensor(x, dtype=torch.float64), torch.tensor(xr, dtype=torch.float64)
    ref = (torch.linalg.vector_norm(xt - xrt, dim=1) / torch.linalg.vector_norm(xt, dim=1)).numpy()
    assert np.max(np.abs(cc.drift(x, xr) - ref) / ref) < 1e-13


def test_drift_exact_special_cases():
    r = np.random.default_rng(1)
    x = r.standard_normal((8, 128)).astype(np.float32)
    xr = r.standard_normal((8, 128)).astype(np.float32)
    assert np.all(cc.drift(x, x) == 0)                   # no drift
    assert np.allclose(cc.drift(x, np.zeros_like(x)), 1.0, rtol=1e-15, atol=0)  # x - 0 = x
    assert np.array_equal(cc.drift(2 * x, 2 * xr), cc.drift(x, xr))  # scaling by 2 is exact throughout
    z = np.zeros((1, 128), np.float32)  # RMS(x) = 0 < eps: the denominator is eps
    rms_ref = np.sqrt(np.sum(xr[:1].astype(np.float64) ** 2) / 128)
    assert cc.drift(z, xr[:1])[0] == pytest.approx(rms_ref / 1e-6, rel=1e-14)


def _drift_f32(x, xr, order):
    """Eq. 2 in float32 with one rounding per operation, the sums of squares taken in the given column order or
    pairwise: evaluations a float32 kernel could perform."""
    x, xr = np.asarray(x, np.float32), np.asarray(xr, np.float32)
    diff = (x - xr).astype(np.float32)

    def ssq(v):
        sq = (v * v).astype(np.float32)
        if order == "pairwise":
            while sq.shape[1] > 1:
                if sq.shape[1] % 2:
                    sq = np.concatenate([sq, np.zeros((sq.shape[0], 1), np.float32)], axis=1)
                sq = (sq[:, 0::2] + sq[:, 1::2]).astype(np.float32)
            return sq[:, 0]
        cols = range(v.shape[1]) if order == "forward" else range(v.shape[1] - 1, -1, -1)
        s = np.zeros(v.shape[0], np.float32)
        for j in cols:
            s = (s + sq[:, j]).astype(np.float32)
        return s

    d = np.float32(x.shape[1])
    rd = np.sqrt((ssq(diff) / d).astype(np.float32)).astype(np.float32)
    rx = np.sqrt((ssq(x) / d).astype(np.float32)).astype(np.float32)
    return (rd / np.maximum(rx, np.float32(1e-6))).astype(np.float32)


@pytest.mark.parametrize("d", [32, 1000, 2048])
def test_drift_rel_bound_covers_float32_evaluations(d):
    # The bound must hold for every order; the orders tried here are ordinary kernel choices.  Values with a large
    # dynamic range within a row make the sums lose the most.
    r = np.random.default_rng(d + 5)
    x = (r.standard_normal((64, d)) * np.exp(2 * r.standard_normal((64, d)))).astype(np.float32)
    xr = (x + r.standard_normal((64, d)) * np.exp(r.standard_normal((64, 1)))).astype(np.float32)
    ref = cc.drift(x, xr)
    bound = cc.drift_rel_bound(d)
    for order in ("forward", "backward", "pairwise"):
        err = np.max(np.abs(_drift_f32(x, xr, order).astype(np.float64) - ref) / ref)
        assert err <= bound, (order, err, bound)
    assert bound < 1e-3  # tight enough to decide between the workloads' distinct drifts


def test_recomputed_rows_hand_example_and_sort():
    # Tokens 0-1 are text, 2-6 visual (P = 5), 7 is state; k = 2 of the visual ones: scores 0.5, 0.9, 0.1, 0.9,
    # 0.2 -> the two 0.9s (visual 1 and 3 -> rows 3 and 5), the tie broken to the lower token.
    s = np.array([0.5, 0.9, 0.1, 0.9, 0.2])
    assert cc.recomputed_rows(s, 8, 2, 2).tolist() == [0, 1, 3, 5, 7]
    assert cc.recomputed_rows(s, 8, 2, 0).tolist() == [0, 1, 7]
    assert cc.recomputed_rows(s, 8, 2, 5).tolist() == list(range(8))
    r = np.random.default_rng(2)
    for _ in range(20):
        P, v0, n, k = 30, int(r.integers(0, 5)), 40, int(r.integers(0, 31))
        sc = r.integers(0, 6, size=P).astype(np.float64)
        ref = set(range(n)) - set(range(v0, v0 + P)) | set((v0 + np.argsort(-sc, kind="stable")[:k]).tolist())
        assert cc.recomputed_rows(sc, n, v0, k).tolist() == sorted(ref)


def test_check_recomputed_rows_accepts_valid_and_catches_planted_mistakes():
    drift = np.array([0.5, 0.9, 0.1, 0.9 * (1 + 1e-7), 0.2, 0.0, 0.0, 0.0])
    n, v0, k = 12, 2, 3  # visual rows 2 .. 9, text 0-1, state 10-11
    good = cc.recomputed_rows(drift, n, v0, k)
    assert good.tolist() == [0, 1, 2, 3, 5, 10, 11]
    cc.check_recomputed_rows(good, drift, n, v0, k, rel=1e-6)
    # A near tie within the allowance may go either way: visual 1 and 3 differ by 1e-7 relative, so with k = 1
    # either is a valid choice.
    cc.check_recomputed_rows(np.array([0, 1, 3, 10, 11]), drift, n, v0, 1, rel=1e-6)
    cc.check_recomputed_rows(np.array([0, 1, 5, 10, 11]), drift, n, v0, 1, rel=1e-6)
    bad = [
        np.array([0, 1, 2, 3, 4, 10, 11]),      # a clearly smaller drift (0.1) chosen over 0.9
        np.array([0, 1, 2, 3, 5, 10]),          # a state row dropped
        np.array([0, 1, 2, 3, 5, 11, 10]),      # not ascending
        np.array([0, 1, 2, 3, 5, 6, 10, 11]),   # one visual row too many
        np.array([0, 1, 3, 5, 10, 11]),         # one too few
    ]
    for rows in bad:
        with pytest.raises(AssertionError):
            cc.check_recomputed_rows(rows, drift, n, v0, k, rel=1e-6)
    # Zero-drift ties go to the lower token: with k = 6 the last pick is among visual 5, 6, 7 (all zero).
    ok = cc.recomputed_rows(drift, n, v0, 6)
    cc.check_recomputed_rows(ok, drift, n, v0, 6, rel=1e-6)
    with pytest.raises(AssertionError):
        cc.check_recomputed_rows(np.array([0, 1, 2, 3, 4, 5, 6, 9, 10, 11]), drift, n, v0, 6, rel=1e-6)


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
