"""Pins for the group-mask oracle (section 5, "Constructing Group Neuron Masks"; Eq. 1 of section 3.4).

Each pin checks the oracle against something fixed independently of it: torch's library vector norms, values
worked out by hand, float32 evaluations in several orders (for the rounding bounds), exhaustive search over
subsets, or a small example worked out by hand.  The mask checker is pinned by planting mistakes in valid masks."""
import itertools

import numpy as np
import pytest
import torch

from oracle import group_masks as gm


def test_neuron_norms_match_library_norm():
    w = np.random.default_rng(1).standard_normal((37, 300)).astype(np.float32) * 0.02
    ref = torch.linalg.vector_norm(torch.tensor(w, dtype=torch.float64), dim=1).numpy()
    assert np.max(np.abs(gm.neuron_norms(w) - ref) / ref) < 1e-14
    assert gm.neuron_norms(np.array([[3.0, 4.0], [0.0, 0.0]])).tolist() == [5.0, 0.0]


def test_scores_match_library_norms_and_hand_values():
    # Eq. 1 as two library norms: the L1 norm of the neuron's activations times the L2 norm of its down row.
    r = np.random.default_rng(2)
    h = r.standard_normal((50, 17)).astype(np.float32)  # [d_ff][T]
    wd = r.standard_normal((50, 64)).astype(np.float32)
    ht, wt = torch.tensor(h, dtype=torch.float64), torch.tensor(wd, dtype=torch.float64)
    ref = (torch.linalg.vector_norm(ht, ord=1, dim=1) * torch.linalg.vector_norm(wt, dim=1)).numpy()
    got = gm.contribution_scores(h, gm.neuron_norms(wd))
    assert np.max(np.abs(got - ref) / ref) < 1e-14
    # By hand: |1| + |-2| + |0.5| = 3.5 times ||(3, 4)|| = 5 -> 17.5; the sign of h does not matter.
    hh = np.array([[1.0, -2.0, 0.5], [-1.0, 2.0, -0.5]])
    assert gm.contribution_scores(hh, gm.neuron_norms(np.array([[3.0, 4.0], [0.0, 2.0]]))).tolist() == [17.5, 7.0]


def _f32_scores(h, norms, order):
    """Eq. 1 in float32, one rounding per operation, |h| summed over t forward or backward: evaluations a float32
    kernel could perform."""
    h = np.abs(np.asarray(h, np.float32))
    ts = range(h.shape[1]) if order == "forward" else range(h.shape[1] - 1, -1, -1)
    s = np.zeros(h.shape[0], np.float32)
    for t in ts:
        s = (s + h[:, t]).astype(np.float32)
    return (s * np.asarray(norms, np.float32)).astype(np.float32)


@pytest.mark.parametrize("T", [1, 51, 130])
def test_score_and_norm_bounds_cover_float32_evaluations(T):
    r = np.random.default_rng(T)
    h = (r.standard_normal((200, T)) * np.exp(2 * r.standard_normal((200, T)))).astype(np.float32)
    wd = (r.standard_normal((200, 2048)) * np.exp(r.standard_normal((200, 2048)))).astype(np.float32)
    n64 = gm.neuron_norms(wd)
    sq = (wd * wd).astype(np.float32)
    for cols in (range(2048), range(2047, -1, -1)):
        s = np.zeros(200, np.float32)
        for j in cols:
            s = (s + sq[:, j]).astype(np.float32)
        n32 = np.sqrt(s).astype(np.float32)
        assert np.max(np.abs(n32 - n64) / n64) <= gm.norm_rel_bound(2048)
    norms = n64.astype(np.float32)  # the scores' norms as float32 inputs
    ref = gm.contribution_scores(h, norms)
    for order in ("forward", "backward"):
        err = np.max(np.abs(_f32_scores(h, norms, order) - ref) / ref)
        assert err <= gm.score_rel_bound(T), (order, err)


def test_top_k_matches_stable_sort_and_breaks_ties_low():
    s = np.array([3, 1, 3, 2, 3, 0], np.float32)
    assert np.flatnonzero(gm.top_k(s, 2)).tolist() == [0, 2]
    assert np.flatnonzero(gm.top_k(s, 4)).tolist() == [0, 2, 3, 4]
    assert gm.top_k(s, 0).sum() == 0 and gm.top_k(s, 9).sum() == 6
    r = np.random.default_rng(3)
    for _ in range(20):
        v = r.integers(0, 5, size=40).astype(np.float32)
        k = int(r.integers(0, 41))
        ref = np.zeros(40, bool)
        ref[np.argsort(-v, kind="stable")[:k]] = True
        assert np.array_equal(gm.top_k(v, k), ref)


def test_worked_example():
    # Two steps, five neurons, two actions, K = 2, unit down-projection rows (norm 1).
    # Step 0 sums |h| = [3, 4, 1, 0, 2] -> candidates {1, 0}; step 1 sums = [0, 1, 5, 4, 2] -> {2, 3}.
    # Summed over the steps: [3, 5, 6, 4, 4]; among the union {0, 1, 2, 3} the top two are 2 (6) and 1 (5).
    h = np.array([[[1, -2], [4, 0], [0, 1], [0, 0], [1, 1]],
                  [[0, 0], [-1, 0], [2, 3], [4, 0], [1, -1]]], np.float32)
    norms = np.ones(5, np.float32)
    assert np.flatnonzero(gm.group_mask(h, norms, 2)).tolist() == [1, 2]
    # K = 3: step 0's top 3 = {1, 0, 4}, step 1's = {2, 3, 4}, so the union is all five neurons;
    # summed top 3 = 2 (6), 1 (5), then 3 and 4 tie at 4 -> the lower index, 3.
    assert np.flatnonzero(gm.group_mask(h, norms, 3)).tolist() == [1, 2, 3]


def _brute_group_mask(c_steps, k):
    """Exhaustive form: the K-subset of the union with the largest summed score (distinct sums)."""
    n = c_steps.shape[1]
    union = set()
    for c in c_steps:
        best = max(itertools.combinations(range(n), k), key=lambda sub: sum(float(c[i]) for i in sub))
        union |= set(best)
    tot = c_steps.astype(np.float64).sum(axis=0)
    best = max(itertools.combinations(sorted(union), k), key=lambda sub: sum(tot[i] for i in sub))
    m = np.zeros(n, np.uint8)
    m[list(best)] = 1
    return m


@pytest.mark.parametrize("seed", range(6))
def test_group_mask_matches_exhaustive_search(seed):
    r = np.random.default_rng(10 + seed)
    S, n, T, k = int(r.integers(1, 4)), 8, 3, int(r.integers(1, 5))
    h = r.standard_normal((S, n, T)).astype(np.float32)
    norms = (0.5 + r.random(n)).astype(np.float32)
    c = np.stack([gm.contribution_scores(hs, norms) for hs in h])
    assert np.array_equal(gm.group_mask(h, norms, k), _brute_group_mask(c, k))


def test_group_mask_special_cases():
    r = np.random.default_rng(20)
    h = r.standard_normal((1, 64, 5)).astype(np.float32)
    norms = (0.5 + r.random(64)).astype(np.float32)
    c = gm.contribution_scores(h[0], norms)
    # One step: the group mask is that step's top K.
    assert np.array_equal(gm.group_mask(h, norms, 20).astype(bool), gm.top_k(c, 20))
    # Identical steps: the same.
    assert np.array_equal(gm.group_mask(np.repeat(h, 4, axis=0), norms, 20).astype(bool), gm.top_k(c, 20))
    # K = 0 and K = d_ff.
    assert gm.group_mask(h, norms, 0).sum() == 0 and gm.group_mask(h, norms, 64).sum() == 64
    # Always exactly K neurons, all of them some step's candidate.
    hs = r.standard_normal((3, 64, 5)).astype(np.float32)
    m = gm.group_mask(hs, norms, 17)
    assert m.sum() == 17
    cand = np.zeros(64, bool)
    for x in hs:
        cand |= gm.top_k(gm.contribution_scores(x, norms), 17)
    assert np.all(cand[m != 0])


def test_coverage_pins():
    # Section 3.4's coverage: the share of a step's summed contribution held by the masked neurons.  A full mask
    # holds all of it, an empty one none, and a single neuron its own share.
    c = np.array([4.0, 1.0, 0.0, 3.0], dtype=np.float32)
    assert gm.coverage(c, np.ones(4, np.uint8)) == 1.0
    assert gm.coverage(c, np.zeros(4, np.uint8)) == 0.0
    assert gm.coverage(c, np.array([0, 0, 0, 1], np.uint8)) == 3.0 / 8.0
    assert gm.coverage(np.zeros(3, np.float32), np.ones(3, np.uint8)) == 0.0


@pytest.mark.parametrize("seed", range(4))
def test_step_top_k_has_the_best_coverage_of_any_k_subset(seed):
    # Brute force on 9 neurons: no K-subset covers more of a step than that step's own top K, so a mask shared
    # by a group can only match or lose coverage against the step-specific one.
    rng = np.random.default_rng(seed)
    c = rng.exponential(size=9).astype(np.float32)
    k = 3
    best = max(gm.coverage(c, np.isin(np.arange(9), s)) for s in itertools.combinations(range(9), k))
    assert gm.coverage(c, gm.top_k(c, k)) == pytest.approx(best, rel=1e-12)


def test_check_group_mask_accepts_valid_and_catches_planted_mistakes():
    # Two steps, six neurons, K = 2.  Step 0: top two {0, 1}; step 1: top two {2, 1}.  Union {0, 1, 2}; summed
    # scores 10.5, 14, 9, ... -> the mask {0, 1}.
    c = np.array([[10.0, 9.0, 1.0, 0.5, 0.2, 0.1],
                  [0.5, 5.0, 8.0, 3.0, 0.1, 0.2]])
    good = np.array([1, 1, 0, 0, 0, 0], np.uint8)
    gm.check_group_mask(good, c, 2, rel=1e-6)
    bad = [
        np.array([1, 1, 1, 0, 0, 0], np.uint8),  # three neurons
        np.array([1, 0, 1, 0, 0, 0], np.uint8),  # 2 (summed 9) kept over 1 (summed 14)
        np.array([1, 0, 0, 1, 0, 0], np.uint8),  # 3 is no step's candidate
    ]
    for m in bad:
        with pytest.raises(AssertionError):
            gm.check_group_mask(m, c, 2, rel=1e-6)
    # Within the allowance either order is valid: neurons 0 and 1 summed 10.5 and 10.5 * (1 + 1e-9).
    c2 = np.array([[10.0, 10.0 * (1 + 1e-9), 1.0], [0.5, 0.5, 0.2]])
    for m in ([1, 0, 0], [0, 1, 0]):
        gm.check_group_mask(np.array(m, np.uint8), c2, 1, rel=1e-6)
    # The oracle's own masks pass on random inputs.
    r = np.random.default_rng(30)
    for _ in range(10):
        h = r.standard_normal((3, 40, 5))
        norms = 0.5 + r.random(40)
        k = int(r.integers(1, 40))
        cs = np.stack([gm.contribution_scores(x, norms) for x in h])
        gm.check_group_mask(gm.group_mask(h, norms, k), cs, k, rel=0.0)
