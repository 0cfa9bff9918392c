"""GPU parity of the group-mask construction (section 5, "Constructing Group Neuron Masks"; Eq. 1) against the
float64 oracle (oracle.group_masks), on the same seeded inputs.

Bars:
- the float32 row norms and Eq. 1 scores within `norm_rel_bound(d)` / `score_rel_bound(T)` of the float64
  values (rounding bounds that hold for any summation order);
- each layer's mask exactly the section-5 decision taken on the GPU's own float32 scores (per-step top K, union,
  top K by summed score, ties to the lower neuron; the sum over steps allowed its float32 rounding), and a valid
  group mask for the float64 scores given their bound (`check_group_mask`);
- where every sum is exact in float32 (activations on a dyadic grid, unit norms), the scores equal the float64
  values exactly, the decision is unique, and the masks equal the oracle's bit for bit;
- repeated calls bit for bit equal."""
import numpy as np
import pytest
import torch

import workloads as wl
from oracle import group_masks as gm

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2609_19104_amd as rm  # noqa: E402
from gpu_helpers import dev_weights  # noqa: E402


@pytest.mark.parametrize("wdtype", ["bf16", "f32"])
@pytest.mark.parametrize("d,d_ff", [(32, 1), (96, 63), (1024, 65), (1024, 4096), (2048, 300)])
def test_neuron_norms(wdtype, d, d_ff):
    layer = wl.make_layer(91, d_ff, d, d_ff, wdtype)
    wd = dev_weights(layer)[2]
    runs = []
    for _ in range(2):
        norms = torch.full((d_ff,), float("nan"), device="cuda")
        rm.rm_neuron_norms(wd, norms)
        runs.append(norms.cpu().numpy())
    assert np.array_equal(runs[0].view(np.uint32), runs[1].view(np.uint32))
    ref = gm.neuron_norms(wl.storage_to_f64(layer.w_down))
    err = np.max(np.abs(runs[0] - ref) / ref)
    print(f"norms: max rel err {err:.2e} (bound {gm.norm_rel_bound(d):.2e})")
    assert err <= gm.norm_rel_bound(d)


def _run(h, norms, k):
    S, L, d_ff, _ = h.shape
    ht, nt = torch.from_numpy(h).cuda(), torch.from_numpy(norms).cuda()
    scores = torch.full((S, L, d_ff), float("nan"), device="cuda")
    mask = torch.full((L, d_ff), 7, dtype=torch.uint8, device="cuda")
    rm.rm_group_masks(ht, nt, k, scores, mask)
    torch.cuda.synchronize()
    return scores.cpu().numpy(), mask.cpu().numpy()


CASES = [
    # S, L, d_ff, T, K, quantum (> 0: many tied scores)
    (1, 1, 1, 1, 1, 0.0),
    (2, 1, 17, 7, 5, 0.0),
    (3, 2, 1000, 51, 300, 0.0),
    (5, 3, 4096, 51, 1229, 0.0),
    (5, 2, 4096, 51, 1229, 0.5),
    (4, 1, 4095, 33, 2048, 1.0),
    (2, 1, 4097, 9, 2000, 1.0),     # just past the 256-thread selection: 1024 threads
    (2, 2, 300, 65, 100, 0.0),      # T past one 64-token chunk: the sums continue across chunks
    (1, 1, 130, 130, 40, 0.5),
    (2, 2, 16384, 8, 4916, 0.0),
    (3, 1, 16384, 4, 8192, 2.0),
    (1, 2, 777, 64, 776, 0.0),
    (2, 1, 512, 10, 0, 0.0),
    (2, 1, 512, 10, 512, 0.0),
]


def _fuzz_cases(n=8, seed=19104):
    # Seeded random shapes: token counts on both sides of one 64-token chunk (odd and even), widths on both sides
    # of the 256-thread selection, K from 0 to d_ff, with and without ties.
    rng = np.random.default_rng(seed)
    for _ in range(n):
        d_ff = int(rng.choice([int(rng.integers(1, 300)), int(rng.integers(3000, 6000))]))
        yield (int(rng.integers(1, 6)), int(rng.integers(1, 4)), d_ff, int(rng.integers(1, 140)),
               int(rng.integers(0, d_ff + 1)), float(rng.choice([0.0, 0.5])))


def _check_masks(h, norms, K, scores, mask, exact):
    S, L, d_ff, T = h.shape
    bound = gm.score_rel_bound(T)
    for l in range(L):
        c64 = np.stack([gm.contribution_scores(h[s, l], norms[l]) for s in range(S)])
        got = scores[:, l].astype(np.float64)
        if exact:
            assert np.array_equal(got, c64), l
            assert np.array_equal(mask[l], gm.group_mask(h[:, l], norms[l], K)), l
        else:
            pos = c64 > 0
            assert np.all(got[~pos] == 0.0)
            assert np.max(np.abs(got[pos] - c64[pos]) / c64[pos]) <= bound, l
        gm.check_group_mask(mask[l], got, K, rel=0.0)  # the decision on its own values
        gm.check_group_mask(mask[l], c64, K, rel=bound)
    assert np.all(mask.sum(axis=1) == K)


@pytest.mark.parametrize("S,L,d_ff,T,K,quantum", CASES + list(_fuzz_cases()))
def test_group_masks(S, L, d_ff, T, K, quantum):
    h = wl.activation_like(92, (S, L, d_ff, T), d_ff, T, quantum=quantum)
    norms = wl.positive_norms(92, (L, d_ff), d_ff)
    if quantum > 0:
        norms[:] = 1.0  # every sum exact: the scores equal the float64 ones and ties are true ties
    scores, mask = _run(h, norms, K)
    _check_masks(h, norms, K, scores, mask, exact=quantum > 0)
    scores2, mask2 = _run(h, norms, K)
    assert np.array_equal(scores.view(np.uint32), scores2.view(np.uint32)) and np.array_equal(mask, mask2)


def test_group_masks_from_identity_list_anchor():
    # End to end on the device: each step's dense activations from rm_anchor_ffn_stack run with the identity
    # lists, then the group masks.  Checked by properties only (the activations are GPU results, so they are
    # not handed to the oracle): K neurons per layer, each of them among some step's K best by the returned
    # scores, and the scores non-negative and finite.
    d, d_ff, L, T, S, K = 256, 1024, 2, 51, 3, 307
    layers = [wl.make_layer(93, l, d, d_ff, "bf16", norm="ones") for l in range(L)]
    lws = [dev_weights(x) for x in layers]
    idx = torch.arange(d_ff, dtype=torch.int32, device="cuda").repeat(L, 1).contiguous()
    cnt = torch.full((L,), d_ff, dtype=torch.int32, device="cuda")
    ws = rm.workspace(d, d_ff, rm.RM_BF16, 1, T, d_ff)
    hs = torch.empty((S, L, d_ff, T), device="cuda")
    for s in range(S):
        x = torch.from_numpy(wl.make_x(93, (1, T, d), s)).cuda()
        y = torch.empty_like(x)
        ya = torch.empty((L, 1, T, d), device="cuda")
        ha = torch.empty((L, 1, d_ff, T), device="cuda")
        rm.rm_anchor_ffn_stack(x, y, lws, idx, cnt, d_ff, ya, ha, ws)
        hs[s] = ha[:, 0]
    norms = torch.empty((L, d_ff), device="cuda")
    for l in range(L):
        rm.rm_neuron_norms(lws[l][2], norms[l])
    scores = torch.empty((S, L, d_ff), device="cuda")
    mask = torch.empty((L, d_ff), dtype=torch.uint8, device="cuda")
    rm.rm_group_masks(hs, norms, K, scores, mask)
    torch.cuda.synchronize()
    sc, m = scores.cpu().numpy(), mask.cpu().numpy()
    assert np.all(np.isfinite(sc)) and np.all(sc >= 0)
    assert np.all(m.sum(axis=1) == K)
    for l in range(L):
        cand = np.zeros(d_ff, bool)
        for s in range(S):
            cand[np.argsort(-sc[s, l], kind="stable")[:K]] = True
        assert np.all(cand[m[l] != 0])


@pytest.mark.parametrize("S,L,d_ff,T,K", [(5, 2, 4096, 51, 1229), (3, 1, 1000, 20, 100)])
def test_step_specific_against_group_shared_coverage(S, L, d_ff, T, K):
    # Section 5 shares one mask across a group; section 3.4's coverage measures what a mask keeps of a step's
    # contribution.  Each step alone (S = 1) gives its own top-K mask; the group call gives the shared one.  Both
    # masks are checked as above, and the shared mask never covers more of a step's float64 contribution than the
    # step's own, up to the scores' rounding allowance (a float32 top K can swap near-tied neurons).
    h = wl.activation_like(94, (S, L, d_ff, T), d_ff, T)
    norms = wl.positive_norms(94, (L, d_ff), d_ff)
    scores, group = _run(h, norms, K)
    _check_masks(h, norms, K, scores, group, exact=False)
    bound = gm.score_rel_bound(T)
    for s in range(S):
        h1 = np.ascontiguousarray(h[s:s + 1])
        s_scores, own = _run(h1, norms, K)
        _check_masks(h1, norms, K, s_scores, own, exact=False)
        for l in range(L):
            c = gm.contribution_scores(h[s, l], norms[l])
            cov_own, cov_group = gm.coverage(c, own[l]), gm.coverage(c, group[l])
            assert 0.0 < cov_group <= cov_own * (1.0 + 2.0 * bound) <= 1.0 + 2.0 * bound
