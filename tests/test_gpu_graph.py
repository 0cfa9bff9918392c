"""The library's calls captured in a HIP graph (through torch.cuda.CUDAGraph) give the eager results on every
replay.  Replays alternate with eager work and synchronizations; the kernels are deterministic, so every
replay must match the eager output bit for bit.  The cases include the one-launch layer form (one sample at
d = 2048 in its list range, single and stacked, and a single layer at d = 1024), whose per-launch tags must
differ on every replay and every eager launch in between."""
import numpy as np
import pytest
import torch

import oracle
import workloads as wl

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2609_19104_amd as rm  # noqa: E402
from gpu_helpers import TOL_BF16, dev_f32, dev_weights, errors  # noqa: E402


def _setup(L, B, norm, seed, d, d_ff, k):
    T = 51
    layers = [wl.make_layer(seed, l, d, d_ff, "bf16", norm=norm) for l in range(L)]
    x = wl.make_x(seed, (B, T, d), 0)
    masks = np.stack([np.stack([wl.uniform_mask(wl.rng(seed, 4, l, b), d_ff, k) for b in range(B)])
                      for l in range(L)]).reshape(L * B, d_ff)
    return layers, x, masks


@pytest.mark.parametrize("L,B,norm,d,d_ff,k", [
    (1, 1, "none", 512, 1024, 300),
    (3, 2, "ones", 512, 1024, 300),
    (1, 1, "random", 2048, 8192, 3000),  # the one-launch layer form
    (2, 1, "ones", 2048, 8192, 3000),    # the one-launch layer form in a stack
    (1, 1, "random", 1024, 4096, 1229),  # the one-launch layer form at d = 1024
])
def test_graph_replays_match_eager(L, B, norm, d, d_ff, k):
    layers, x, masks = _setup(L, B, norm, 40 + L, d, d_ff, k)
    lws = [dev_weights(l) for l in layers]
    d_ff, d = layers[0].d_ff, layers[0].d
    T = x.shape[1]
    mask_t = torch.from_numpy(masks).cuda()
    idx = torch.empty((L * B, d_ff), dtype=torch.int32, device="cuda")
    cnt = torch.empty((L * B,), dtype=torch.int32, device="cuda")
    xt = dev_f32(x)
    y = torch.empty_like(xt)
    ws = rm.workspace(d, d_ff, rm.RM_BF16, B, T, k, device="cuda")

    def step():
        rm.rm_mask_compact(mask_t, idx, cnt)
        if L == 1:
            rm.rm_sparse_ffn_layer(xt, y, lws[0], idx, cnt, k, ws)
        else:
            rm.rm_sparse_ffn_stack(xt, y, lws, idx, cnt, k, ws)

    step()
    torch.cuda.synchronize()
    y_eager = y.clone()

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm up on a side stream before capture
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()

    other_x = dev_f32(wl.make_x(99, x.shape, 1))
    other_y = torch.empty_like(other_x)
    other_ws = rm.workspace(d, d_ff, rm.RM_BF16, B, T, k, device="cuda")
    for r in range(4):
        y.fill_(float("nan"))
        idx.fill_(7)
        cnt.fill_(-1)
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, y_eager), f"replay {r} differs from the eager result"
        # eager work between replays, on other buffers
        if L == 1:
            rm.rm_sparse_ffn_layer(other_x, other_y, lws[0], idx, cnt, k, other_ws)
        else:
            rm.rm_sparse_ffn_stack(other_x, other_y, lws, idx, cnt, k, other_ws)
        torch.cuda.synchronize()

    ref = np.stack([oracle.ffn_stack(x[b], [lay.f64() for lay in layers],
                                     [masks[l * B + b].astype(np.float64) for l in range(L)]) for b in range(B)])
    ey, ed = errors(y.cpu().numpy(), ref, x)
    assert ey <= TOL_BF16 and ed <= TOL_BF16
