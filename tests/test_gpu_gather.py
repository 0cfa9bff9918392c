"""GPU checks of the compact row buffers (rm_gather_stack_rows; section 4.1's shared compact buffers).

Bars: the copies are bit-exact (rows past a count are zero); a stack or an Eq. 4 delta step run on the compact
layers with the identity lists gives the same y, bit for bit, as the same call on the original weights with the
group's lists (same kernels, same slot order)."""
import numpy as np
import pytest
import torch

import workloads as wl

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2609_19104_amd as rm  # noqa: E402
from gpu_helpers import compact, dev_f32, dev_weights  # noqa: E402


def _setup(d, d_ff, L, T, k, wdtype, seed):
    layers = [wl.make_layer(seed, l, d, d_ff, wdtype, norm="random") for l in range(L)]
    masks = np.stack([wl.uniform_mask(wl.rng(seed, 4, l), d_ff, max(1, k - 9 * l)) for l in range(L)])
    idx, cnt = compact(masks)
    return layers, [dev_weights(x) for x in layers], masks, idx, cnt


def _compact_layers(lws, out, L):
    return [(out[l, 0], out[l, 1], out[l, 2], lws[l][3]) for l in range(L)]


@pytest.mark.parametrize("wdtype", ["bf16", "f32"])
@pytest.mark.parametrize("d,d_ff,L,k,max_count", [(256, 1000, 3, 300, 320), (1024, 4096, 2, 1229, 1229),
                                                   (96, 64, 1, 64, 64), (512, 777, 2, 1, 40)])
def test_gather_rows_bit_exact(wdtype, d, d_ff, L, k, max_count):
    layers, lws, masks, idx, cnt = _setup(d, d_ff, L, 4, k, wdtype, 111)
    out = torch.full((L, 3, max_count, d), float("nan"), device="cuda").to(lws[0][0].dtype)
    rm.rm_gather_stack_rows(lws, idx, cnt, max_count, out)
    torch.cuda.synchronize()
    got = out.view(torch.int16 if wdtype == "bf16" else torch.int32).cpu().numpy()
    for l, layer in enumerate(layers):
        rows = np.flatnonzero(masks[l])[:max_count]
        for m, w in enumerate((layer.w_gate, layer.w_up, layer.w_down)):
            w = np.ascontiguousarray(w).view(np.int16 if wdtype == "bf16" else np.int32)
            assert np.array_equal(got[l, m, :len(rows)], w[rows])
            assert np.all(got[l, m, len(rows):] == 0)


def test_compact_layers_give_the_same_stack_and_delta_step():
    d, d_ff, L, T, k = 1024, 4096, 3, 51, 1229
    layers, lws, masks, idx, cnt = _setup(d, d_ff, L, T, k, "bf16", 112)
    out = torch.empty((L, 3, k, d), dtype=torch.bfloat16, device="cuda")
    rm.rm_gather_stack_rows(lws, idx, cnt, k, out)
    clw = _compact_layers(lws, out, L)
    ident = torch.arange(k, dtype=torch.int32, device="cuda").repeat(L, 1).contiguous()
    x = dev_f32(wl.make_x(112, (1, T, d), 0))
    ws = rm.workspace(d, d_ff, rm.RM_BF16, 1, T, k)
    ws_c = rm.workspace(d, k, rm.RM_BF16, 1, T, k)
    y1, y2 = torch.empty_like(x), torch.empty_like(x)
    rm.rm_sparse_ffn_stack(x, y1, lws, idx, cnt, k, ws)
    rm.rm_sparse_ffn_stack(x, y2, clw, ident, cnt, k, ws_c)
    torch.cuda.synchronize()
    assert torch.equal(y1.view(torch.int32), y2.view(torch.int32))
    # Eq. 4: the anchor's h_anchor slots follow the list order, so the compact delta step reuses them.
    ya = torch.empty((L, 1, T, d), device="cuda")
    ha = torch.empty((L, 1, k, T), device="cuda")
    rm.rm_anchor_ffn_stack(x, torch.empty_like(x), lws, idx, cnt, k, ya, ha,
                           rm.workspace(d, d_ff, rm.RM_BF16, 1, T, d_ff))
    xt = x + 0.05
    rm.rm_delta_ffn_stack(xt, y1, lws, idx, cnt, k, ya, ha, ws)
    rm.rm_delta_ffn_stack(xt, y2, clw, ident, cnt, k, ya, ha, ws_c)
    torch.cuda.synchronize()
    assert torch.equal(y1.view(torch.int32), y2.view(torch.int32))
