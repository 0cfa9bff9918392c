"""GPU parity of the Context Cache's visual-token recomputation (section 4.1, Eq. 2 and Eq. 3) against the oracle
(oracle.context_cache) on the same seeded inputs.

Bars:
- the float32 Eq. 2 drift within `drift_rel_bound(d)` of the float64 value (a rounding bound that holds for any
  summation order);
- the recomputed row list exactly the top-k of the GPU's own float32 drifts (ties to the lower token; an integer
  decision on the values it returns), and a valid top-k of the float64 drifts given that bound
  (`check_recomputed_rows`: the count, every non-visual row, ascending, no dropped row above a chosen one);
- repeated calls bit for bit equal;
- every recomputed row of y within max-abs relative error 2e-2 of the float64 FFN (bf16 weights, inputs rounded to
  bf16, float32 accumulation); every other row of y left bit for bit as the reference output."""
import numpy as np
import pytest
import torch

import workloads as wl
from oracle import context_cache as cc

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2609_19104_amd as rm  # noqa: E402
from gpu_helpers import TOL_BF16, dev_f32  # noqa: E402


def _bf16(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()


def _select(x, x_ref, v0, P, k):
    n_tok = x.shape[0]
    drift = torch.full((max(P, 1),), float("nan"), device="cuda")
    rows = torch.full((n_tok,), -5, dtype=torch.int32, device="cuda")
    count = torch.full((1,), -5, dtype=torch.int32, device="cuda")
    rm.rm_context_select(dev_f32(x), dev_f32(x_ref), v0, P, k, drift if P > 0 else None, rows, count)
    torch.cuda.synchronize()
    c = int(count.item())
    return drift.cpu().numpy()[:P], rows.cpu().numpy()[:c], c


SELECT_CASES = [
    # n_tok, d, v0, P, k, quantum (> 0: rounded differences, so tied drifts)
    (850, 2048, 0, 768, 308, 0.0),
    (100, 64, 10, 80, 0, 0.0),
    (100, 64, 10, 80, 80, 0.0),
    (33, 96, 0, 33, 5, 0.0),
    (50, 128, 40, 0, 0, 0.0),
    (300, 256, 20, 256, 103, 0.5),
    (16384, 32, 0, 16384, 4000, 0.0),
    (4096, 32, 0, 4000, 1500, 0.5),   # the last size of the 256-thread selection
    (4097, 32, 1, 4000, 1500, 0.5),   # one row more: 1024 threads
]


def _check_selection(x, x_ref, v0, P, k, drift, rows, count):
    n_tok, d = x.shape
    ref = cc.drift(x[v0:v0 + P], x_ref[v0:v0 + P])
    bound = cc.drift_rel_bound(d)
    got = drift.astype(np.float64)
    zero = ref == 0.0
    assert np.all(got[zero] == 0.0)
    err = float(np.max(np.abs(got[~zero] - ref[~zero]) / ref[~zero])) if np.any(~zero) else 0.0
    print(f"drift: max rel err {err:.2e} against float64 (bound {bound:.2e})")
    assert err <= bound
    assert count == n_tok - P + k
    assert np.array_equal(rows, cc.recomputed_rows(got, n_tok, v0, k))  # the decision on its own values
    cc.check_recomputed_rows(rows, ref, n_tok, v0, k, rel=bound)


@pytest.mark.parametrize("n_tok,d,v0,P,k,quantum", SELECT_CASES)
def test_drift_and_row_selection(n_tok, d, v0, P, k, quantum):
    r = np.random.default_rng(n_tok + d)
    x_ref = r.standard_normal((n_tok, d)).astype(np.float32)
    delta = r.standard_normal((n_tok, d)) * np.exp(r.standard_normal((n_tok, 1)))
    if quantum > 0:
        delta = np.round(delta / quantum) * quantum
        delta[::3] = 0.0  # rows without drift: exact zeros, tied
    x = (x_ref + delta).astype(np.float32)
    drift, rows, count = _select(x, x_ref, v0, P, k)
    _check_selection(x, x_ref, v0, P, k, drift, rows, count)
    drift2, rows2, count2 = _select(x, x_ref, v0, P, k)
    assert np.array_equal(drift.view(np.uint32), drift2.view(np.uint32))
    assert count2 == count and np.array_equal(rows2, rows)


def _run_ffn(w, x, y_ref, rows, count, max_rows, act, packed=False):
    xt, yt = dev_f32(x), dev_f32(y_ref)
    rt = torch.from_numpy(np.concatenate([rows, np.full(w.n_tok - len(rows), -1)]).astype(np.int32)).cuda()
    ct = torch.tensor([count], dtype=torch.int32, device="cuda")
    ws = rm.context_workspace(w.d, w.d_ff, w.n_tok, max_rows, act=act)
    ws.fill_(0x7F)  # the path must not rely on a cleared workspace
    wg, wu, wd = _bf16(w.layer.w_gate), _bf16(w.layer.w_up), _bf16(w.w_down_t)
    if packed:
        pk = rm.rm_context_pack(wg, wu, wd, act=act)
        rm.rm_context_ffn_packed(xt, yt, pk, rt, ct, max_rows, ws, act=act)
    else:
        rm.rm_context_ffn(xt, yt, wg, wu, wd, rt, ct, max_rows, ws, act=act)
    torch.cuda.synchronize()
    return yt.cpu().numpy()


def _check_update(w, x, y_ref, y, rows, act):
    keep = np.setdiff1d(np.arange(w.n_tok), rows)
    assert np.array_equal(y[keep].view(np.uint32), y_ref[keep].view(np.uint32))
    chk = rows
    if len(chk) == 0:
        return
    wg, wu, _, _ = w.layer.f64()
    wdt = wl.storage_to_f64(w.w_down_t)
    ref = cc.ffn_out(x[chk], wg, wu, wdt, act)
    err = np.max(np.abs(y[chk] - ref)) / np.max(np.abs(ref))
    print(f"recomputed rows: rel err {err:.3e} over {len(chk)} rows")
    assert err <= TOL_BF16


FFN_CASES = [
    # d, d_ff, n_tok, v0, P, k, max_rows, act
    (128, 256, 70, 5, 60, 20, 40, "gelu_tanh"),
    (512, 2048, 300, 0, 256, 100, 160, "silu"),
    (256, 1024, 200, 0, 200, 199, 200, "gelu_tanh"),
    (64, 128, 30, 0, 30, 0, 5, "gelu_tanh"),
]


@pytest.mark.parametrize("packed", [False, True], ids=["row-major", "packed"])
@pytest.mark.parametrize("d,d_ff,n_tok,v0,P,k,max_rows,act", FFN_CASES)
def test_context_ffn_parity(d, d_ff, n_tok, v0, P, k, max_rows, act, packed):
    w = wl.context_workload(n_tok=n_tok, v0=v0, P=P, d=d, d_ff=d_ff, seed=7 + d)
    drift = cc.drift(w.x[v0:v0 + P], w.x_ref[v0:v0 + P])
    rows = cc.recomputed_rows(drift, n_tok, v0, k)
    count = min(len(rows), max_rows)  # rows past max_rows are not recomputed
    y = _run_ffn(w, w.x, w.y_ref, rows, count, max_rows, act, packed=packed)
    _check_update(w, w.x, w.y_ref, y, rows[:count], act)


def _blocked_reference(m):
    """The documented blocked layout, written out with NumPy: 64 x 64 blocks, row tiles outermost, the blocks of a
    tile consecutive along K; in a block, row r's eight 16-byte pieces with piece p at position p ^ swz(r % 16),
    swz(r) = (r ^ (r >> 3)) & 7."""
    R, K = m.shape
    out = np.empty(R * K, dtype=m.dtype)
    swz = lambda r: (r ^ (r >> 3)) & 7  # noqa: E731
    for t in range(R // 64):
        for kb in range(K // 64):
            blk = m[t * 64:(t + 1) * 64, kb * 64:(kb + 1) * 64].reshape(64, 8, 8)
            img = np.empty_like(blk)
            for r in range(64):
                for p in range(8):
                    img[r, p ^ swz(r % 16)] = blk[r, p]
            base = (t * (K // 64) + kb) * 4096
            out[base:base + 4096] = img.reshape(-1)
    return out


def test_context_pack_layout_and_packed_matches_row_major_bit_for_bit():
    d, d_ff = 192, 256  # d not a multiple of 128: the down product runs 64-column tiles
    w = wl.context_workload(n_tok=90, v0=10, P=70, d=d, d_ff=d_ff, seed=21)
    wg, wu, wd = _bf16(w.layer.w_gate), _bf16(w.layer.w_up), _bf16(w.w_down_t)
    pk = rm.rm_context_pack(wg, wu, wd).cpu().numpy().view(np.uint16)
    mats = [w.layer.w_gate, w.layer.w_up, w.w_down_t]
    ref = np.concatenate([_blocked_reference(np.ascontiguousarray(m).view(np.uint16)) for m in mats])
    assert np.array_equal(pk, ref)
    rows = cc.recomputed_rows(cc.drift(w.x[10:80], w.x_ref[10:80]), 90, 10, 30)
    y_row = _run_ffn(w, w.x, w.y_ref, rows, len(rows), len(rows), "gelu_tanh")
    y_pk = _run_ffn(w, w.x, w.y_ref, rows, len(rows), len(rows), "gelu_tanh", packed=True)
    assert np.array_equal(y_row.view(np.uint32), y_pk.view(np.uint32))
    _check_update(w, w.x, w.y_ref, y_pk, rows, "gelu_tanh")


def test_context_ffn_with_no_rows_leaves_y():
    w = wl.context_workload(n_tok=40, v0=0, P=40, d=128, d_ff=256, seed=9)
    y = _run_ffn(w, w.x, w.y_ref, np.zeros(0, np.int32), 0, 8, "gelu_tanh")
    assert np.array_equal(y.view(np.uint32), w.y_ref.view(np.uint32))


def test_context_cache_full_size_end_to_end():
    # The VLM layer of a pi0.5-style model: 850 rows (768 visual), rho_p = 0.4 -> 308 + 82 rows recomputed,
    # d = 2048, d_ff = 16384, GeGLU.  Selection on the GPU, checked against float64 Eq. 2; the FFN run on the rows
    # the GPU chose and every one of them checked, as is every kept row.
    w = wl.context_workload()
    drift, rows, count = _select(w.x, w.x_ref, w.v0, w.P, w.k)
    _check_selection(w.x, w.x_ref, w.v0, w.P, w.k, drift, rows, count)
    assert count == 390
    y = _run_ffn(w, w.x, w.y_ref, rows, count, count, "gelu_tanh")
    _check_update(w, w.x, w.y_ref, y, rows, "gelu_tanh")


def _fuzz_cases(n=10, seed=2609):
    rng = np.random.default_rng(seed)
    for _ in range(n):
        d = int(rng.choice([64, 128, 192, 320]))
        d_ff = int(rng.choice([128, 256, 384]))
        n_tok = int(rng.integers(1, 600))
        v0 = int(rng.integers(0, n_tok))
        P = int(rng.integers(0, n_tok - v0 + 1))
        k = int(rng.integers(0, P + 1))
        rows_total = n_tok - P + k
        max_rows = int(rng.integers(max(1, rows_total // 2), n_tok + 1)) if rows_total else int(rng.integers(1, 9))
        yield d, d_ff, n_tok, v0, P, k, max_rows, str(rng.choice(["silu", "gelu_tanh"])), bool(rng.integers(0, 2))


@pytest.mark.parametrize("d,d_ff,n_tok,v0,P,k,max_rows,act,packed", list(_fuzz_cases()))
def test_context_ffn_random_shapes(d, d_ff, n_tok, v0, P, k, max_rows, act, packed):
    # Seeded random shapes: widths of 1 to 5 K stages and 1 to 3 weight tiles, row counts below, at and above
    # one 256-row tile, lists cut by max_rows, both activations, both weight layouts.
    w = wl.context_workload(n_tok=n_tok, v0=v0, P=P, d=d, d_ff=d_ff, seed=3 + d + d_ff + n_tok)
    rows = cc.recomputed_rows(cc.drift(w.x[v0:v0 + P], w.x_ref[v0:v0 + P]), n_tok, v0, k)
    count = min(len(rows), max_rows)
    y = _run_ffn(w, w.x, w.y_ref, rows, count, max_rows, act, packed=packed)
    _check_update(w, w.x, w.y_ref, y, rows[:count], act)
