"""Host-side checks of the C ABI: the library loads, exports exactly what include/rmuscle.h declares, sizes
workspaces, and rejects bad arguments before enqueuing anything (no GPU needed: every call here fails
validation or is pure host arithmetic)."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2609_19104_amd as rm

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "rmuscle.h")


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:rm_status|const char \*)\s*(rm_\w+)\s*\(", text, re.M)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(rm.LIB_PATH):
        pytest.skip("librmuscle.so not built")
    return rm.load_library()


def test_header_declares_the_abi():
    assert _declared() == sorted(rm.EXPORTED)


def test_exports_match_header(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", rm.LIB_PATH], capture_output=True, text=True, check=True)
    exported = sorted({l.split()[-1] for l in out.stdout.splitlines() if re.search(r"\brm_\w+$", l)})
    assert exported == _declared()
    for name in _declared():
        assert getattr(lib, name) is not None


def test_status_strings(lib):
    for st in (rm.RM_OK, rm.RM_ERR_INVALID_ARG, rm.RM_ERR_SHAPE, rm.RM_ERR_DTYPE, rm.RM_ERR_ALIGN,
               rm.RM_ERR_WORKSPACE, rm.RM_ERR_HIP):
        assert rm.status_string(st).startswith("RM_")
    assert "unknown" in rm.status_string(42)


def _size(d, d_ff, wdtype, B, T, k):
    out = ctypes.c_size_t(0)
    s = rm.FfnShape(d, d_ff, wdtype, 1e-6)
    st = rm.load_library().rm_workspace_size(ctypes.byref(s), B, T, k, ctypes.byref(out))
    return st, out.value


def test_workspace_size_values(lib):
    # bf16, d=1024, d_ff=4096, T=51, K=1229: at least xn (51 x 1024 bf16) and H (64 tokens x 1248 slots bf16).
    st, n = _size(1024, 4096, rm.RM_BF16, 1, 51, 1229)
    assert st == rm.RM_OK
    assert n >= 51 * 1024 * 2 + 64 * 1248 * 2
    assert n % 256 == 0
    # Monotone in every size argument.
    assert _size(1024, 4096, rm.RM_BF16, 2, 51, 1229)[1] > n
    assert _size(1024, 4096, rm.RM_BF16, 1, 52, 1229)[1] > n
    assert _size(1024, 4096, rm.RM_BF16, 1, 51, 4096)[1] >= n
    assert _size(256, 1024, rm.RM_F32, 1, 8, 256)[0] == rm.RM_OK
    assert _size(1024, 4096, rm.RM_BF16, 1, 51, 0)[0] == rm.RM_OK


@pytest.mark.parametrize("args,expected", [
    ((1000, 4096, 1, 1, 51, 10), rm.RM_ERR_SHAPE),       # d not a multiple of 32
    ((0, 4096, 1, 1, 51, 10), rm.RM_ERR_INVALID_ARG),
    ((1024, 0, 1, 1, 51, 0), rm.RM_ERR_INVALID_ARG),
    ((1024, 4096, 7, 1, 51, 10), rm.RM_ERR_DTYPE),
    ((1024, 4096, 1, 0, 51, 10), rm.RM_ERR_INVALID_ARG),
    ((1024, 4096, 1, 1, 0, 10), rm.RM_ERR_INVALID_ARG),
    ((1024, 4096, 1, 1, 51, 4097), rm.RM_ERR_SHAPE),     # max_count > d_ff
    ((1024, 4096, 1, 1, 51, -1), rm.RM_ERR_SHAPE),
])
def test_workspace_size_rejects(lib, args, expected):
    st, _ = _size(*args)
    assert st == expected
    assert rm.last_error() != ""


FAKE = 0x10000  # a 16-byte aligned address that is never dereferenced: validation fails first


def _layer_call(lib, *, shape=(1024, 4096, 1), B=1, T=51, x=FAKE, y=FAKE, idx=FAKE, cnt=FAKE, k=100,
                ws=FAKE * 16, ws_bytes=1 << 30, w=(FAKE, FAKE, FAKE, None)):
    s = rm.FfnShape(shape[0], shape[1], shape[2], 1e-6)
    lw = rm.LayerWeights(*w)
    return lib.rm_sparse_ffn_layer(ctypes.byref(s), ctypes.byref(lw), B, T, x, y, idx, cnt, k, ws, ws_bytes, None)


@pytest.mark.parametrize("kw,expected", [
    (dict(x=None), rm.RM_ERR_INVALID_ARG),
    (dict(idx=None), rm.RM_ERR_INVALID_ARG),
    (dict(cnt=None), rm.RM_ERR_INVALID_ARG),
    (dict(w=(None, FAKE, FAKE, None)), rm.RM_ERR_INVALID_ARG),
    (dict(w=(FAKE + 2, FAKE, FAKE, None)), rm.RM_ERR_ALIGN),
    (dict(w=(FAKE, FAKE, FAKE, FAKE + 4)), rm.RM_ERR_ALIGN),
    (dict(x=FAKE + 4, y=FAKE + 4), rm.RM_ERR_ALIGN),
    (dict(idx=FAKE + 2), rm.RM_ERR_ALIGN),
    (dict(k=5000), rm.RM_ERR_SHAPE),
    (dict(k=-3), rm.RM_ERR_SHAPE),
    (dict(shape=(1000, 4096, 1)), rm.RM_ERR_SHAPE),
    (dict(shape=(1024, 4096, 9)), rm.RM_ERR_DTYPE),
    (dict(B=0), rm.RM_ERR_INVALID_ARG),
    (dict(B=70000), rm.RM_ERR_SHAPE),
    (dict(T=-1), rm.RM_ERR_INVALID_ARG),
    (dict(ws=None), rm.RM_ERR_INVALID_ARG),
    (dict(ws_bytes=100), rm.RM_ERR_WORKSPACE),
    (dict(y=FAKE + 16), rm.RM_ERR_INVALID_ARG),               # y overlaps x without being x
    (dict(ws=FAKE), rm.RM_ERR_INVALID_ARG),                   # workspace overlaps x
])
def test_layer_rejects_before_launch(lib, kw, expected):
    assert _layer_call(lib, **kw) == expected
    assert rm.last_error() != ""


def test_stack_and_dense_reject(lib):
    s = rm.FfnShape(1024, 4096, 1, 1e-6)
    arr = (rm.LayerWeights * 2)(rm.LayerWeights(FAKE, FAKE, FAKE, None), rm.LayerWeights(FAKE, None, FAKE, None))
    st = lib.rm_sparse_ffn_stack(ctypes.byref(s), arr, 2, 1, 51, FAKE, FAKE, FAKE, FAKE, 10, FAKE * 16, 1 << 30, None)
    assert st == rm.RM_ERR_INVALID_ARG and "layer 1" in rm.last_error()
    st = lib.rm_sparse_ffn_stack(ctypes.byref(s), arr, 0, 1, 51, FAKE, FAKE, FAKE, FAKE, 10, FAKE * 16, 1 << 30, None)
    assert st == rm.RM_ERR_INVALID_ARG
    lw = rm.LayerWeights(FAKE, FAKE, FAKE, None)
    st = lib.rm_dense_ffn_ref(ctypes.byref(s), ctypes.byref(lw), 1, 51, FAKE, FAKE, FAKE * 16, 64, None)
    assert st == rm.RM_ERR_WORKSPACE


def test_mask_compact_rejects(lib):
    assert lib.rm_mask_compact(None, 1, 16, FAKE, FAKE * 2, None) == rm.RM_ERR_INVALID_ARG
    assert lib.rm_mask_compact(FAKE, 0, 16, FAKE * 2, FAKE * 3, None) == rm.RM_ERR_INVALID_ARG
    assert lib.rm_mask_compact(FAKE, 1, 16, FAKE * 2 + 1, FAKE * 3, None) == rm.RM_ERR_ALIGN
    assert lib.rm_mask_compact(FAKE, 4, 16, FAKE + 8, FAKE * 3, None) == rm.RM_ERR_INVALID_ARG  # idx overlaps mask


def test_profile_hook_rejects_unknown_kernel(lib):
    assert lib.rm_profile_kernel_events(5, None, None) == rm.RM_ERR_INVALID_ARG
    assert lib.rm_profile_kernel_events(rm.RM_KERNEL_GATEUP, None, None) == rm.RM_OK


def test_layer_kernels_query(lib):
    both = (1 << rm.RM_KERNEL_GATEUP) | (1 << rm.RM_KERNEL_DOWN)
    assert rm.rm_layer_kernels(1024, 4096, rm.RM_BF16, 1, 51, 1229) == both
    assert rm.rm_layer_kernels(256, 1024, rm.RM_F32, 1, 8, 256) == both
    # One sample's long list at d = 2048: one launch on a 256-unit device, else the two.
    assert rm.rm_layer_kernels(2048, 16384, rm.RM_BF16, 1, 51, 4916) in (both, 1 << rm.RM_KERNEL_LAYER)
    assert rm.rm_layer_kernels(2048, 16384, rm.RM_BF16, 2, 51, 4916) == both
    with pytest.raises(rm.RmError):
        rm.rm_layer_kernels(1000, 4096, rm.RM_BF16, 1, 51, 10)
    assert lib.rm_layer_kernels(None, 1, 51, 10, None) == rm.RM_ERR_INVALID_ARG


def test_binding_refuses_cpu_tensors():
    import torch
    x = torch.zeros(1, 4, 32)
    with pytest.raises((ValueError, RuntimeError)):
        rm.rm_dense_ffn_ref(x, x, (torch.zeros(8, 32), torch.zeros(8, 32), torch.zeros(8, 32), None),
                            torch.zeros(16, dtype=torch.uint8))


def test_profile_hook_accepts_every_kernel_id(lib):
    for k in (rm.RM_KERNEL_GATEUP, rm.RM_KERNEL_DOWN, rm.RM_KERNEL_SCORES, rm.RM_KERNEL_GROUP_SELECT,
              rm.RM_KERNEL_LAYER):
        assert lib.rm_profile_kernel_events(k, None, None) == rm.RM_OK
    assert lib.rm_profile_kernel_events(5, None, None) == rm.RM_ERR_INVALID_ARG
    assert lib.rm_profile_kernel_events(-1, None, None) == rm.RM_ERR_INVALID_ARG


def test_activation_and_gate_are_validated(lib):
    s = rm.FfnShape(1024, 4096, 1, 1e-6, 7)  # unknown activation
    lw = rm.LayerWeights(FAKE, FAKE, FAKE, None, None)
    st = lib.rm_sparse_ffn_layer(ctypes.byref(s), ctypes.byref(lw), 1, 51, FAKE, FAKE, FAKE, FAKE, 100, FAKE * 16,
                                 1 << 30, None)
    assert st == rm.RM_ERR_INVALID_ARG and "act" in rm.last_error()
    s = rm.FfnShape(1024, 4096, 1, 1e-6, rm.RM_ACT_GELU_TANH)
    lw = rm.LayerWeights(FAKE, FAKE, FAKE, None, FAKE + 4)  # misaligned gate
    st = lib.rm_sparse_ffn_layer(ctypes.byref(s), ctypes.byref(lw), 1, 51, FAKE, FAKE, FAKE, FAKE, 100, FAKE * 16,
                                 1 << 30, None)
    assert st == rm.RM_ERR_ALIGN
    lw = rm.LayerWeights(FAKE, FAKE, FAKE, None, FAKE)  # gate overlapping y (x == y == FAKE)
    st = lib.rm_sparse_ffn_layer(ctypes.byref(s), ctypes.byref(lw), 1, 51, FAKE, FAKE, FAKE * 2, FAKE * 3, 100,
                                 FAKE * 16, 1 << 30, None)
    assert st == rm.RM_ERR_INVALID_ARG and "out_gate" in rm.last_error()


def test_masked_calls_reject(lib):
    s = rm.FfnShape(1024, 4096, 1, 1e-6)
    lw = rm.LayerWeights(FAKE, FAKE, FAKE, None)
    base = dict(B=1, T=51, x=FAKE, y=FAKE, mask=FAKE * 64, idx=FAKE * 128, cnt=FAKE * 256, k=100)

    def call(**kw):
        a = dict(base, **kw)
        return lib.rm_masked_ffn_layer(ctypes.byref(s), ctypes.byref(lw), a["B"], a["T"], a["x"], a["y"], a["mask"],
                                       a["idx"], a["cnt"], a["k"], FAKE * 1024, 1 << 30, None)
    assert call(mask=None) == rm.RM_ERR_INVALID_ARG
    assert call(idx=FAKE * 64 + 8) == rm.RM_ERR_INVALID_ARG   # idx overlaps the mask
    assert call(cnt=FAKE * 128 + 4) == rm.RM_ERR_INVALID_ARG  # count overlaps idx
    arr = (rm.LayerWeights * 2)(lw, lw)
    assert lib.rm_masked_ffn_stack(ctypes.byref(s), arr, 0, 1, 51, FAKE, FAKE, FAKE * 64, FAKE * 128, FAKE * 256, 100,
                                   FAKE * 1024, 1 << 30, None) == rm.RM_ERR_INVALID_ARG


def test_anchor_and_delta_reject(lib):
    s = rm.FfnShape(1024, 4096, 1, 1e-6)
    arr = (rm.LayerWeights * 2)(rm.LayerWeights(FAKE, FAKE, FAKE, None), rm.LayerWeights(FAKE, FAKE, FAKE, None))
    args = (FAKE, FAKE, FAKE * 64, FAKE * 128, 100)

    def anchor(ya, ha, ws_bytes=1 << 30, k=100):
        return lib.rm_anchor_ffn_stack(ctypes.byref(s), arr, 2, 1, 51, *args[:4], k, ya, ha, FAKE * 4096, ws_bytes,
                                       None)
    assert anchor(None, FAKE * 512) == rm.RM_ERR_INVALID_ARG
    assert anchor(FAKE * 512 + 4, FAKE * 1024) == rm.RM_ERR_ALIGN
    assert anchor(FAKE * 512, None) == rm.RM_ERR_INVALID_ARG            # h_anchor needed when max_count > 0
    assert anchor(FAKE * 512, FAKE * 512 + 64) == rm.RM_ERR_INVALID_ARG  # y_anchor and h_anchor overlap
    ws_sparse = _size(1024, 4096, rm.RM_BF16, 1, 51, 100)[1]
    assert anchor(FAKE * 512, FAKE * 1024, ws_bytes=ws_sparse) == rm.RM_ERR_WORKSPACE  # anchors need the dense size
    st = lib.rm_delta_ffn_stack(ctypes.byref(s), arr, 2, 1, 51, *args[:4], 100, None, FAKE * 1024, FAKE * 4096,
                                1 << 30, None)
    assert st == rm.RM_ERR_INVALID_ARG


def test_gather_norms_and_group_masks_reject(lib):
    s = rm.FfnShape(1024, 4096, 1, 1e-6)
    arr = (rm.LayerWeights * 1)(rm.LayerWeights(FAKE, FAKE, FAKE, None))
    assert lib.rm_gather_stack_rows(ctypes.byref(s), arr, 1, FAKE * 64, FAKE * 128, 0, FAKE * 256,
                                    None) == rm.RM_ERR_SHAPE
    assert lib.rm_gather_stack_rows(ctypes.byref(s), arr, 1, FAKE * 64, FAKE * 128, 100, FAKE,
                                    None) == rm.RM_ERR_INVALID_ARG  # out overlaps the weights
    assert lib.rm_neuron_norms(FAKE, 4096, 1000, rm.RM_BF16, FAKE * 64, None) == rm.RM_ERR_SHAPE
    assert lib.rm_neuron_norms(FAKE, 4096, 1024, 3, FAKE * 64, None) == rm.RM_ERR_DTYPE
    assert lib.rm_neuron_norms(FAKE, 4096, 1024, rm.RM_BF16, FAKE, None) == rm.RM_ERR_INVALID_ARG  # overlap
    gm = lib.rm_group_masks
    assert gm(FAKE, 5, 18, 20000, 51, FAKE * 64, 100, FAKE * 128, FAKE * 256, None) == rm.RM_ERR_SHAPE
    assert gm(FAKE, 5, 18, 4096, 51, FAKE * 64, 4097, FAKE * 128, FAKE * 256, None) == rm.RM_ERR_SHAPE
    assert gm(FAKE, 300, 300, 4096, 51, FAKE * 64, 100, FAKE * 128, FAKE * 256, None) == rm.RM_ERR_SHAPE
    assert gm(FAKE, 5, 18, 4096, 51, FAKE * 64, 100, FAKE * 128, FAKE * 128 + 4, None) == rm.RM_ERR_INVALID_ARG
    assert gm(None, 5, 18, 4096, 51, FAKE * 64, 100, FAKE * 128, FAKE * 256, None) == rm.RM_ERR_INVALID_ARG


def _ctx_size(d, d_ff, n_tok, max_rows, wdtype=rm.RM_BF16):
    out = ctypes.c_size_t(0)
    s = rm.FfnShape(d, d_ff, wdtype, 1e-6, rm.RM_ACT_GELU_TANH)
    return rm.load_library().rm_context_workspace_size(ctypes.byref(s), n_tok, max_rows, ctypes.byref(out)), out.value


def test_context_calls_validate(lib):
    st, n = _ctx_size(2048, 16384, 850, 390)
    assert st == rm.RM_OK and n >= 512 * 2048 * 2 + 512 * 16384 * 2 and n % 256 == 0
    assert _ctx_size(2048, 16384, 850, 391)[1] >= n
    assert _ctx_size(2048, 16384, 850, 900)[0] == rm.RM_ERR_SHAPE     # max_rows > n_tok
    assert _ctx_size(2048, 16384, 850, 390, rm.RM_F32)[0] == rm.RM_ERR_DTYPE
    assert _ctx_size(2080, 16384, 850, 390)[0] == rm.RM_ERR_SHAPE     # d not a multiple of 64
    assert _ctx_size(2048, 16320, 850, 390)[0] == rm.RM_ERR_SHAPE     # d_ff not a multiple of 128
    sel = lib.rm_context_select
    assert sel(FAKE, FAKE * 64, 850, 2048, 0, 768, 769, FAKE * 128, FAKE * 256, FAKE * 512, None) == rm.RM_ERR_SHAPE
    assert sel(FAKE, FAKE * 64, 850, 2048, 100, 768, 10, FAKE * 128, FAKE * 256, FAKE * 512, None) == rm.RM_ERR_SHAPE
    assert sel(FAKE, FAKE * 64, 20000, 32, 0, 10, 1, FAKE * 128, FAKE * 256, FAKE * 512, None) == rm.RM_ERR_SHAPE
    assert sel(FAKE, FAKE * 64, 850, 2048, 0, 768, 10, None, FAKE * 256, FAKE * 512, None) == rm.RM_ERR_INVALID_ARG
    assert sel(FAKE, FAKE * 64, 850, 2048, 0, 768, 10, FAKE * 128, FAKE * 128 + 64, FAKE * 512,
               None) == rm.RM_ERR_INVALID_ARG  # rows overlap drift
    s = rm.FfnShape(2048, 16384, rm.RM_BF16, 1e-6, rm.RM_ACT_GELU_TANH)
    ffn = lib.rm_context_ffn
    assert ffn(ctypes.byref(s), FAKE, FAKE, FAKE, 850, FAKE * 64, FAKE * 128, FAKE * 256, 390, FAKE * 512,
               FAKE * 4096, 100, None) == rm.RM_ERR_WORKSPACE
    assert ffn(ctypes.byref(s), FAKE, FAKE, FAKE, 850, FAKE * 64, FAKE * 128, FAKE * 256, 390, FAKE * 64,
               FAKE * 4096, 1 << 30, None) == rm.RM_ERR_INVALID_ARG  # y is x
    assert ffn(ctypes.byref(s), None, FAKE, FAKE, 850, FAKE * 64, FAKE * 128, FAKE * 256, 390, FAKE * 512,
               FAKE * 4096, 1 << 30, None) == rm.RM_ERR_INVALID_ARG
    # Inputs the launches only read must not overlap what they write (y, the workspace).
    W, mb = 1 << 36, 2048 * 16384 * 2
    y, ws = FAKE * 512, 1 << 34
    for wg, wu, wd, rows, cnt in [(W, W + mb, W + 2 * mb, y + 64, FAKE * 256),      # rows inside y
                                  (W, W + mb, W + 2 * mb, FAKE * 128, ws + 8),      # count inside the workspace
                                  (W, W + mb, ws + 4096, FAKE * 128, FAKE * 256),   # w_down_t inside the workspace
                                  (y - 16, W + mb, W + 2 * mb, FAKE * 128, FAKE * 256)]:  # w_gate over y
        assert ffn(ctypes.byref(s), wg, wu, wd, 850, FAKE * 64, rows, cnt, 390, y, ws, 1 << 30,
                   None) == rm.RM_ERR_INVALID_ARG


def test_context_pack_calls_validate(lib):
    s = rm.FfnShape(2048, 16384, rm.RM_BF16, 1e-6, rm.RM_ACT_GELU_TANH)
    n = ctypes.c_size_t(0)
    assert lib.rm_context_pack_size(ctypes.byref(s), ctypes.byref(n)) == rm.RM_OK
    assert n.value == 3 * 2048 * 16384 * 2
    odd = rm.FfnShape(2048, 16320, rm.RM_BF16, 1e-6, rm.RM_ACT_GELU_TANH)  # d_ff not a multiple of 128
    assert lib.rm_context_pack_size(ctypes.byref(odd), ctypes.byref(n)) == rm.RM_ERR_SHAPE
    assert lib.rm_context_pack_size(ctypes.byref(s), None) == rm.RM_ERR_INVALID_ARG
    big = 3 * 2048 * 16384 * 2
    pack = lib.rm_context_pack
    W = 1 << 32  # the packed buffer, well away from the fake weights
    assert pack(ctypes.byref(s), None, FAKE, FAKE, W, big, None) == rm.RM_ERR_INVALID_ARG
    assert pack(ctypes.byref(s), FAKE, FAKE, FAKE, W, big - 1, None) == rm.RM_ERR_WORKSPACE
    assert pack(ctypes.byref(s), FAKE + 8, FAKE, FAKE, W, big, None) == rm.RM_ERR_ALIGN
    assert pack(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, big, None) == rm.RM_ERR_INVALID_ARG  # packed over w_gate
    assert pack(ctypes.byref(odd), FAKE, FAKE, FAKE, W, big, None) == rm.RM_ERR_SHAPE
    fp = lib.rm_context_ffn_packed
    assert fp(ctypes.byref(s), None, 850, FAKE * 64, FAKE * 128, FAKE * 256, 390, FAKE * 512, FAKE * 4096, 1 << 30,
              None) == rm.RM_ERR_INVALID_ARG
    assert fp(ctypes.byref(s), W, 850, FAKE * 64, FAKE * 128, FAKE * 256, 390, W + 64, FAKE * 4096, 1 << 30,
              None) == rm.RM_ERR_INVALID_ARG  # y inside the packed weights
    assert fp(ctypes.byref(s), W, 850, FAKE * 64, FAKE * 128, FAKE * 256, 390, FAKE * 512, FAKE * 4096, 100,
              None) == rm.RM_ERR_WORKSPACE
    assert fp(ctypes.byref(odd), W, 850, FAKE * 64, FAKE * 128, FAKE * 256, 390, FAKE * 512, FAKE * 4096, 1 << 30,
              None) == rm.RM_ERR_SHAPE


def test_lists_must_not_overlap_what_the_layer_writes(lib):
    # idx and count are read while y and the workspace are written; overlapping them is rejected before any
    # launch (every pointer below fails that check, so nothing is dereferenced).
    s = rm.FfnShape(1024, 4096, rm.RM_BF16, 1e-6, rm.RM_ACT_SILU)
    x, y, ws = FAKE * 64, FAKE * 128, 1 << 34
    w = rm.LayerWeights(1 << 36, (1 << 36) + (1 << 24), (1 << 36) + (1 << 25), None, None)
    layer = lib.rm_sparse_ffn_layer
    for idx, cnt in [(y + 256, FAKE), (ws + 1024, FAKE), (FAKE, y + 4), (FAKE, ws)]:
        assert layer(ctypes.byref(s), ctypes.byref(w), 1, 51, x, y, idx, cnt, 1229, ws, 1 << 30,
                     None) == rm.RM_ERR_INVALID_ARG
    # A stack's lists span L blocks: layer 2's block reaching into y is caught too.
    ws_arr = (rm.LayerWeights * 3)(w, w, w)
    idx = y - 2 * 4096 * 4 - 64
    assert lib.rm_sparse_ffn_stack(ctypes.byref(s), ws_arr, 3, 1, 51, x, y, idx, FAKE, 1229, ws, 1 << 30,
                                   None) == rm.RM_ERR_INVALID_ARG


def test_noalloc_layer_rejects_calls_beyond_its_scratch_before_touching_the_device(lib):
    # rm_sparse_ffn_layer_noalloc sizes the call from the shape alone and refuses one that needs more than
    # RM_NOALLOC_SCRATCH_BYTES without any device call (this host has no GPU).
    fake = ctypes.c_void_p(0x100000)
    w = rm.LayerWeights(0x100000, 0x200000, 0x300000, None, None)

    def call(d, d_ff, wdtype, B, T, k):
        s = rm.FfnShape(d, d_ff, wdtype, 1e-6, rm.RM_ACT_SILU)
        return lib.rm_sparse_ffn_layer_noalloc(ctypes.byref(s), ctypes.byref(w), B, T, fake, fake, fake, fake, k,
                                               None)

    big = (4096, 16384, rm.RM_BF16, 64, 64, 16384)
    assert _size(*big)[1] > rm.NOALLOC_SCRATCH_BYTES
    assert call(*big) == rm.RM_ERR_WORKSPACE
    assert "holds" in rm.last_error() and str(rm.NOALLOC_SCRATCH_BYTES) in rm.last_error()
    assert call(1000, 4096, rm.RM_BF16, 1, 51, 10) == rm.RM_ERR_SHAPE
    assert call(1024, 4096, rm.RM_BF16, 1, 51, 4097) == rm.RM_ERR_SHAPE
    assert call(1024, 4096, rm.RM_BF16, 0, 51, 10) == rm.RM_ERR_INVALID_ARG
    # Every configuration of the action expert fits.
    for cfg in ((256, 1024, rm.RM_F32, 1, 8, 256), (1024, 4096, rm.RM_BF16, 1, 51, 1229),
                (2048, 16384, rm.RM_BF16, 1, 51, 16384), (1024, 4096, rm.RM_BF16, 16, 51, 1229)):
        assert _size(*cfg)[1] <= rm.NOALLOC_SCRATCH_BYTES
