"""Python binding of librmuscle.so, the Action Cache sparse-FFN hot path for MI355X (gfx950).

Argument marshalling only: every function checks tensor devices, dtypes and shapes, turns them into raw
device pointers plus the current HIP stream, and calls the C ABI function of the same name (declared in
include/rmuscle.h).  All computation runs in the library's HIP kernels; there is no fallback.  If the library
is not built, or no GPU is present, the calls raise.

Layouts (see include/rmuscle.h for the full contract):
  mask  uint8/bool [N][d_ff] -> idx int32 [N][d_ff] (ascending, -1 tail), count int32 [N]
  x, y  float32 [B][T][d];  weights [d_ff][d] float32 or bfloat16, row n = neuron n (w_down neuron-major)
  idx   int32 [B][d_ff] per layer ([L][B][d_ff] for a stack), count int32 [B] ([L][B])
  Eq. 4 anchor state: y_anchor float32 [L][B][T][d], h_anchor float32 [L][B][max_count][T]
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence, Tuple

import torch

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
# The in-tree build; RMUSCLE_LIB may name another build of the same library (e.g. for A/B timing).
LIB_PATH = os.environ.get("RMUSCLE_LIB") or os.path.join(PKG_DIR, "librmuscle.so")

NOALLOC_SCRATCH_BYTES = 32 << 20  # RM_NOALLOC_SCRATCH_BYTES

RM_OK = 0
RM_ERR_INVALID_ARG = -1
RM_ERR_SHAPE = -2
RM_ERR_DTYPE = -3
RM_ERR_ALIGN = -4
RM_ERR_WORKSPACE = -5
RM_ERR_HIP = -6

RM_F32 = 0
RM_BF16 = 1
RM_ACT_SILU = 0
RM_ACT_GELU_TANH = 1
ACTS = {"silu": RM_ACT_SILU, "gelu_tanh": RM_ACT_GELU_TANH}
RM_KERNEL_GATEUP = 0
RM_KERNEL_DOWN = 1
RM_KERNEL_SCORES = 2
RM_KERNEL_GROUP_SELECT = 3
RM_KERNEL_LAYER = 4

EXPORTED = ("rm_mask_compact", "rm_workspace_size", "rm_sparse_ffn_layer", "rm_sparse_ffn_layer_noalloc",
            "rm_sparse_ffn_stack",
            "rm_masked_ffn_layer", "rm_masked_ffn_stack", "rm_dense_ffn_ref", "rm_anchor_ffn_stack",
            "rm_delta_ffn_stack", "rm_gather_stack_rows", "rm_context_select", "rm_context_workspace_size",
            "rm_context_ffn", "rm_context_pack_size", "rm_context_pack", "rm_context_ffn_packed", "rm_neuron_norms",
            "rm_group_masks",
            "rm_profile_kernel_events", "rm_layer_kernels", "rm_stream_read",
            "rm_status_string", "rm_last_error")

# (w_gate, w_up, w_down, norm_g) or (w_gate, w_up, w_down, norm_g, out_gate); norm_g and out_gate may be None.
Layer = Tuple[Optional[torch.Tensor], ...]


class RmError(RuntimeError):
    def __init__(self, status: int, detail: str):
        self.status = status
        self.detail = detail
        super().__init__(f"{status_string(status)}: {detail}")


class FfnShape(ctypes.Structure):
    _fields_ = [("d", ctypes.c_int32), ("d_ff", ctypes.c_int32), ("wdtype", ctypes.c_int32),
                ("norm_eps", ctypes.c_float), ("act", ctypes.c_int32)]


class LayerWeights(ctypes.Structure):
    _fields_ = [("w_gate", ctypes.c_void_p), ("w_up", ctypes.c_void_p), ("w_down", ctypes.c_void_p),
                ("norm_g", ctypes.c_void_p), ("out_gate", ctypes.c_void_p)]


_lib: Optional[ctypes.CDLL] = None


def library_path() -> str:
    return LIB_PATH


def load_library() -> ctypes.CDLL:
    """Load librmuscle.so (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built: run `python -m paper_2609_19104_amd.build` "
                           "(or __graft_entry__.build()) first")
    lib = ctypes.CDLL(LIB_PATH)
    i32, vp, sz = ctypes.c_int32, ctypes.c_void_p, ctypes.c_size_t
    sp, wp = ctypes.POINTER(FfnShape), ctypes.POINTER(LayerWeights)
    sigs = {
        "rm_mask_compact": [vp, i32, i32, vp, vp, vp],
        "rm_workspace_size": [sp, i32, i32, i32, ctypes.POINTER(sz)],
        "rm_sparse_ffn_layer": [sp, wp, i32, i32, vp, vp, vp, vp, i32, vp, sz, vp],
        "rm_sparse_ffn_layer_noalloc": [sp, wp, i32, i32, vp, vp, vp, vp, i32, vp],
        "rm_sparse_ffn_stack": [sp, wp, i32, i32, i32, vp, vp, vp, vp, i32, vp, sz, vp],
        "rm_masked_ffn_layer": [sp, wp, i32, i32, vp, vp, vp, vp, vp, i32, vp, sz, vp],
        "rm_masked_ffn_stack": [sp, wp, i32, i32, i32, vp, vp, vp, vp, vp, i32, vp, sz, vp],
        "rm_dense_ffn_ref": [sp, wp, i32, i32, vp, vp, vp, sz, vp],
        "rm_anchor_ffn_stack": [sp, wp, i32, i32, i32, vp, vp, vp, vp, i32, vp, vp, vp, sz, vp],
        "rm_delta_ffn_stack": [sp, wp, i32, i32, i32, vp, vp, vp, vp, i32, vp, vp, vp, sz, vp],
        "rm_gather_stack_rows": [sp, wp, i32, vp, vp, i32, vp, vp],
        "rm_context_select": [vp, vp, i32, i32, i32, i32, i32, vp, vp, vp, vp],
        "rm_context_workspace_size": [sp, i32, i32, ctypes.POINTER(sz)],
        "rm_context_ffn": [sp, vp, vp, vp, i32, vp, vp, vp, i32, vp, vp, sz, vp],
        "rm_context_pack_size": [sp, ctypes.POINTER(sz)],
        "rm_context_pack": [sp, vp, vp, vp, vp, sz, vp],
        "rm_context_ffn_packed": [sp, vp, i32, vp, vp, vp, i32, vp, vp, sz, vp],
        "rm_neuron_norms": [vp, i32, i32, i32, vp, vp],
        "rm_group_masks": [vp, i32, i32, i32, i32, vp, i32, vp, vp, vp],
        "rm_profile_kernel_events": [i32, vp, vp],
        "rm_layer_kernels": [sp, i32, i32, i32, ctypes.POINTER(ctypes.c_uint32)],
        "rm_stream_read": [vp, sz, i32, vp, vp],
        "rm_status_string": [i32],
        "rm_last_error": [],
    }
    for name, args in sigs.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_char_p if name in ("rm_status_string", "rm_last_error") else ctypes.c_int
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load_library().rm_status_string(status).decode()


def last_error() -> str:
    return load_library().rm_last_error().decode()


def _check(status: int) -> None:
    if status != RM_OK:
        raise RmError(status, last_error())


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _need_cuda(name: str, t: torch.Tensor, dtypes, ndim: Optional[int] = None) -> None:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on a HIP device, got {t.device}")
    if t.dtype not in dtypes:
        raise ValueError(f"{name} has dtype {t.dtype}, expected one of {dtypes}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dims, got {tuple(t.shape)}")


def wdtype_of(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return RM_BF16
    if t.dtype == torch.float32:
        return RM_F32
    raise ValueError(f"weights must be float32 or bfloat16, got {t.dtype}")


def _shape(layer: Layer, eps: float, act: str = "silu") -> FfnShape:
    wg = layer[0]
    if act not in ACTS:
        raise ValueError(f"act must be one of {sorted(ACTS)}, got {act!r}")
    return FfnShape(int(wg.shape[1]), int(wg.shape[0]), wdtype_of(wg), float(eps), ACTS[act])


def _weights(layer: Layer, B: Optional[int] = None) -> LayerWeights:
    if len(layer) not in (4, 5):
        raise ValueError("a layer is (w_gate, w_up, w_down, norm_g[, out_gate])")
    wg, wu, wd, g = layer[:4]
    gate = layer[4] if len(layer) == 5 else None
    d_ff, d = wg.shape
    for name, w in (("w_gate", wg), ("w_up", wu), ("w_down", wd)):
        _need_cuda(name, w, (wg.dtype,), 2)
        if tuple(w.shape) != (d_ff, d):
            raise ValueError(f"{name} has shape {tuple(w.shape)}, expected {(d_ff, d)} (neuron-major)")
    if g is not None:
        _need_cuda("norm_g", g, (torch.float32,), 1)
        if g.shape[0] != d:
            raise ValueError("norm_g must have d entries")
    if gate is not None:
        _need_cuda("out_gate", gate, (torch.float32,))
        if B is not None and gate.numel() != B * d:
            raise ValueError(f"out_gate must be [B][d] = [{B}][{d}]")
    return LayerWeights(wg.data_ptr(), wu.data_ptr(), wd.data_ptr(), _ptr(g), _ptr(gate))


def _activations(x: torch.Tensor, y: torch.Tensor, d: int) -> Tuple[int, int]:
    _need_cuda("x", x, (torch.float32,), 3)
    _need_cuda("y", y, (torch.float32,), 3)
    if x.shape != y.shape or x.shape[2] != d:
        raise ValueError(f"x {tuple(x.shape)} and y {tuple(y.shape)} must both be [B][T][{d}]")
    return int(x.shape[0]), int(x.shape[1])


# ----------------------------------------------------------------------------------------------------------
# The C ABI calls
# ----------------------------------------------------------------------------------------------------------

def rm_mask_compact(mask: torch.Tensor, idx: torch.Tensor, count: torch.Tensor, stream=None) -> None:
    """mask uint8/bool [N][d_ff] -> idx int32 [N][d_ff] (ascending, -1 tail) and count int32 [N]."""
    _need_cuda("mask", mask, (torch.uint8, torch.bool), 2)
    n, d_ff = mask.shape
    _need_cuda("idx", idx, (torch.int32,))
    _need_cuda("count", count, (torch.int32,))
    if idx.numel() != n * d_ff or count.numel() != n:
        raise ValueError("idx must hold N*d_ff and count N entries")
    _check(load_library().rm_mask_compact(mask.data_ptr(), n, d_ff, idx.data_ptr(), count.data_ptr(),
                                          _stream(stream)))


def rm_workspace_size(d: int, d_ff: int, wdtype: int, B: int, T: int, max_count: int, eps: float = 1e-6) -> int:
    out = ctypes.c_size_t(0)
    shape = FfnShape(d, d_ff, wdtype, eps)
    _check(load_library().rm_workspace_size(ctypes.byref(shape), B, T, max_count, ctypes.byref(out)))
    return int(out.value)


def rm_layer_kernels(d: int, d_ff: int, wdtype: int, B: int, T: int, max_count: int, eps: float = 1e-6) -> int:
    """Bit mask of the RM_KERNEL_* ids a single-layer call of this shape launches on the current device."""
    out = ctypes.c_uint32(0)
    shape = FfnShape(d, d_ff, wdtype, eps)
    _check(load_library().rm_layer_kernels(ctypes.byref(shape), B, T, max_count, ctypes.byref(out)))
    return int(out.value)


def workspace(d: int, d_ff: int, wdtype: int, B: int, T: int, max_count: int, device="cuda") -> torch.Tensor:
    """Allocate a workspace tensor (uint8) of the size rm_workspace_size asks for."""
    return torch.empty(rm_workspace_size(d, d_ff, wdtype, B, T, max_count), dtype=torch.uint8, device=device)


def _ws(ws: torch.Tensor) -> Tuple[int, int]:
    _need_cuda("ws", ws, (torch.uint8,))
    return ws.data_ptr(), ws.numel()


def rm_sparse_ffn_layer(x: torch.Tensor, y: torch.Tensor, layer: Layer, idx: torch.Tensor, count: torch.Tensor,
                        max_count: int, ws: torch.Tensor, eps: float = 1e-6, act: str = "silu", stream=None) -> None:
    """y = x + masked GLU FFN over the listed neurons (y may be x); act "silu" (SwiGLU) or "gelu_tanh" (GeGLU)."""
    shape = _shape(layer, eps, act)
    B, T = _activations(x, y, shape.d)
    w = _weights(layer, B)
    _need_cuda("idx", idx, (torch.int32,))
    _need_cuda("count", count, (torch.int32,))
    if idx.numel() != B * shape.d_ff or count.numel() != B:
        raise ValueError("idx must be [B][d_ff] and count [B]")
    wp, wn = _ws(ws)
    _check(load_library().rm_sparse_ffn_layer(ctypes.byref(shape), ctypes.byref(w), B, T, x.data_ptr(),
                                              y.data_ptr(), idx.data_ptr(), count.data_ptr(), int(max_count),
                                              wp, wn, _stream(stream)))


def rm_sparse_ffn_layer_noalloc(x: torch.Tensor, y: torch.Tensor, layer: Layer, idx: torch.Tensor,
                                count: torch.Tensor, max_count: int, eps: float = 1e-6, act: str = "silu",
                                stream=None) -> None:
    """rm_sparse_ffn_layer with the library's own per-device scratch instead of a workspace (no allocation; calls
    that may overlap on one GPU must be ordered by the caller)."""
    shape = _shape(layer, eps, act)
    B, T = _activations(x, y, shape.d)
    w = _weights(layer, B)
    _need_cuda("idx", idx, (torch.int32,))
    _need_cuda("count", count, (torch.int32,))
    if idx.numel() != B * shape.d_ff or count.numel() != B:
        raise ValueError("idx must be [B][d_ff] and count [B]")
    _check(load_library().rm_sparse_ffn_layer_noalloc(ctypes.byref(shape), ctypes.byref(w), B, T, x.data_ptr(),
                                                      y.data_ptr(), idx.data_ptr(), count.data_ptr(),
                                                      int(max_count), _stream(stream)))


def _stack_args(x: torch.Tensor, y: torch.Tensor, layers: Sequence[Layer], idx: torch.Tensor,
                count: torch.Tensor, eps: float, act: str):
    L = len(layers)
    if L == 0:
        raise ValueError("at least one layer")
    shape = _shape(layers[0], eps, act)
    B, T = _activations(x, y, shape.d)
    arr = (LayerWeights * L)()
    for l, layer in enumerate(layers):
        s = _shape(layer, eps, act)
        if (s.d, s.d_ff, s.wdtype) != (shape.d, shape.d_ff, shape.wdtype):
            raise ValueError("every layer of a stack must have the same shape and dtype")
        arr[l] = _weights(layer, B)
    _need_cuda("idx", idx, (torch.int32,))
    _need_cuda("count", count, (torch.int32,))
    if idx.numel() != L * B * shape.d_ff or count.numel() != L * B:
        raise ValueError("idx must be [L][B][d_ff] and count [L][B]")
    return shape, arr, L, B, T


def _anchor_state(y_anchor: torch.Tensor, h_anchor: torch.Tensor, L: int, B: int, T: int, d: int,
                  max_count: int) -> None:
    _need_cuda("y_anchor", y_anchor, (torch.float32,))
    _need_cuda("h_anchor", h_anchor, (torch.float32,))
    if tuple(y_anchor.shape) != (L, B, T, d):
        raise ValueError(f"y_anchor has shape {tuple(y_anchor.shape)}, expected {(L, B, T, d)}")
    if tuple(h_anchor.shape) != (L, B, max_count, T):
        raise ValueError(f"h_anchor has shape {tuple(h_anchor.shape)}, expected {(L, B, max_count, T)}")


def rm_sparse_ffn_stack(x: torch.Tensor, y: torch.Tensor, layers: Sequence[Layer], idx: torch.Tensor,
                        count: torch.Tensor, max_count: int, ws: torch.Tensor, eps: float = 1e-6, act: str = "silu",
                        stream=None) -> None:
    """L masked FFN layers in order; idx [L][B][d_ff], count [L][B]."""
    shape, arr, L, B, T = _stack_args(x, y, layers, idx, count, eps, act)
    wp, wn = _ws(ws)
    _check(load_library().rm_sparse_ffn_stack(ctypes.byref(shape), arr, L, B, T, x.data_ptr(), y.data_ptr(),
                                              idx.data_ptr(), count.data_ptr(), int(max_count), wp, wn,
                                              _stream(stream)))


def _masks(mask: torch.Tensor, idx: torch.Tensor, count: torch.Tensor, n: int, d_ff: int) -> None:
    _need_cuda("mask", mask, (torch.uint8, torch.bool))
    _need_cuda("idx", idx, (torch.int32,))
    _need_cuda("count", count, (torch.int32,))
    if mask.numel() != n * d_ff or idx.numel() != n * d_ff or count.numel() != n:
        raise ValueError(f"mask and idx must hold {n} x d_ff={d_ff} and count {n} entries")


def rm_masked_ffn_layer(x: torch.Tensor, y: torch.Tensor, layer: Layer, mask: torch.Tensor, idx: torch.Tensor,
                        count: torch.Tensor, max_count: int, ws: torch.Tensor, eps: float = 1e-6, act: str = "silu",
                        stream=None) -> None:
    """rm_mask_compact(mask -> idx, count) + rm_sparse_ffn_layer, the compaction inside the layer's first launch."""
    shape = _shape(layer, eps, act)
    B, T = _activations(x, y, shape.d)
    w = _weights(layer, B)
    _masks(mask, idx, count, B, shape.d_ff)
    wp, wn = _ws(ws)
    _check(load_library().rm_masked_ffn_layer(ctypes.byref(shape), ctypes.byref(w), B, T, x.data_ptr(),
                                              y.data_ptr(), mask.data_ptr(), idx.data_ptr(), count.data_ptr(),
                                              int(max_count), wp, wn, _stream(stream)))


def rm_masked_ffn_stack(x: torch.Tensor, y: torch.Tensor, layers: Sequence[Layer], mask: torch.Tensor,
                        idx: torch.Tensor, count: torch.Tensor, max_count: int, ws: torch.Tensor, eps: float = 1e-6,
                        act: str = "silu", stream=None) -> None:
    """rm_mask_compact of [L][B] masks + rm_sparse_ffn_stack, the compaction inside the stack's first launch."""
    shape, arr, L, B, T = _stack_args(x, y, layers, idx, count, eps, act)
    _masks(mask, idx, count, L * B, shape.d_ff)
    wp, wn = _ws(ws)
    _check(load_library().rm_masked_ffn_stack(ctypes.byref(shape), arr, L, B, T, x.data_ptr(), y.data_ptr(),
                                              mask.data_ptr(), idx.data_ptr(), count.data_ptr(), int(max_count),
                                              wp, wn, _stream(stream)))


def rm_anchor_ffn_stack(x: torch.Tensor, y: torch.Tensor, layers: Sequence[Layer], idx: torch.Tensor,
                        count: torch.Tensor, max_count: int, y_anchor: torch.Tensor, h_anchor: torch.Tensor,
                        ws: torch.Tensor, eps: float = 1e-6, act: str = "silu", stream=None) -> None:
    """Eq. 4 anchor step: L dense layers; keeps y_a [L][B][T][d] and h_a of the group's lists [L][B][max_count][T].
    The workspace is sized with max_count = d_ff."""
    shape, arr, L, B, T = _stack_args(x, y, layers, idx, count, eps, act)
    _anchor_state(y_anchor, h_anchor, L, B, T, shape.d, int(max_count))
    wp, wn = _ws(ws)
    _check(load_library().rm_anchor_ffn_stack(ctypes.byref(shape), arr, L, B, T, x.data_ptr(), y.data_ptr(),
                                              idx.data_ptr(), count.data_ptr(), int(max_count),
                                              y_anchor.data_ptr(), h_anchor.data_ptr(), wp, wn, _stream(stream)))


def rm_delta_ffn_stack(x: torch.Tensor, y: torch.Tensor, layers: Sequence[Layer], idx: torch.Tensor,
                       count: torch.Tensor, max_count: int, y_anchor: torch.Tensor, h_anchor: torch.Tensor,
                       ws: torch.Tensor, eps: float = 1e-6, act: str = "silu", stream=None) -> None:
    """Eq. 4 non-anchor step: y = x + y_a + (h - h_a) W_down over the listed neurons, per layer."""
    shape, arr, L, B, T = _stack_args(x, y, layers, idx, count, eps, act)
    _anchor_state(y_anchor, h_anchor, L, B, T, shape.d, int(max_count))
    wp, wn = _ws(ws)
    _check(load_library().rm_delta_ffn_stack(ctypes.byref(shape), arr, L, B, T, x.data_ptr(), y.data_ptr(),
                                             idx.data_ptr(), count.data_ptr(), int(max_count),
                                             y_anchor.data_ptr(), h_anchor.data_ptr(), wp, wn, _stream(stream)))


def rm_dense_ffn_ref(x: torch.Tensor, y: torch.Tensor, layer: Layer, ws: torch.Tensor, eps: float = 1e-6,
                     act: str = "silu", stream=None) -> None:
    """y = x + dense GLU FFN (every neuron)."""
    shape = _shape(layer, eps, act)
    B, T = _activations(x, y, shape.d)
    w = _weights(layer, B)
    wp, wn = _ws(ws)
    _check(load_library().rm_dense_ffn_ref(ctypes.byref(shape), ctypes.byref(w), B, T, x.data_ptr(), y.data_ptr(),
                                           wp, wn, _stream(stream)))


def rm_gather_stack_rows(layers: Sequence[Layer], idx: torch.Tensor, count: torch.Tensor, max_count: int,
                         out: torch.Tensor, stream=None) -> None:
    """Compact copies of each layer's listed rows: out [L][3][max_count][d] (w_gate, w_up, w_down rows), rows past
    a layer's count zero; idx [L][d_ff], count [L] (one list per layer)."""
    L = len(layers)
    if L == 0:
        raise ValueError("at least one layer")
    shape = _shape(layers[0], 1e-6)
    arr = (LayerWeights * L)()
    for l, layer in enumerate(layers):
        arr[l] = _weights(layer)
    _need_cuda("idx", idx, (torch.int32,))
    _need_cuda("count", count, (torch.int32,))
    _need_cuda("out", out, (layers[0][0].dtype,))
    if idx.numel() != L * shape.d_ff or count.numel() != L or out.numel() != L * 3 * max_count * shape.d:
        raise ValueError("idx must be [L][d_ff], count [L] and out [L][3][max_count][d]")
    _check(load_library().rm_gather_stack_rows(ctypes.byref(shape), arr, L, idx.data_ptr(), count.data_ptr(),
                                               int(max_count), out.data_ptr(), _stream(stream)))


def rm_context_select(x: torch.Tensor, x_ref: torch.Tensor, v0: int, P: int, k: int, drift: Optional[torch.Tensor],
                      rows: torch.Tensor, count: torch.Tensor, stream=None) -> None:
    """Eq. 2 drift of the visual rows [v0, v0 + P) of x [N][d] against x_ref, and the rows to recompute: every
    non-visual row plus the k visual rows of largest drift (ascending, in rows[:count[0]])."""
    _need_cuda("x", x, (torch.float32,), 2)
    _need_cuda("x_ref", x_ref, (torch.float32,), 2)
    if x.shape != x_ref.shape:
        raise ValueError("x and x_ref must have the same shape")
    n_tok, d = x.shape
    if drift is not None:
        _need_cuda("drift", drift, (torch.float32,))
        if drift.numel() < P:
            raise ValueError("drift must hold P entries")
    _need_cuda("rows", rows, (torch.int32,))
    _need_cuda("count", count, (torch.int32,))
    if rows.numel() < n_tok or count.numel() < 1:
        raise ValueError("rows must hold N entries and count one")
    _check(load_library().rm_context_select(x.data_ptr(), x_ref.data_ptr(), n_tok, d, int(v0), int(P), int(k),
                                            _ptr(drift), rows.data_ptr(), count.data_ptr(), _stream(stream)))


def context_workspace(d: int, d_ff: int, n_tok: int, max_rows: int, act: str = "gelu_tanh", device="cuda"):
    """A workspace tensor (uint8) of the size rm_context_workspace_size asks for."""
    out = ctypes.c_size_t(0)
    shape = FfnShape(d, d_ff, RM_BF16, 1e-6, ACTS[act])
    _check(load_library().rm_context_workspace_size(ctypes.byref(shape), n_tok, max_rows, ctypes.byref(out)))
    return torch.empty(int(out.value), dtype=torch.uint8, device=device)


def rm_context_ffn(x: torch.Tensor, y: torch.Tensor, w_gate: torch.Tensor, w_up: torch.Tensor,
                   w_down_t: torch.Tensor, rows: torch.Tensor, count: torch.Tensor, max_rows: int, ws: torch.Tensor,
                   act: str = "gelu_tanh", stream=None) -> None:
    """Eq. 3: y[rows[:count]] = F(x[rows[:count]]); other rows of y (the reference outputs) are left as they are.
    w_gate, w_up bf16 [d_ff][d]; w_down_t bf16 [d][d_ff] (nn.Linear layout)."""
    _need_cuda("x", x, (torch.float32,), 2)
    _need_cuda("y", y, (torch.float32,), 2)
    if x.shape != y.shape:
        raise ValueError("x and y must have the same shape")
    n_tok, d = x.shape
    _need_cuda("w_gate", w_gate, (torch.bfloat16,), 2)
    d_ff = w_gate.shape[0]
    for name, w, shp in (("w_gate", w_gate, (d_ff, d)), ("w_up", w_up, (d_ff, d)), ("w_down_t", w_down_t, (d, d_ff))):
        _need_cuda(name, w, (torch.bfloat16,), 2)
        if tuple(w.shape) != shp:
            raise ValueError(f"{name} has shape {tuple(w.shape)}, expected {shp}")
    _need_cuda("rows", rows, (torch.int32,))
    _need_cuda("count", count, (torch.int32,))
    if act not in ACTS:
        raise ValueError(f"act must be one of {sorted(ACTS)}")
    shape = FfnShape(d, d_ff, RM_BF16, 1e-6, ACTS[act])
    wp, wn = _ws(ws)
    _check(load_library().rm_context_ffn(ctypes.byref(shape), w_gate.data_ptr(), w_up.data_ptr(),
                                         w_down_t.data_ptr(), n_tok, x.data_ptr(), rows.data_ptr(), count.data_ptr(),
                                         int(max_rows), y.data_ptr(), wp, wn, _stream(stream)))


def rm_context_pack(w_gate: torch.Tensor, w_up: torch.Tensor, w_down_t: torch.Tensor, act: str = "gelu_tanh",
                    stream=None) -> torch.Tensor:
    """The layer's three matrices in the blocked layout rm_context_ffn_packed reads (a uint8 tensor of
    3 * d * d_ff * 2 bytes, allocated here).  Run once per layer when the weights are loaded."""
    _need_cuda("w_gate", w_gate, (torch.bfloat16,), 2)
    d_ff, d = w_gate.shape
    for name, w, shp in (("w_up", w_up, (d_ff, d)), ("w_down_t", w_down_t, (d, d_ff))):
        _need_cuda(name, w, (torch.bfloat16,), 2)
        if tuple(w.shape) != shp:
            raise ValueError(f"{name} has shape {tuple(w.shape)}, expected {shp}")
    if act not in ACTS:
        raise ValueError(f"act must be one of {sorted(ACTS)}")
    shape = FfnShape(d, d_ff, RM_BF16, 1e-6, ACTS[act])
    n = ctypes.c_size_t(0)
    lib = load_library()
    _check(lib.rm_context_pack_size(ctypes.byref(shape), ctypes.byref(n)))
    packed = torch.empty(int(n.value), dtype=torch.uint8, device=w_gate.device)
    _check(lib.rm_context_pack(ctypes.byref(shape), w_gate.data_ptr(), w_up.data_ptr(), w_down_t.data_ptr(),
                               packed.data_ptr(), packed.numel(), _stream(stream)))
    return packed


def rm_context_ffn_packed(x: torch.Tensor, y: torch.Tensor, packed: torch.Tensor, rows: torch.Tensor,
                          count: torch.Tensor, max_rows: int, ws: torch.Tensor, act: str = "gelu_tanh",
                          stream=None) -> None:
    """rm_context_ffn with the weights from rm_context_pack (d_ff follows from the packed size)."""
    _need_cuda("x", x, (torch.float32,), 2)
    _need_cuda("y", y, (torch.float32,), 2)
    if x.shape != y.shape:
        raise ValueError("x and y must have the same shape")
    n_tok, d = x.shape
    _need_cuda("packed", packed, (torch.uint8,))
    if packed.numel() % (6 * d) != 0:
        raise ValueError("packed does not hold the three matrices of a layer with this d")
    d_ff = packed.numel() // (6 * d)
    _need_cuda("rows", rows, (torch.int32,))
    _need_cuda("count", count, (torch.int32,))
    if act not in ACTS:
        raise ValueError(f"act must be one of {sorted(ACTS)}")
    shape = FfnShape(d, d_ff, RM_BF16, 1e-6, ACTS[act])
    wp, wn = _ws(ws)
    _check(load_library().rm_context_ffn_packed(ctypes.byref(shape), packed.data_ptr(), n_tok, x.data_ptr(),
                                                rows.data_ptr(), count.data_ptr(), int(max_rows), y.data_ptr(), wp,
                                                wn, _stream(stream)))


def rm_neuron_norms(w_down: torch.Tensor, norms: torch.Tensor, stream=None) -> None:
    """||W_down[n]||_2 per neuron (Eq. 1's weight factor): w_down [d_ff][d] -> norms float32 [d_ff]."""
    _need_cuda("w_down", w_down, (torch.float32, torch.bfloat16), 2)
    d_ff, d = w_down.shape
    _need_cuda("norms", norms, (torch.float32,))
    if norms.numel() != d_ff:
        raise ValueError(f"norms must hold d_ff={d_ff} entries")
    _check(load_library().rm_neuron_norms(w_down.data_ptr(), d_ff, d, wdtype_of(w_down), norms.data_ptr(),
                                          _stream(stream)))


def rm_group_masks(h: torch.Tensor, norms: torch.Tensor, k: int, scores: torch.Tensor, mask: torch.Tensor,
                   stream=None) -> None:
    """Group masks (section 5): h float32 [S][L][d_ff][T], norms [L][d_ff] -> scores float32 [S][L][d_ff] and
    mask uint8 [L][d_ff]."""
    _need_cuda("h", h, (torch.float32,), 4)
    S, L, d_ff, T = h.shape
    _need_cuda("norms", norms, (torch.float32,))
    _need_cuda("scores", scores, (torch.float32,))
    _need_cuda("mask", mask, (torch.uint8, torch.bool))
    if norms.numel() != L * d_ff or scores.numel() != S * L * d_ff or mask.numel() != L * d_ff:
        raise ValueError("norms must be [L][d_ff], scores [S][L][d_ff] and mask [L][d_ff]")
    _check(load_library().rm_group_masks(h.data_ptr(), S, L, d_ff, T, norms.data_ptr(), int(k), scores.data_ptr(),
                                         mask.data_ptr(), _stream(stream)))


def rm_profile_kernel_events(kernel: int, ev_begin: Optional[int], ev_end: Optional[int]) -> None:
    """Arm raw hipEvent_t handles around the next launch of `kernel` (an RM_KERNEL_* id)."""
    _check(load_library().rm_profile_kernel_events(kernel, ev_begin, ev_end))


def rm_stream_read(buf: torch.Tensor, workgroups: int, sink: torch.Tensor, stream=None) -> None:
    """Measurement: a plain streaming read of the whole of `buf` (any dtype, 16-byte multiple); sink int32/uint8
    scratch of at least workgroups * 512 * 4 bytes."""
    if buf.device.type != "cuda" or not buf.is_contiguous():
        raise ValueError("buf must be a contiguous device tensor")
    _need_cuda("sink", sink, (torch.int32, torch.uint8))
    if sink.numel() * sink.element_size() < workgroups * 512 * 4:
        raise ValueError("sink must hold workgroups * 512 uint32")
    _check(load_library().rm_stream_read(buf.data_ptr(), buf.numel() * buf.element_size(), int(workgroups),
                                         sink.data_ptr(), _stream(stream)))
