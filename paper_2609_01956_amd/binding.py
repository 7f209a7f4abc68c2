"""Python binding of the C ABI in include/kan.h (ctypes).

Argument marshalling only: every step of the computation runs in the HIP
kernels of ``libkan.so``.  The raw entry points keep the C names
(``kan_basis_eval``, ``kan_layer_forward``, ``kan_status_string``) and take
device addresses as integers; ``basis``, ``layer_forward`` and ``mlp_forward``
accept torch tensors on a ROCm device and launch on torch's current stream.

The library must have been built (``python -m paper_2609_01956_amd.build``);
loading raises if it is missing.  There is no fallback of any kind.
"""
from __future__ import annotations

import ctypes
import os
import threading
from typing import Iterable, Optional, Sequence, Tuple

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libkan.so")

KAN_OK = 0
KAN_ERR_INVALID_ARG = 1
KAN_ERR_UNSUPPORTED = 2
KAN_ERR_DEVICE = 3
KAN_ERR_SCRATCH_LIMIT = 4
KAN_NOALLOC_SCRATCH_BYTES = 16 << 20

KAN_F32 = 0
KAN_BF16 = 1

EXPORTED_SYMBOLS = ("kan_basis_eval", "kan_basis_eval_cdb", "kan_layer_forward", "kan_layer_forward_workspace_bytes",
                    "kan_layer_packed_bytes", "kan_layer_pack", "kan_layer_forward_packed",
                    "kan_layer_forward_packed_workspace_bytes",
                    "kan_layer_plan", "kan_layer_forward_noalloc", "kan_layer_backward",
                    "kan_layer_backward_workspace_bytes", "kan_layer_forward_span",
                    "kan_layer_forward_span_workspace_bytes", "kan_status_string",
                    "kan_abi_version")

_VP = ctypes.c_void_p
_I32P = ctypes.POINTER(ctypes.c_int32)


class kan_grid(ctypes.Structure):
    _fields_ = [("grid_size", ctypes.c_int32), ("spline_order", ctypes.c_int32),
                ("grid_lo", ctypes.c_float), ("grid_hi", ctypes.c_float)]


class KanError(RuntimeError):
    pass


_lock = threading.Lock()
_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libkan.so once; raise if it has not been built."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(path):
                raise RuntimeError(
                    f"{path} is missing: build the HIP library first "
                    "(python -m paper_2609_01956_amd.build)")
            lib = ctypes.CDLL(path)
            lib.kan_basis_eval.argtypes = [ctypes.POINTER(kan_grid), ctypes.c_int, ctypes.c_void_p,
                                           ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p]
            lib.kan_basis_eval.restype = ctypes.c_int
            lib.kan_basis_eval_cdb.argtypes = lib.kan_basis_eval.argtypes
            lib.kan_basis_eval_cdb.restype = ctypes.c_int
            g = ctypes.POINTER(kan_grid)
            lib.kan_layer_forward.argtypes = [g, ctypes.c_int, ctypes.c_int64, ctypes.c_int32,
                                              ctypes.c_int32, _VP, _VP, _VP, _VP, ctypes.c_size_t,
                                              _VP, _VP]
            lib.kan_layer_forward.restype = ctypes.c_int
            lib.kan_layer_forward_workspace_bytes.argtypes = [g, ctypes.c_int, ctypes.c_int64,
                                                              ctypes.c_int32, ctypes.c_int32,
                                                              ctypes.POINTER(ctypes.c_size_t)]
            lib.kan_layer_forward_workspace_bytes.restype = ctypes.c_int
            lib.kan_layer_packed_bytes.argtypes = [g, ctypes.c_int, ctypes.c_int32,
                                                   ctypes.c_int32, ctypes.POINTER(ctypes.c_size_t)]
            lib.kan_layer_packed_bytes.restype = ctypes.c_int
            lib.kan_layer_pack.argtypes = [g, ctypes.c_int, ctypes.c_int32, ctypes.c_int32, _VP,
                                           _VP, _VP, ctypes.c_size_t, _VP]
            lib.kan_layer_pack.restype = ctypes.c_int
            lib.kan_layer_forward_packed.argtypes = [g, ctypes.c_int, ctypes.c_int64,
                                                     ctypes.c_int32, ctypes.c_int32, _VP, _VP,
                                                     ctypes.c_size_t, _I32P, _VP,
                                                     ctypes.c_size_t, _VP, _VP]
            lib.kan_layer_forward_packed.restype = ctypes.c_int
            lib.kan_layer_forward_packed_workspace_bytes.argtypes = [
                g, ctypes.c_int, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, _I32P,
                ctypes.POINTER(ctypes.c_size_t)]
            lib.kan_layer_forward_packed_workspace_bytes.restype = ctypes.c_int
            lib.kan_layer_plan.argtypes = [g, ctypes.c_int, ctypes.c_int64, ctypes.c_int32,
                                           ctypes.c_int32, _I32P, _I32P]
            lib.kan_layer_plan.restype = ctypes.c_int
            lib.kan_layer_forward_noalloc.argtypes = [g, ctypes.c_int, ctypes.c_int64,
                                                      ctypes.c_int32, ctypes.c_int32, _VP, _VP,
                                                      _VP, _VP, _VP]
            lib.kan_layer_forward_noalloc.restype = ctypes.c_int
            lib.kan_layer_backward.argtypes = [g, ctypes.c_int, ctypes.c_int64, ctypes.c_int32,
                                               ctypes.c_int32, _VP, _VP, _VP, _VP, _VP, _VP, _VP,
                                               _VP, ctypes.c_size_t, _VP]
            lib.kan_layer_backward.restype = ctypes.c_int
            lib.kan_layer_backward_workspace_bytes.argtypes = [g, ctypes.c_int, ctypes.c_int64,
                                                               ctypes.c_int32, ctypes.c_int32,
                                                               ctypes.POINTER(ctypes.c_size_t)]
            lib.kan_layer_backward_workspace_bytes.restype = ctypes.c_int
            lib.kan_layer_forward_span.argtypes = lib.kan_layer_forward.argtypes
            lib.kan_layer_forward_span.restype = ctypes.c_int
            lib.kan_layer_forward_span_workspace_bytes.argtypes = \
                lib.kan_layer_forward_workspace_bytes.argtypes
            lib.kan_layer_forward_span_workspace_bytes.restype = ctypes.c_int
            lib.kan_status_string.argtypes = [ctypes.c_int]
            lib.kan_status_string.restype = ctypes.c_char_p
            lib.kan_abi_version.argtypes = []
            lib.kan_abi_version.restype = ctypes.c_int32
            _lib = lib
    return _lib


# ----------------------------------------------------------- raw C entry points

def make_grid(grid_size: int, grid_lo: float = -1.0, grid_hi: float = 1.0,
              spline_order: int = 3) -> kan_grid:
    return kan_grid(int(grid_size), int(spline_order), float(grid_lo), float(grid_hi))


def kan_status_string(status: int) -> str:
    return load_library().kan_status_string(int(status)).decode()


def kan_abi_version() -> int:
    return int(load_library().kan_abi_version())


def kan_basis_eval(grid: kan_grid, dtype: int, x: int, n: int, phi: int, stream: int = 0) -> int:
    """Raw call: device addresses as integers; returns the kan_status code."""
    return int(load_library().kan_basis_eval(ctypes.byref(grid), int(dtype), ctypes.c_void_p(x),
                                             int(n), ctypes.c_void_p(phi), ctypes.c_void_p(stream)))


def _shape_arg(shape):
    """None, or a forced workgroup shape (rf, wk, nw, cs) / "rf,wk[,nw[,cs]]"
    as an int32[4] (nw defaults to 4, cs to 1)."""
    if shape is None:
        return None
    if isinstance(shape, str):
        shape = [int(t) for t in shape.split(",")]
    v = list(shape) + [4, 1][len(shape) - 2:] if len(shape) < 4 else list(shape)
    if len(v) != 4:
        raise ValueError("a shape is (rf, wk[, nw[, cs]])")
    return (ctypes.c_int32 * 4)(*[int(t) for t in v])


def kan_basis_eval_cdb(grid: kan_grid, dtype: int, x: int, n: int, phi: int,
                       stream: int = 0) -> int:
    """Raw call: device addresses as integers; returns the kan_status code."""
    return int(load_library().kan_basis_eval_cdb(ctypes.byref(grid), int(dtype), _VP(x), int(n),
                                                 _VP(phi), _VP(stream)))


def kan_layer_forward(grid: kan_grid, dtype: int, batch: int, in_features: int,
                      out_features: int, x: int, coef: int, base_w: int, workspace: int,
                      workspace_bytes: int, y: int, stream: int = 0) -> int:
    """Raw call: device addresses as integers; returns the kan_status code."""
    return int(load_library().kan_layer_forward(
        ctypes.byref(grid), int(dtype), int(batch), int(in_features), int(out_features),
        _VP(x), _VP(coef), _VP(base_w), _VP(workspace), ctypes.c_size_t(workspace_bytes),
        _VP(y), _VP(stream)))


def kan_layer_forward_noalloc(grid: kan_grid, dtype: int, batch: int, in_features: int,
                              out_features: int, x: int, coef: int, base_w: int, y: int,
                              stream: int = 0) -> int:
    """Raw call: device addresses as integers; returns the kan_status code."""
    return int(load_library().kan_layer_forward_noalloc(
        ctypes.byref(grid), int(dtype), int(batch), int(in_features), int(out_features),
        _VP(x), _VP(coef), _VP(base_w), _VP(y), _VP(stream)))


def kan_layer_backward(grid: kan_grid, dtype: int, batch: int, in_features: int,
                       out_features: int, x: int, coef: int, base_w: int, dy: int, dx: int,
                       dcoef: int, dbase_w: int, workspace: int, workspace_bytes: int,
                       stream: int = 0) -> int:
    """Raw call: device addresses as integers (0 for NULL); returns the kan_status code."""
    return int(load_library().kan_layer_backward(
        ctypes.byref(grid), int(dtype), int(batch), int(in_features), int(out_features),
        _VP(x), _VP(coef), _VP(base_w), _VP(dy), _VP(dx), _VP(dcoef), _VP(dbase_w),
        _VP(workspace), ctypes.c_size_t(workspace_bytes), _VP(stream)))


def kan_layer_forward_span(grid: kan_grid, dtype: int, batch: int, in_features: int,
                           out_features: int, x: int, coef: int, base_w: int, workspace: int,
                           workspace_bytes: int, y: int, stream: int = 0) -> int:
    """Raw call: device addresses as integers; returns the kan_status code."""
    return int(load_library().kan_layer_forward_span(
        ctypes.byref(grid), int(dtype), int(batch), int(in_features), int(out_features),
        _VP(x), _VP(coef), _VP(base_w), _VP(workspace), ctypes.c_size_t(workspace_bytes),
        _VP(y), _VP(stream)))


def kan_layer_forward_span_workspace_bytes(grid: kan_grid, dtype: int, batch: int,
                                           in_features: int, out_features: int) -> Tuple[int, int]:
    """Raw call: returns (kan_status, bytes)."""
    n = ctypes.c_size_t(0)
    st = int(load_library().kan_layer_forward_span_workspace_bytes(
        ctypes.byref(grid), int(dtype), int(batch), int(in_features), int(out_features),
        ctypes.byref(n)))
    return st, int(n.value)


def kan_layer_backward_workspace_bytes(grid: kan_grid, dtype: int, batch: int, in_features: int,
                                       out_features: int) -> Tuple[int, int]:
    """Raw call: returns (kan_status, bytes)."""
    n = ctypes.c_size_t(0)
    st = int(load_library().kan_layer_backward_workspace_bytes(
        ctypes.byref(grid), int(dtype), int(batch), int(in_features), int(out_features),
        ctypes.byref(n)))
    return st, int(n.value)


def kan_layer_forward_workspace_bytes(grid: kan_grid, dtype: int, batch: int, in_features: int,
                                      out_features: int) -> Tuple[int, int]:
    """Raw call: returns (kan_status, bytes)."""
    n = ctypes.c_size_t(0)
    st = int(load_library().kan_layer_forward_workspace_bytes(
        ctypes.byref(grid), int(dtype), int(batch), int(in_features), int(out_features),
        ctypes.byref(n)))
    return st, int(n.value)


def kan_layer_packed_bytes(grid: kan_grid, dtype: int, in_features: int,
                           out_features: int) -> Tuple[int, int]:
    """Raw call: returns (kan_status, bytes)."""
    n = ctypes.c_size_t(0)
    st = int(load_library().kan_layer_packed_bytes(ctypes.byref(grid), int(dtype),
                                                   int(in_features), int(out_features),
                                                   ctypes.byref(n)))
    return st, int(n.value)


def kan_layer_plan(grid: kan_grid, dtype: int, batch: int, in_features: int,
                   out_features: int, shape=None) -> Tuple[int, Tuple[int, ...]]:
    """Raw call: returns (kan_status, (rf, wk, nw, cs, sparse, k_splits));
    `shape` forces a workgroup shape (see _shape_arg), None takes the
    library's choice."""
    plan = (ctypes.c_int32 * 6)()
    st = int(load_library().kan_layer_plan(ctypes.byref(grid), int(dtype), int(batch),
                                           int(in_features), int(out_features),
                                           _shape_arg(shape), plan))
    return st, tuple(int(v) for v in plan)


def kan_layer_pack(grid: kan_grid, dtype: int, in_features: int, out_features: int, coef: int,
                   base_w: int, packed: int, packed_bytes: int, stream: int = 0) -> int:
    """Raw call: device addresses as integers; returns the kan_status code."""
    return int(load_library().kan_layer_pack(
        ctypes.byref(grid), int(dtype), int(in_features), int(out_features), _VP(coef),
        _VP(base_w), _VP(packed), ctypes.c_size_t(packed_bytes), _VP(stream)))


def kan_layer_forward_packed(grid: kan_grid, dtype: int, batch: int, in_features: int,
                             out_features: int, x: int, packed: int, packed_bytes: int, y: int,
                             stream: int = 0, shape=None, workspace: int = 0,
                             workspace_bytes: int = 0) -> int:
    """Raw call: device addresses as integers; returns the kan_status code.
    `shape` forces a workgroup shape (see _shape_arg); `workspace` (0: none)
    holds the partial sums of a split contraction."""
    return int(load_library().kan_layer_forward_packed(
        ctypes.byref(grid), int(dtype), int(batch), int(in_features), int(out_features),
        _VP(x), _VP(packed), ctypes.c_size_t(packed_bytes), _shape_arg(shape), _VP(workspace),
        ctypes.c_size_t(workspace_bytes), _VP(y), _VP(stream)))


def kan_layer_forward_packed_workspace_bytes(grid: kan_grid, dtype: int, batch: int,
                                             in_features: int, out_features: int,
                                             shape=None) -> Tuple[int, int]:
    """Raw call: returns (kan_status, bytes)."""
    n = ctypes.c_size_t(0)
    st = int(load_library().kan_layer_forward_packed_workspace_bytes(
        ctypes.byref(grid), int(dtype), int(batch), int(in_features), int(out_features),
        _shape_arg(shape), ctypes.byref(n)))
    return st, int(n.value)


def check(status: int) -> None:
    """Map a kan_status to an exception."""
    if status == KAN_OK:
        return
    msg = kan_status_string(status)
    if status in (KAN_ERR_INVALID_ARG, KAN_ERR_SCRATCH_LIMIT):
        raise ValueError(msg)
    if status == KAN_ERR_UNSUPPORTED:
        raise NotImplementedError(msg)
    raise KanError(msg)


# ------------------------------------------------------------ torch marshalling

def _torch():
    import torch
    return torch


def _dtype_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.float32:
        return KAN_F32
    if t.dtype == torch.bfloat16:
        return KAN_BF16
    raise NotImplementedError(f"dtype {t.dtype} is not supported (float32 or bfloat16)")


def _require_device(*ts) -> None:
    for t in ts:
        if not t.is_cuda:
            raise ValueError("tensors must live on the GPU")
        if not t.is_contiguous():
            raise ValueError("tensors must be contiguous")
    dev = ts[0].device
    for t in ts[1:]:
        if t.device != dev:
            raise ValueError("tensors must live on one device")


def _stream(device) -> int:
    return int(_torch().cuda.current_stream(device).cuda_stream)


def basis(x, grid_size: int, grid_lo: float = -1.0, grid_hi: float = 1.0, out=None,
          spline_order: int = 3, method: str = "tp"):
    """phi[..., j] = N_j(x[...]) for j < grid_size + spline_order: the
    truncated-power form (kan_basis_eval, method "tp") or the Cox-de Boor
    recursion (kan_basis_eval_cdb, method "cdb")."""
    if method not in ("tp", "cdb"):
        raise ValueError("method is 'tp' or 'cdb'")
    torch = _torch()
    _require_device(x)
    nb = int(grid_size) + int(spline_order)
    if out is None:
        out = torch.empty(tuple(x.shape) + (nb,), dtype=x.dtype, device=x.device)
    else:
        _require_device(x, out)
        if out.dtype != x.dtype or tuple(out.shape) != tuple(x.shape) + (nb,):
            raise ValueError("out must have shape x.shape + (G + k,) and x's dtype")
    with torch.cuda.device(x.device):
        fn = kan_basis_eval if method == "tp" else kan_basis_eval_cdb
        check(fn(make_grid(grid_size, grid_lo, grid_hi, spline_order), _dtype_code(x),
                             x.data_ptr(),
                             x.numel(), out.data_ptr(), _stream(x.device)))
    return out


class PackedLayer:
    """Weights of one layer packed by kan_layer_pack (device buffer + shape)."""

    def __init__(self, buf, grid_size, grid_lo, grid_hi, n_in, n_out, dtype, spline_order=3):
        self.buf = buf
        self.spline_order = int(spline_order)
        self.grid_size, self.grid_lo, self.grid_hi = int(grid_size), float(grid_lo), float(grid_hi)
        self.n_in, self.n_out = int(n_in), int(n_out)
        self.dtype = dtype

    @property
    def nbytes(self) -> int:
        return int(self.buf.numel())


def _check_weights(coef, base_w, grid_size, spline_order=3):
    _require_device(coef, base_w)
    if base_w.dim() != 2 or coef.dim() != 3:
        raise ValueError("expected coef [out, in, G+3], base_w [out, in]")
    n_out, n_in = base_w.shape
    if tuple(coef.shape) != (n_out, n_in, int(grid_size) + int(spline_order)):
        raise ValueError("coef / base_w shapes do not match each other and the grid")
    if coef.dtype != base_w.dtype:
        raise ValueError("coef and base_w must share one dtype")
    return n_in, n_out


def pack_layer(coef, base_w, grid_size: int, grid_lo: float = -1.0, grid_hi: float = 1.0,
               out: Optional[PackedLayer] = None, spline_order: int = 3) -> PackedLayer:
    """kan_layer_pack: coef [out, in, G + 3], base_w [out, in] -> PackedLayer
    (device buffer from torch's allocator, filled on torch's current stream)."""
    torch = _torch()
    n_in, n_out = _check_weights(coef, base_w, grid_size, spline_order)
    dt = _dtype_code(coef)
    g = make_grid(grid_size, grid_lo, grid_hi, spline_order)
    st, nbytes = kan_layer_packed_bytes(g, dt, n_in, n_out)
    check(st)
    if out is None:
        buf = torch.empty(nbytes, dtype=torch.uint8, device=coef.device)
        out = PackedLayer(buf, grid_size, grid_lo, grid_hi, n_in, n_out, coef.dtype, spline_order)
    elif out.nbytes < nbytes or out.buf.device != coef.device:
        raise ValueError("packed buffer too small or on another device")
    else:
        # the buffer now holds these weights: its geometry follows them
        out.grid_size, out.grid_lo, out.grid_hi = int(grid_size), float(grid_lo), float(grid_hi)
        out.n_in, out.n_out, out.dtype = int(n_in), int(n_out), coef.dtype
        out.spline_order = int(spline_order)
    with torch.cuda.device(coef.device):
        check(kan_layer_pack(g, dt, n_in, n_out, coef.data_ptr(), base_w.data_ptr(),
                             out.buf.data_ptr(), out.nbytes, _stream(coef.device)))
    return out


def layer_forward_packed(x, packed: PackedLayer, out=None, shape=None, workspace=None,
                         split: bool = True):
    """kan_layer_forward_packed: x [B, in] with packed weights -> y [B, out].
    `shape` forces a workgroup shape (rf, wk[, nw[, cs]]) for tests and tuning.
    For batches too small to fill the GPU the contraction is split across
    workgroups; its partial sums go to `workspace` (a uint8 device tensor)
    when large enough, else to a fresh one from torch's allocator; split=False
    runs the layer unsplit."""
    torch = _torch()
    _require_device(x)
    if x.dim() != 2 or x.shape[1] != packed.n_in:
        raise ValueError("x must be [B, in] with the packed layer's in")
    if x.dtype != packed.dtype or packed.buf.device != x.device:
        raise ValueError("x must match the packed layer's dtype and device")
    B = x.shape[0]
    if out is None:
        out = torch.empty((B, packed.n_out), dtype=x.dtype, device=x.device)
    else:
        _require_device(x, out)
        if out.dtype != x.dtype or tuple(out.shape) != (B, packed.n_out):
            raise ValueError("out must be [B, out] with x's dtype")
    g = make_grid(packed.grid_size, packed.grid_lo, packed.grid_hi, packed.spline_order)
    dt = _dtype_code(x)
    ws_ptr, ws_bytes = 0, 0
    if split:
        st, need = kan_layer_forward_packed_workspace_bytes(g, dt, B, packed.n_in, packed.n_out,
                                                            shape)
        check(st)
        if need > 0:
            if workspace is None or workspace.numel() < need or workspace.device != x.device:
                workspace = torch.empty(need, dtype=torch.uint8, device=x.device)
            ws_ptr, ws_bytes = workspace.data_ptr(), workspace.numel()
    with torch.cuda.device(x.device):
        check(kan_layer_forward_packed(g, dt, B, packed.n_in, packed.n_out, x.data_ptr(),
                                       packed.buf.data_ptr(), packed.nbytes, out.data_ptr(),
                                       _stream(x.device), shape=shape, workspace=ws_ptr,
                                       workspace_bytes=ws_bytes))
    return out


def layer_forward(x, coef, base_w, grid_size: int, grid_lo: float = -1.0, grid_hi: float = 1.0,
                  out=None, packed: Optional[PackedLayer] = None, shape=None,
                  spline_order: int = 3):
    """One KAN layer: x [B, in], coef [out, in, G + 3], base_w [out, in] -> y
    [B, out], all of one dtype on one device.  Packs the weights (kan_layer_pack,
    into `packed` if given, else a fresh buffer) and runs
    kan_layer_forward_packed, both on torch's current stream; `shape` forces a
    workgroup shape."""
    _require_device(x)
    n_in, _ = _check_weights(coef, base_w, grid_size, spline_order)
    if x.dim() != 2 or x.shape[1] != n_in:
        raise ValueError("x must be [B, in] with coef's in")
    if coef.dtype != x.dtype:
        raise ValueError("x, coef and base_w must share one dtype")
    p = pack_layer(coef, base_w, grid_size, grid_lo, grid_hi, out=packed,
                   spline_order=spline_order)
    return layer_forward_packed(x, p, out=out, shape=shape)


def mlp_forward(x, layers: Sequence[Tuple[object, object]], grid_size: int, grid_lo: float = -1.0,
                grid_hi: float = 1.0, return_all: bool = False, spline_order: int = 3):
    """Stacked KAN layers; each output feeds the next layer unchanged (values
    off the grid are handled by the clamp of the basis)."""
    h = x
    outs = []
    for coef, base_w in layers:
        h = layer_forward(h, coef, base_w, grid_size, grid_lo, grid_hi,
                          spline_order=spline_order)
        outs.append(h)
    return outs if return_all else h


def layer_backward(x, coef, base_w, dy, grid_size: int, grid_lo: float = -1.0,
                   grid_hi: float = 1.0, need_dx: bool = True, need_dw: bool = True,
                   workspace=None, out=None):
    """Gradients of one KAN layer (kan_layer_backward): x [B, in], coef [out,
    in, G + 3], base_w [out, in], dy [B, out], all of one dtype on one device
    -> (dx [B, in] or None, dcoef or None, dbase_w or None), enqueued on
    torch's current stream.  `workspace` (a uint8 device tensor) is used when
    large enough, else a fresh one is taken from torch's allocator; `out`, a
    (dx, dcoef, dbase_w) tuple of tensors shaped like x, coef and base_w,
    receives the gradients instead of fresh tensors."""
    torch = _torch()
    _require_device(x, dy)
    n_in, n_out = _check_weights(coef, base_w, grid_size)
    if x.dim() != 2 or x.shape[1] != n_in or dy.shape != (x.shape[0], n_out):
        raise ValueError("x must be [B, in] and dy [B, out] for the weights' in and out")
    if not (x.dtype == dy.dtype == coef.dtype):
        raise ValueError("x, dy and the weights must share one dtype")
    if not (need_dx or need_dw):
        raise ValueError("nothing to compute")
    B = x.shape[0]
    dt = _dtype_code(x)
    g = make_grid(grid_size, grid_lo, grid_hi)
    st, nbytes = kan_layer_backward_workspace_bytes(g, dt, B, n_in, n_out)
    check(st)
    if workspace is None or workspace.numel() < nbytes or workspace.device != x.device:
        workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=x.device)
    if out is not None:
        dx, dC, dW = out
        for t, like in ((dx, x), (dC, coef), (dW, base_w)):
            if t is not None and (t.shape != like.shape or t.dtype != like.dtype or
                                  t.device != like.device or not t.is_contiguous()):
                raise ValueError("out tensors must match x, coef and base_w")
        dx = dx if need_dx else None
        dC, dW = (dC, dW) if need_dw else (None, None)
    else:
        dx = torch.empty_like(x) if need_dx else None
        dC = torch.empty_like(coef) if need_dw else None
        dW = torch.empty_like(base_w) if need_dw else None
    ptr = lambda t: 0 if t is None else t.data_ptr()
    with torch.cuda.device(x.device):
        check(kan_layer_backward(g, dt, B, n_in, n_out, x.data_ptr(), coef.data_ptr(),
                                 base_w.data_ptr(), dy.data_ptr(), ptr(dx), ptr(dC), ptr(dW),
                                 workspace.data_ptr(), workspace.numel(), _stream(x.device)))
    return dx, dC, dW


def layer_forward_span(x, coef, base_w, grid_size: int, grid_lo: float = -1.0,
                       grid_hi: float = 1.0, out=None, spline_order: int = 3, workspace=None):
    """kan_layer_forward_span: the layer on its nonzero terms only (the k + 1
    bases whose support holds each input, and SiLU); x [B, in], coef [out, in,
    G + k], base_w [out, in] -> y [B, out], on torch's current stream."""
    torch = _torch()
    _require_device(x)
    n_in, n_out = _check_weights(coef, base_w, grid_size, spline_order)
    if x.dim() != 2 or x.shape[1] != n_in or x.dtype != coef.dtype:
        raise ValueError("x must be [B, in] with the weights' in and dtype")
    B = x.shape[0]
    dt = _dtype_code(x)
    g = make_grid(grid_size, grid_lo, grid_hi, spline_order)
    st, nbytes = kan_layer_forward_span_workspace_bytes(g, dt, B, n_in, n_out)
    check(st)
    if workspace is None or workspace.numel() < nbytes or workspace.device != x.device:
        workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=x.device)
    if out is None:
        out = torch.empty((B, n_out), dtype=x.dtype, device=x.device)
    with torch.cuda.device(x.device):
        check(kan_layer_forward_span(g, dt, B, n_in, n_out, x.data_ptr(), coef.data_ptr(),
                                     base_w.data_ptr(), workspace.data_ptr(), workspace.numel(),
                                     out.data_ptr(), _stream(x.device)))
    return out
