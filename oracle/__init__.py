"""Float64 CPU oracle for the InKAN KAN-layer forward.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  The product path
(the HIP library and its Python binding) never imports, loads or calls it, and
this package imports nothing from the product.

The arithmetic lives in ``kan_oracle.c`` (plain C, IEEE double, OpenMP over
independent rows); this module only builds it with gcc when no build is present
and marshals numpy arrays.  Each function cites the passage of the paper it
follows:

* ``knots``        -- uniform simple knots (Sec. 2, Step 3), read as
                      t_j = lo + (j - k) h for j = 0..G+2k.
* ``basis_tp``     -- truncated-power form (eq. general_truncated / eq. truncated)
                      with the bounded coordinate of eq. bounded.
* ``basis_cdb``    -- Cox-de Boor recursion (eq. cdb0, eq. cdbk).
* ``basis_seg``    -- cubic segment form T(tau) M_B-spline (eq. bspline_matrix).
* ``silu``         -- x / (1 + exp(-x)), the residual branch of eq. kan_forward.
* ``layer``        -- the KAN layer, eq. kan_forward.
* ``mlp``          -- layers applied in sequence, optionally with bf16 storage
                      rounding of every tensor (round-to-nearest-even).
* ``round_bf16``   -- double -> nearest bfloat16 value, ties to even.
* ``basis_tp_deriv`` -- dN_j/dx of the clamped form (eq. general_truncated
                      differentiated, times the derivative of eq. bounded's
                      clamp).
* ``silu_deriv``   -- sigma'(x) = s + x s (1 - s), s = 1 / (1 + exp(-x)).
* ``layer_backward`` -- gradients of eq. kan_forward for an upstream dy:
                      (dx, dC, dWb).

Pins (``tests/test_oracle_*.py``): closed forms printed by the paper, the
paper's M_B-spline matrix, scipy's B-spline basis elements, the three routes
against each other, partition of unity, support, symmetry, C^2 smoothness,
linear precision, layer special cases and pure-Python brute force.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "kan_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None

_D = ctypes.POINTER(ctypes.c_double)
_I64 = ctypes.c_int64


def build(force: bool = False) -> str:
    """Compile ``kan_oracle.c`` into ``liboracle.so`` with gcc (IEEE double)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-fno-fast-math",
               "-Wall", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_LIB):
                build()
            lib = ctypes.CDLL(_LIB)
            lib.kan_oracle_knots.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_double,
                                             ctypes.c_double, _D]
            lib.kan_oracle_basis_tp.argtypes = [_D, _I64, ctypes.c_int, ctypes.c_int,
                                                ctypes.c_double, ctypes.c_double, ctypes.c_int, _D]
            lib.kan_oracle_basis_cdb.argtypes = [_D, _I64, ctypes.c_int, ctypes.c_int,
                                                 ctypes.c_double, ctypes.c_double, _D]
            lib.kan_oracle_basis_seg.argtypes = [_D, _I64, ctypes.c_int, ctypes.c_double,
                                                 ctypes.c_double, _D]
            lib.kan_oracle_silu.argtypes = [_D, _I64, _D]
            lib.kan_oracle_layer.argtypes = [_D, _I64, ctypes.c_int, ctypes.c_int, _D, _D,
                                             ctypes.c_int, ctypes.c_int, ctypes.c_double,
                                             ctypes.c_double, ctypes.c_int, ctypes.c_int, _D]
            lib.kan_oracle_round_bf16.argtypes = [_D, _I64, _D]
            lib.kan_oracle_basis_tp_deriv.argtypes = [_D, _I64, ctypes.c_int, ctypes.c_int,
                                                      ctypes.c_double, ctypes.c_double, _D]
            lib.kan_oracle_silu_deriv.argtypes = [_D, _I64, _D]
            lib.kan_oracle_layer_backward.argtypes = [_D, _I64, ctypes.c_int, ctypes.c_int, _D,
                                                      _D, _D, ctypes.c_int, ctypes.c_int,
                                                      ctypes.c_double, ctypes.c_double, _D, _D,
                                                      _D]
            lib.kan_oracle_num_threads.restype = ctypes.c_int
            lib.kan_oracle_set_threads.argtypes = [ctypes.c_int]
            _lib = lib
    return _lib


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _p(a: np.ndarray):
    return a.ctypes.data_as(_D)


def _check_grid(G: int, k: int, lo: float, hi: float) -> None:
    if not (1 <= k <= 7):
        raise ValueError("oracle supports spline degree 1..7")
    if not (1 <= G <= 8192):
        raise ValueError("grid size out of range")
    if not (np.isfinite(lo) and np.isfinite(hi) and lo < hi):
        raise ValueError("grid range must be finite with lo < hi")


def num_threads() -> int:
    return int(_load().kan_oracle_num_threads())


def set_threads(n: int) -> None:
    _load().kan_oracle_set_threads(int(n))


def knots(G: int, lo: float = -1.0, hi: float = 1.0, k: int = 3) -> np.ndarray:
    """t_j = lo + (j - k) h, h = (hi - lo)/G, j = 0..G+2k (Sec. 2, Step 3)."""
    _check_grid(G, k, lo, hi)
    t = np.empty(G + 2 * k + 1, dtype=np.float64)
    _load().kan_oracle_knots(G, k, lo, hi, _p(t))
    return t


def basis_tp(x, G: int, lo: float = -1.0, hi: float = 1.0, k: int = 3,
             clamp: bool = True) -> np.ndarray:
    """Truncated-power basis, shape x.shape + (G + k,) (eq. general_truncated,
    eq. truncated; clamp to [0, k+1] per eq. bounded)."""
    _check_grid(G, k, lo, hi)
    xa = _f64(x)
    out = np.empty(xa.shape + (G + k,), dtype=np.float64)
    _load().kan_oracle_basis_tp(_p(xa), xa.size, G, k, lo, hi, int(bool(clamp)), _p(out))
    return out


def basis_cdb(x, G: int, lo: float = -1.0, hi: float = 1.0, k: int = 3) -> np.ndarray:
    """Cox-de Boor basis, shape x.shape + (G + k,) (eq. cdb0, eq. cdbk)."""
    _check_grid(G, k, lo, hi)
    xa = _f64(x)
    out = np.empty(xa.shape + (G + k,), dtype=np.float64)
    _load().kan_oracle_basis_cdb(_p(xa), xa.size, G, k, lo, hi, _p(out))
    return out


def basis_seg(x, G: int, lo: float = -1.0, hi: float = 1.0) -> np.ndarray:
    """Cubic segment-form basis, shape x.shape + (G + 3,) (eq. bspline_matrix)."""
    _check_grid(G, 3, lo, hi)
    xa = _f64(x)
    out = np.empty(xa.shape + (G + 3,), dtype=np.float64)
    _load().kan_oracle_basis_seg(_p(xa), xa.size, G, lo, hi, _p(out))
    return out


def silu(x) -> np.ndarray:
    """sigma(x) = x / (1 + exp(-x)) (residual branch of eq. kan_forward)."""
    xa = _f64(x)
    out = np.empty_like(xa)
    _load().kan_oracle_silu(_p(xa), xa.size, _p(out))
    return out


def layer(x, C, Wb, G: int, lo: float = -1.0, hi: float = 1.0, k: int = 3,
          basis: str = "tp", bf16_operands: bool = False) -> np.ndarray:
    """KAN layer y = Phi(x) C^T + silu(x) Wb^T (eq. kan_forward).

    x: [B, in]; C: [out, in, G + k]; Wb: [out, in]  ->  y: [B, out], float64.
    ``basis`` selects the truncated-power ("tp") or Cox-de Boor ("cdb") route.
    ``bf16_operands`` rounds every basis and SiLU value to bfloat16 before the
    contraction (what a bf16 matrix unit consumes); sums stay in double.
    """
    _check_grid(G, k, lo, hi)
    xa = _f64(x)
    Ca = _f64(C)
    Wa = _f64(Wb)
    if xa.ndim != 2:
        raise ValueError("x must be [B, in]")
    B, n_in = xa.shape
    n_out = Wa.shape[0]
    if Ca.shape != (n_out, n_in, G + k) or Wa.shape != (n_out, n_in):
        raise ValueError("coefficient shapes do not match x and the grid")
    kind = {"tp": 0, "cdb": 1}[basis]
    y = np.empty((B, n_out), dtype=np.float64)
    _load().kan_oracle_layer(_p(xa), B, n_in, n_out, _p(Ca), _p(Wa), G, k, lo, hi, kind,
                             int(bool(bf16_operands)), _p(y))
    return y


def round_bf16(v) -> np.ndarray:
    """Nearest bfloat16 value of each double, ties to even, as float64."""
    va = _f64(v)
    out = np.empty_like(va)
    _load().kan_oracle_round_bf16(_p(va), va.size, _p(out))
    return out


def mlp(x, layers, G: int, lo: float = -1.0, hi: float = 1.0, k: int = 3,
        bf16: bool = False, bf16_operands: bool = False, return_all: bool = False):
    """Apply ``layer`` for each (C, Wb) in ``layers``; each output feeds the next
    layer unchanged (off-grid values are handled by the clamp).  With ``bf16``
    every stored tensor -- the input, the coefficients and each layer's output --
    is rounded to bfloat16 first, mirroring bf16 storage with wide accumulation;
    ``bf16_operands`` additionally rounds the basis and SiLU operands of every
    contraction.  Returns the last output, or every layer's (input, output)
    pair."""
    h = _f64(x)
    if bf16:
        h = round_bf16(h)
    trace = []
    for C, Wb in layers:
        Ca, Wa = _f64(C), _f64(Wb)
        if bf16:
            Ca, Wa = round_bf16(Ca), round_bf16(Wa)
        y = layer(h, Ca, Wa, G, lo, hi, k, bf16_operands=bf16_operands)
        if bf16:
            y = round_bf16(y)
        trace.append((h, y))
        h = y
    return trace if return_all else h


def basis_tp_deriv(x, G: int, lo: float = -1.0, hi: float = 1.0, k: int = 3) -> np.ndarray:
    """dN_j/dx of the clamped truncated-power basis, shape x.shape + (G + k,):
    eq. general_truncated differentiated in x, times the derivative of the
    clamp of eq. bounded (1 for 0 < u < k + 1, else 0)."""
    _check_grid(G, k, lo, hi)
    xa = _f64(x)
    out = np.empty(xa.shape + (G + k,), dtype=np.float64)
    _load().kan_oracle_basis_tp_deriv(_p(xa), xa.size, G, k, lo, hi, _p(out))
    return out


def silu_deriv(x) -> np.ndarray:
    """sigma'(x) for sigma(x) = x / (1 + exp(-x))."""
    xa = _f64(x)
    out = np.empty_like(xa)
    _load().kan_oracle_silu_deriv(_p(xa), xa.size, _p(out))
    return out


def layer_backward(x, C, Wb, dy, G: int, lo: float = -1.0, hi: float = 1.0, k: int = 3):
    """Gradients of sum(dy * y) for y = layer(x, C, Wb) (eq. kan_forward):
    returns (dx [B, in], dC [out, in, G + k], dWb [out, in]), float64."""
    _check_grid(G, k, lo, hi)
    xa, Ca, Wa, ga = _f64(x), _f64(C), _f64(Wb), _f64(dy)
    if xa.ndim != 2:
        raise ValueError("x must be [B, in]")
    B, n_in = xa.shape
    n_out = Wa.shape[0]
    if Ca.shape != (n_out, n_in, G + k) or Wa.shape != (n_out, n_in) or ga.shape != (B, n_out):
        raise ValueError("shapes of C, Wb and dy do not match x and the grid")
    dx = np.empty((B, n_in))
    dC = np.empty((n_out, n_in, G + k))
    dW = np.empty((n_out, n_in))
    _load().kan_oracle_layer_backward(_p(xa), B, n_in, n_out, _p(Ca), _p(Wa), _p(ga), G, k, lo,
                                      hi, _p(dx), _p(dC), _p(dW))
    return dx, dC, dW
