"""Seeded synthetic inputs for the KAN-layer forward.

This module draws random numbers and nothing else: it holds none of the
method's arithmetic, so the HIP path and any float64 reference can consume the
same arrays.  Shapes and distributions follow the workloads the paper's
method is exercised on (uniform grid on [-1, 1], inputs mostly on the grid with
an optional off-grid fraction, Gaussian spline coefficients and base weights);
the second argument of every N(0, s) below is a standard deviation.

``round_to_bf16_f32`` is storage rounding (float32 -> nearest bfloat16, ties to
even, returned as float32) used to build bf16 inputs; it is not part of the
method.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Tuple

import numpy as np


@dataclasses.dataclass(frozen=True)
class LayerShape:
    batch: int
    n_in: int
    n_out: int
    grid_size: int
    lo: float = -1.0
    hi: float = 1.0
    off_grid_frac: float = 0.0     # fraction of x drawn from U(-4, 4) instead of U(lo, hi)
    coef_std: Optional[float] = None  # default 0.1
    base_std: Optional[float] = None  # default 1/n_in


# The named workloads.  Seeds are 42 + index (42 is the paper's first seed).
WORKLOADS = {
    "c1_layer_2x5_g5": dict(idx=0, layers=[(2, 5)], batch=1024, G=5),
    "c2_layer_64x64_g5": dict(idx=1, layers=[(64, 64)], batch=4096, G=5),
    "c3_layer_256x256_g10_offgrid": dict(idx=2, layers=[(256, 256)], batch=16384, G=10,
                                         off_grid_frac=0.1),
    "c4_layer_128x128_g50": dict(idx=3, layers=[(128, 128)], batch=8192, G=50, coef_scale_g=True),
    "c4_layer_128x128_g100": dict(idx=3, layers=[(128, 128)], batch=8192, G=100, coef_scale_g=True),
    "c4_layer_128x128_g200": dict(idx=3, layers=[(128, 128)], batch=8192, G=200, coef_scale_g=True),
    "c5_mlp_784_256_256_10_g10": dict(idx=4, layers=[(784, 256), (256, 256), (256, 10)],
                                      batch=65536, G=10),
}


def round_to_bf16_f32(a: np.ndarray) -> np.ndarray:
    """float32 -> nearest bfloat16 (ties to even), returned as float32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    nan = np.isnan(a)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    out = r.astype(np.uint32).view(np.float32).copy()
    out[nan] = np.float32("nan")
    return out


def draw_x(rng: np.random.Generator, batch: int, n_in: int, lo: float = -1.0, hi: float = 1.0,
           off_grid_frac: float = 0.0) -> np.ndarray:
    """x ~ U(lo, hi), with a fraction ``off_grid_frac`` replaced by U(-4, 4).
    Both arrays are drawn full-size so the result does not depend on the mask."""
    x = rng.uniform(lo, hi, size=(batch, n_in)).astype(np.float32)
    if off_grid_frac > 0.0:
        m = rng.random(size=(batch, n_in)) < off_grid_frac
        wide = rng.uniform(-4.0, 4.0, size=(batch, n_in)).astype(np.float32)
        x = np.where(m, wide, x).astype(np.float32)
    return x


def draw_weights(rng: np.random.Generator, n_in: int, n_out: int, G: int, k: int = 3,
                 coef_std: float = 0.1, base_std: Optional[float] = None
                 ) -> Tuple[np.ndarray, np.ndarray]:
    """C ~ N(0, coef_std) of shape [out, in, G + k]; Wb ~ N(0, base_std), [out, in]."""
    if base_std is None:
        base_std = 1.0 / n_in
    C = rng.normal(0.0, coef_std, size=(n_out, n_in, G + k)).astype(np.float32)
    Wb = rng.normal(0.0, base_std, size=(n_out, n_in)).astype(np.float32)
    return C, Wb


def make_layer(shape: LayerShape, seed: int, k: int = 3):
    """(x, C, Wb) float32 arrays for one layer of the given shape."""
    rng = np.random.default_rng(seed)
    x = draw_x(rng, shape.batch, shape.n_in, shape.lo, shape.hi, shape.off_grid_frac)
    C, Wb = draw_weights(rng, shape.n_in, shape.n_out, shape.grid_size, k,
                         0.1 if shape.coef_std is None else shape.coef_std,
                         shape.base_std)
    return x, C, Wb


def make_workload(name: str, batch: Optional[int] = None):
    """Inputs of a named workload: dict with x [B, in0] and a list of (C, Wb).

    x and the weights come from two separate streams of the workload's seed, so
    ``batch`` (default: the workload's own) changes only x, and the weights are
    the same at every batch size."""
    spec = WORKLOADS[name]
    B = spec["batch"] if batch is None else batch
    G = spec["G"]
    seed = 42 + spec["idx"]
    rng_x = np.random.default_rng([seed, G, 0])
    rng_w = np.random.default_rng([seed, G, 1])
    n_in0 = spec["layers"][0][0]
    x = draw_x(rng_x, B, n_in0, -1.0, 1.0, spec.get("off_grid_frac", 0.0))
    coef_std = 0.1 / np.sqrt(G) if spec.get("coef_scale_g") else 0.1
    layers: List[Tuple[np.ndarray, np.ndarray]] = []
    for (n_in, n_out) in spec["layers"]:
        layers.append(draw_weights(rng_w, n_in, n_out, G, 3, coef_std, 1.0 / n_in))
    return dict(name=name, G=G, lo=-1.0, hi=1.0, x=x, layers=layers)
