"""GPU parity for spline degrees other than 3 (eq. general_truncated with the
clamp to [0, k + 1]) and for grids whose 1 / h and lo / h are not exact in
fp32 (the coordinate then carries the rounding residual of 1 / h as a second
term), against the float64 oracle through the C ABI.  Tolerances as for the
cubic: basis max-abs <= 1e-6 (fp32), partition of unity <= 1e-5 on
[lo, hi], layer normwise <= 1e-5 (fp32) and <= 2e-2 (bf16)."""
import math

import numpy as np
import pytest

import oracle
from paper_2609_01956_amd import binding as kb
from paper_2609_01956_amd import workloads as wl
from gpu_common import (BF16_LAYER_TOL, F32_BASIS_TOL, F32_LAYER_TOL, PU_TOL, device, normwise,
                        say, to_dev, to_host64, torch)

pytestmark = pytest.mark.gpu


def _points(G, k, lo, hi, n=20000, seed=0):
    """Random points over the whole knot range and past it, every knot and one
    fp32 ulp either side, and the grid ends."""
    rng = np.random.default_rng(seed)
    h = (hi - lo) / G
    t = oracle.knots(G, lo, hi, k=k).astype(np.float32)
    x = rng.uniform(lo - (k + 1.5) * h, hi + (k + 1.5) * h, n).astype(np.float32)
    extra = np.array([lo, hi], np.float32)
    return np.concatenate([x, t, np.nextafter(t, np.float32(np.inf)),
                           np.nextafter(t, np.float32(-np.inf)), extra]).astype(np.float32)


def _off_support(x, G, k, lo, hi, margin_h=1e-12):
    """[n, G+k] mask of inputs outside basis j's support by more than
    margin_h * h (the fp32 coordinate's rounding can move a point that close
    to a support end to either side of it when 1 / h is not exact)."""
    t = oracle.knots(G, lo, hi, k=k)
    xd = np.asarray(x, np.float64)[:, None]
    margin = margin_h * (hi - lo) / G
    return (xd < t[None, :G + k] - margin) | (xd > t[None, k + 1:G + 2 * k + 1] + margin)


@pytest.mark.parametrize("k", [1, 2, 4, 5, 6, 7])
@pytest.mark.parametrize("G", [5, 10, 50])
def test_basis_other_degrees(k, G):
    x = _points(G, k, -1.0, 1.0, seed=10 * k + G)
    say(f"basis degree {k} G={G}")
    phi = kb.basis(to_dev(x, torch.float32), G, spline_order=k)
    torch.cuda.synchronize()
    got = to_host64(phi)
    ref = oracle.basis_tp(x, G, k=k)
    assert np.abs(got - ref).max() <= F32_BASIS_TOL, np.abs(got - ref).max()
    assert np.all(got[_off_support(x, G, k, -1.0, 1.0)] == 0.0)
    xs = np.linspace(-1, 1, 2001, dtype=np.float32)
    pu = kb.basis(to_dev(xs, torch.float32), G, spline_order=k).double().sum(dim=1)
    assert float((pu - 1.0).abs().max()) <= PU_TOL


GRIDS = [(1000, 0.0, 3.0), (200, -math.pi, math.pi), (10, 100.0, 103.0), (37, -0.3, 2.9)]


@pytest.mark.parametrize("G,lo,hi", GRIDS)
def test_basis_non_dyadic_grids(G, lo, hi):
    lo32, hi32 = float(np.float32(lo)), float(np.float32(hi))
    x = _points(G, 3, lo32, hi32, seed=G)
    say(f"basis grid G={G} [{lo32}, {hi32}]")
    phi = kb.basis(to_dev(x, torch.float32), G, lo32, hi32)
    torch.cuda.synchronize()
    got = to_host64(phi)
    ref = oracle.basis_tp(x, G, lo32, hi32)
    assert np.abs(got - ref).max() <= F32_BASIS_TOL, np.abs(got - ref).max()
    assert np.all(got[_off_support(x, G, 3, lo32, hi32, margin_h=1e-5)] == 0.0)


def _layer_case(B, n_in, n_out, G, k, lo, hi, dtype_name, seed):
    rng = np.random.default_rng(seed)
    h = (hi - lo) / G
    x = rng.uniform(lo - 2 * h, hi + 2 * h, (B, n_in)).astype(np.float32)
    _, C, Wb = wl.make_layer(wl.LayerShape(B, n_in, n_out, G), seed, k=k)
    if dtype_name == "bf16":
        x, C, Wb = (wl.round_to_bf16_f32(a) for a in (x, C, Wb))
    return x, C, Wb


@pytest.mark.parametrize("dtype_name", ["f32", "bf16"])
@pytest.mark.parametrize("k,G,n_in,n_out", [(1, 5, 9, 40), (2, 10, 17, 64), (4, 8, 7, 256),
                                            (5, 20, 12, 100), (7, 5, 3, 33)])
def test_layer_other_degrees(k, G, n_in, n_out, dtype_name):
    B = 300
    x, C, Wb = _layer_case(B, n_in, n_out, G, k, -1.0, 1.0, dtype_name, seed=k + G)
    dt = torch.float32 if dtype_name == "f32" else torch.bfloat16
    say(f"layer degree {k} {dtype_name} G={G} in={n_in} out={n_out}")
    y = kb.layer_forward(to_dev(x, dt), to_dev(C, dt), to_dev(Wb, dt), G, spline_order=k)
    torch.cuda.synchronize()
    ref = oracle.layer(x, C, Wb, G, k=k)
    tol = F32_LAYER_TOL
    if dtype_name == "bf16":
        ref, tol = oracle.round_bf16(ref), BF16_LAYER_TOL
    assert normwise(to_host64(y), ref) <= tol


@pytest.mark.parametrize("dtype_name", ["f32", "bf16"])
@pytest.mark.parametrize("G,lo,hi", [(10, -math.pi, math.pi), (200, 0.0, 3.0), (10, 100.0, 103.0)])
def test_layer_non_dyadic_grids(G, lo, hi, dtype_name):
    """The fused layer on grids whose 1 / h is not exact: the bf16 G = 10
    cases run the structured-sparse shapes, the rest the dense ones."""
    lo32, hi32 = float(np.float32(lo)), float(np.float32(hi))
    B, n_in, n_out = 400, 13, 256
    x, C, Wb = _layer_case(B, n_in, n_out, G, 3, lo32, hi32, dtype_name, seed=G)
    dt = torch.float32 if dtype_name == "f32" else torch.bfloat16
    say(f"layer grid {dtype_name} G={G} [{lo32}, {hi32}]")
    y = kb.layer_forward(to_dev(x, dt), to_dev(C, dt), to_dev(Wb, dt), G, lo32, hi32)
    torch.cuda.synchronize()
    ref = oracle.layer(x, C, Wb, G, lo32, hi32)
    tol = F32_LAYER_TOL
    if dtype_name == "bf16":
        ref, tol = oracle.round_bf16(ref), BF16_LAYER_TOL
    assert normwise(to_host64(y), ref) <= tol


@pytest.mark.parametrize("dtype_name", ["f32", "bf16"])
def test_backward_non_dyadic_grid(dtype_name):
    G, lo, hi = 10, float(np.float32(-math.pi)), float(np.float32(math.pi))
    B, n_in, n_out = 300, 9, 40
    x, C, Wb = _layer_case(B, n_in, n_out, G, 3, lo, hi, dtype_name, seed=3)
    dy = np.random.default_rng(4).normal(0, 1, (B, n_out)).astype(np.float32)
    if dtype_name == "bf16":
        dy = wl.round_to_bf16_f32(dy)
    dt = torch.float32 if dtype_name == "f32" else torch.bfloat16
    say(f"backward grid {dtype_name}")
    outs = kb.layer_backward(to_dev(x, dt), to_dev(C, dt), to_dev(Wb, dt), to_dev(dy, dt), G,
                             lo, hi)
    torch.cuda.synchronize()
    refs = oracle.layer_backward(x, C, Wb, dy, G, lo, hi)
    tol = F32_LAYER_TOL if dtype_name == "f32" else BF16_LAYER_TOL
    for got, ref in zip(outs, refs):
        if dtype_name == "bf16":
            ref = oracle.round_bf16(ref)
        assert normwise(to_host64(got), ref) <= tol
