"""GPU parity of the span-sparse layer forward (eq. kan_forward on the k + 1
nonzero bases per input and the SiLU term) against the float64 oracle through
the C ABI, at the layer tolerances of the method: normwise <= 1e-5 (fp32) and
<= 2e-2 (bf16, reference rounded to bf16 like the output).  The shapes span
several output tiles, ragged row blocks, feature splits over workgroups (with
the fixed-order reduce) and one split only, every degree the library takes,
and the widest grid one feature's weight tile fits in LDS."""
import math

import numpy as np
import pytest

import oracle
from paper_2609_01956_amd import binding as kb
from paper_2609_01956_amd import workloads as wl
from gpu_common import (BF16_LAYER_TOL, F32_LAYER_TOL, device, normwise, say, to_dev, to_host64,
                        torch)

pytestmark = pytest.mark.gpu


def _dt(name):
    return torch.float32 if name == "f32" else torch.bfloat16


def _case(B, n_in, n_out, G, k, lo, hi, dtype_name, seed, off=2.0):
    rng = np.random.default_rng(seed)
    h = (hi - lo) / G
    x = rng.uniform(lo - off * h, hi + off * h, (B, n_in)).astype(np.float32)
    _, C, Wb = wl.make_layer(wl.LayerShape(B, n_in, n_out, G), seed, k=k)
    if dtype_name == "bf16":
        x, C, Wb = (wl.round_to_bf16_f32(a) for a in (x, C, Wb))
    return x, C, Wb


def _check(y, x, C, Wb, G, k, lo, hi, dtype_name):
    ref = oracle.layer(x, C, Wb, G, lo, hi, k=k)
    tol = F32_LAYER_TOL
    if dtype_name == "bf16":
        ref, tol = oracle.round_bf16(ref), BF16_LAYER_TOL
    err = normwise(to_host64(y), ref)
    assert err <= tol, err


# (B, in, out, G): 64-output tiles in two groups, 45 outputs in one padded
# tile, 10 outputs at 16 per thread, 300 outputs over five tiles, 17 outputs
# at 32 per thread, and B = 1
SHAPES = [(777, 37, 128, 50), (300, 13, 45, 100), (257, 40, 10, 200), (33, 7, 300, 5),
          (100, 5, 17, 20), (1, 3, 64, 10)]


@pytest.mark.parametrize("dtype_name", ["f32", "bf16"])
@pytest.mark.parametrize("B,n_in,n_out,G", SHAPES)
def test_span_layer_cubic(B, n_in, n_out, G, dtype_name):
    x, C, Wb = _case(B, n_in, n_out, G, 3, -1.0, 1.0, dtype_name, seed=B + G)
    dt = _dt(dtype_name)
    say(f"span {dtype_name} B={B} in={n_in} out={n_out} G={G}")
    y = kb.layer_forward_span(to_dev(x, dt), to_dev(C, dt), to_dev(Wb, dt), G)
    torch.cuda.synchronize()
    _check(y, x, C, Wb, G, 3, -1.0, 1.0, dtype_name)


@pytest.mark.parametrize("dtype_name", ["f32", "bf16"])
@pytest.mark.parametrize("k,G", [(1, 100), (2, 37), (5, 64), (7, 9)])
def test_span_layer_other_degrees(k, G, dtype_name):
    B, n_in, n_out = 260, 11, 70
    x, C, Wb = _case(B, n_in, n_out, G, k, -1.0, 1.0, dtype_name, seed=100 + k)
    dt = _dt(dtype_name)
    say(f"span degree {k} {dtype_name} G={G}")
    y = kb.layer_forward_span(to_dev(x, dt), to_dev(C, dt), to_dev(Wb, dt), G, spline_order=k)
    torch.cuda.synchronize()
    _check(y, x, C, Wb, G, k, -1.0, 1.0, dtype_name)


@pytest.mark.parametrize("G,lo,hi", [(200, 0.0, 3.0), (10, -math.pi, math.pi),
                                     (10, 100.0, 103.0)])
def test_span_layer_non_dyadic_grids(G, lo, hi):
    lo32, hi32 = float(np.float32(lo)), float(np.float32(hi))
    x, C, Wb = _case(400, 13, 96, G, 3, lo32, hi32, "f32", seed=G)
    say(f"span grid G={G} [{lo32}, {hi32}]")
    y = kb.layer_forward_span(to_dev(x, torch.float32), to_dev(C, torch.float32),
                              to_dev(Wb, torch.float32), G, lo32, hi32)
    torch.cuda.synchronize()
    _check(y, x, C, Wb, G, 3, lo32, hi32, "f32")


def test_span_layer_widest_grid():
    """G + k + 1 = 512 columns: the widest weight tile (16 outputs) in LDS;
    inputs reach past both grid ends (the clamp)."""
    G = 508
    x, C, Wb = _case(130, 3, 40, G, 3, -1.0, 1.0, "f32", seed=7, off=50.0)
    say("span widest grid G=508")
    y = kb.layer_forward_span(to_dev(x, torch.float32), to_dev(C, torch.float32),
                              to_dev(Wb, torch.float32), G)
    torch.cuda.synchronize()
    _check(y, x, C, Wb, G, 3, -1.0, 1.0, "f32")


def test_span_matches_dense_layer():
    """The span-sparse and dense layers agree (both fp32): they differ only in
    the exact zeros the span form leaves out and the order of the sums."""
    G, B, n_in, n_out = 100, 1000, 64, 128
    x, C, Wb = _case(B, n_in, n_out, G, 3, -1.0, 1.0, "f32", seed=5)
    xs, Cs, Ws = (to_dev(a, torch.float32) for a in (x, C, Wb))
    say("span vs dense G=100")
    ys = kb.layer_forward_span(xs, Cs, Ws, G)
    yd = kb.layer_forward(xs, Cs, Ws, G)
    torch.cuda.synchronize()
    assert normwise(to_host64(ys), to_host64(yd)) <= F32_LAYER_TOL


@pytest.mark.parametrize("dtype_name", ["f32", "bf16"])
def test_span_nan_row(dtype_name):
    """A NaN input makes its row NaN in every output (as the dense layer and
    the oracle); the other rows are unaffected."""
    G, B, n_in, n_out = 50, 300, 9, 40
    x, C, Wb = _case(B, n_in, n_out, G, 3, -1.0, 1.0, dtype_name, seed=11)
    x[17, 4] = np.nan
    dt = _dt(dtype_name)
    say(f"span NaN row {dtype_name}")
    y = to_host64(kb.layer_forward_span(to_dev(x, dt), to_dev(C, dt), to_dev(Wb, dt), G))
    assert np.all(np.isnan(y[17]))
    keep = np.ones(B, bool)
    keep[17] = False
    assert np.all(np.isfinite(y[keep]))
    ref = oracle.layer(x[keep], C, Wb, G)
    tol = F32_LAYER_TOL
    if dtype_name == "bf16":
        ref, tol = oracle.round_bf16(ref), BF16_LAYER_TOL
    assert normwise(y[keep], ref) <= tol


def test_span_empty_batch():
    G = 50
    _, C, Wb = _case(1, 8, 16, G, 3, -1.0, 1.0, "f32", seed=1)
    x = np.zeros((0, 8), np.float32)
    y = kb.layer_forward_span(to_dev(x, torch.float32), to_dev(C, torch.float32),
                              to_dev(Wb, torch.float32), G)
    torch.cuda.synchronize()
    assert tuple(y.shape) == (0, 16)


@pytest.mark.parametrize("dtype_name", ["f32", "bf16"])
@pytest.mark.parametrize("G", [50, 200])
def test_span_grid_sweep_full_size(G, dtype_name):
    """The grid-sweep layer (batch 8192, 128 -> 128) at full size: 256
    sampled rows against the oracle, and every output finite."""
    w = kb_workload(G)
    x, (C, Wb) = w["x"], w["layers"][0]
    if dtype_name == "bf16":
        x, C, Wb = (wl.round_to_bf16_f32(a) for a in (x, C, Wb))
    dt = _dt(dtype_name)
    say(f"span grid sweep G={G} {dtype_name}")
    y = to_host64(kb.layer_forward_span(to_dev(x, dt), to_dev(C, dt), to_dev(Wb, dt), G))
    assert np.all(np.isfinite(y))
    rows = np.random.default_rng(G).choice(x.shape[0], 256, replace=False)
    ref = oracle.layer(x[rows], C, Wb, G)
    tol = F32_LAYER_TOL
    if dtype_name == "bf16":
        ref, tol = oracle.round_bf16(ref), BF16_LAYER_TOL
    assert normwise(y[rows], ref) <= tol


def kb_workload(G):
    return wl.make_workload(f"c4_layer_128x128_g{G}")


def test_span_reuses_workspace():
    """Two calls on one caller workspace, the second smaller: each matches the
    oracle (the partial-sum area is fully rewritten by every call)."""
    G = 100
    x1, C1, W1 = _case(600, 30, 64, G, 3, -1.0, 1.0, "f32", seed=21)
    x2, C2, W2 = _case(90, 30, 64, G, 3, -1.0, 1.0, "f32", seed=22)
    g = kb.make_grid(G)
    st, nbytes = kb.kan_layer_forward_span_workspace_bytes(g, kb.KAN_F32, 600, 30, 64)
    assert st == 0
    ws = torch.empty(nbytes, dtype=torch.uint8, device=device())
    say("span workspace reuse")
    ya = kb.layer_forward_span(to_dev(x1, torch.float32), to_dev(C1, torch.float32),
                               to_dev(W1, torch.float32), G, workspace=ws)
    yb = kb.layer_forward_span(to_dev(x2, torch.float32), to_dev(C2, torch.float32),
                               to_dev(W2, torch.float32), G, workspace=ws)
    torch.cuda.synchronize()
    _check(ya, x1, C1, W1, G, 3, -1.0, 1.0, "f32")
    _check(yb, x2, C2, W2, G, 3, -1.0, 1.0, "f32")
