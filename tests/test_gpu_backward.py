"""GPU parity of kan_layer_backward (dx on the matrix cores with the clamped
derivative contracted in the epilogue, or for narrow layers at large batches
on the vector ALUs over the window's columns; dC and dWb on the matrix cores with
the basis regenerated in registers, batch splits summed in a fixed order)
against the float64 oracle's layer_backward, through the C ABI.  Tolerances,
normwise max|g - ref| / max|ref| per gradient: 1e-5 in fp32, 2e-2 in bf16
(reference on the same bf16-rounded tensors, rounded to bf16)."""
import numpy as np
import pytest

import oracle
from paper_2609_01956_amd import binding as kb
from paper_2609_01956_amd import workloads as wl
from gpu_common import (BF16_LAYER_TOL, F32_LAYER_TOL, device, normwise, say, to_dev, to_host64,
                        torch)

pytestmark = pytest.mark.gpu


def _case(B, n_in, n_out, G, seed, dtype_name, off=0.1):
    x, C, Wb = wl.make_layer(wl.LayerShape(B, n_in, n_out, G, off_grid_frac=off), seed)
    dy = np.random.default_rng(seed + 1).normal(0, 1, (B, n_out)).astype(np.float32)
    if dtype_name == "bf16":
        x, C, Wb, dy = (wl.round_to_bf16_f32(a) for a in (x, C, Wb, dy))
    return x, C, Wb, dy


def _run(x, C, Wb, dy, G, dtype_name, need_dx=True, need_dw=True):
    dt = torch.float32 if dtype_name == "f32" else torch.bfloat16
    outs = kb.layer_backward(to_dev(x, dt), to_dev(C, dt), to_dev(Wb, dt), to_dev(dy, dt), G,
                             need_dx=need_dx, need_dw=need_dw)
    torch.cuda.synchronize()
    return [None if o is None else to_host64(o) for o in outs]


def _check(got, ref, dtype_name, what):
    tol = F32_LAYER_TOL if dtype_name == "f32" else BF16_LAYER_TOL
    if dtype_name == "bf16":
        ref = oracle.round_bf16(ref)
    e = normwise(got, ref)
    assert e <= tol, (what, e)


BWD_SHAPES = [
    # (B, in, out, G): 16 columns per feature (G <= 12) with an odd feature
    # count and a ragged batch; 32 (G = 13..28) and more (G = 50, 200: the
    # two lane halves of a feature added); outputs of one fragment, two, four,
    # eight and beyond one 256-output tile (several dx output chunks)
    (300, 9, 10, 5),
    (257, 17, 64, 10),
    (1000, 12, 100, 12),
    (513, 7, 256, 10),
    (129, 5, 40, 20),
    (97, 3, 33, 50),
    (64, 4, 20, 200),
    (200, 6, 300, 8),
    (33, 1, 1, 10),
]


@pytest.mark.parametrize("dtype_name", ["f32", "bf16"])
@pytest.mark.parametrize("B,n_in,n_out,G", BWD_SHAPES)
def test_backward_matches_oracle(B, n_in, n_out, G, dtype_name):
    x, C, Wb, dy = _case(B, n_in, n_out, G, seed=B + n_in + G, dtype_name=dtype_name)
    say(f"backward {dtype_name} B={B} in={n_in} out={n_out} G={G}")
    dx, dC, dW = _run(x, C, Wb, dy, G, dtype_name)
    rx, rC, rW = oracle.layer_backward(x, C, Wb, dy, G)
    _check(dx, rx, dtype_name, "dx")
    _check(dC, rC, dtype_name, "dC")
    _check(dW, rW, dtype_name, "dWb")


# Layers of at most 16 outputs from 16384 rows on take dx on the vector-ALU
# kernel (an fp32 weight table in the workspace, one batch row per lane, 8
# features staged at a time): outputs 1, 3, 7, 10 and 16, grids 1 .. 26, odd
# feature counts and partial feature chunks, batches that end inside a 64-row
# workgroup.
NARROW_BWD = [
    (16384, 9, 10, 10),
    (16400, 17, 1, 5),
    (16411, 33, 16, 10),
    (16384, 5, 3, 26),
    (16390, 3, 7, 1),
    (16384, 6, 4, 58),   # the largest table: 64 columns x 4 floats per feature
    (65536, 37, 10, 10),  # two feature groups of 3 and 2 chunks, the last chunk ragged
]


@pytest.mark.parametrize("dtype_name", ["f32", "bf16"])
@pytest.mark.parametrize("B,n_in,n_out,G", NARROW_BWD)
def test_backward_narrow_dx(B, n_in, n_out, G, dtype_name):
    x, C, Wb, dy = _case(B, n_in, n_out, G, seed=B + n_in + n_out, dtype_name=dtype_name)
    say(f"backward narrow dx {dtype_name} B={B} in={n_in} out={n_out} G={G}")
    dx, dC, dW = _run(x, C, Wb, dy, G, dtype_name)
    rx, rC, rW = oracle.layer_backward(x, C, Wb, dy, G)
    _check(dx, rx, dtype_name, "dx")
    _check(dC, rC, dtype_name, "dC")
    _check(dW, rW, dtype_name, "dWb")


def test_backward_narrow_dx_nan_and_determinism():
    """A NaN input on the narrow dx kernel: NaN at its own dx entry only (the
    SiLU derivative carries it), every other entry as the oracle's; repeats
    are bit-identical."""
    B, n_in, n_out, G = 16500, 11, 10, 10
    x, C, Wb, dy = _case(B, n_in, n_out, G, seed=8, dtype_name="f32")
    x[16450, 4] = np.nan
    say("backward narrow dx nan / determinism")
    dx, _, _ = _run(x, C, Wb, dy, G, "f32", need_dw=False)
    dx2, _, _ = _run(x, C, Wb, dy, G, "f32", need_dw=False)
    np.testing.assert_array_equal(dx, dx2)
    assert np.isnan(dx[16450, 4])
    ok = np.ones_like(dx, bool)
    ok[16450, 4] = False
    assert not np.any(np.isnan(dx[ok]))
    xr = x.copy()
    xr[16450, 4] = 0.0
    rx, _, _ = oracle.layer_backward(xr, C, Wb, dy, G)
    assert normwise(dx[ok], rx[ok]) <= F32_LAYER_TOL


@pytest.mark.parametrize("dtype_name", ["f32", "bf16"])
def test_backward_partial_outputs_and_determinism(dtype_name):
    """dx alone, the weight gradients alone, and bit-identical repeats."""
    B, n_in, n_out, G = 700, 11, 70, 10
    x, C, Wb, dy = _case(B, n_in, n_out, G, seed=77, dtype_name=dtype_name)
    say(f"backward partial outputs {dtype_name}")
    dx, dC, dW = _run(x, C, Wb, dy, G, dtype_name, need_dw=False)
    assert dC is None and dW is None
    dx2, _, _ = _run(x, C, Wb, dy, G, dtype_name)
    np.testing.assert_array_equal(dx, dx2)
    n1, dC1, dW1 = _run(x, C, Wb, dy, G, dtype_name, need_dx=False)
    _, dC2, dW2 = _run(x, C, Wb, dy, G, dtype_name)
    assert n1 is None
    np.testing.assert_array_equal(dC1, dC2)
    np.testing.assert_array_equal(dW1, dW2)
    rx, rC, rW = oracle.layer_backward(x, C, Wb, dy, G)
    _check(dx, rx, dtype_name, "dx")
    _check(dC1, rC, dtype_name, "dC")


def test_backward_nan_input_and_empty_batch():
    B, n_in, n_out, G = 100, 6, 20, 10
    x, C, Wb, dy = _case(B, n_in, n_out, G, seed=3, dtype_name="f32")
    x[7, 2] = np.nan
    say("backward nan / empty")
    dx, dC, dW = _run(x, C, Wb, dy, G, "f32")
    assert np.isnan(dx[7, 2]) and np.all(np.isnan(dC[:, 2, :])) and np.all(np.isnan(dW[:, 2]))
    ok = np.ones_like(dx, bool)
    ok[7, 2] = False
    xr = x.copy()
    xr[7, 2] = 0.0
    rx, _, _ = oracle.layer_backward(xr, C, Wb, dy, G)
    assert normwise(dx[ok], rx[ok]) <= F32_LAYER_TOL
    # an empty batch: zero weight gradients
    dt = torch.float32
    e = kb.layer_backward(torch.empty(0, n_in, device=device()), to_dev(C, dt), to_dev(Wb, dt),
                          torch.empty(0, n_out, device=device()), G)
    torch.cuda.synchronize()
    assert e[0].shape == (0, n_in)
    assert torch.count_nonzero(e[1]) == 0 and torch.count_nonzero(e[2]) == 0


@pytest.mark.parametrize("dtype_name", ["f32", "bf16"])
def test_backward_c5_first_layer_sampled(dtype_name):
    """The 784 -> 256 layer of the MLP workload at batch 8192: dx on sampled
    rows, dC / dWb on sampled (output, feature) pairs, each computed by the
    oracle from the full batch's rows it needs."""
    W = wl.make_workload("c5_mlp_784_256_256_10_g10", batch=8192)
    G = W["G"]
    x = W["x"]
    C, Wb = W["layers"][0]
    dy = np.random.default_rng(5).normal(0, 1, (x.shape[0], C.shape[0])).astype(np.float32)
    if dtype_name == "bf16":
        x, C, Wb, dy = (wl.round_to_bf16_f32(a) for a in (x, C, Wb, dy))
    say(f"backward c5 layer 1 {dtype_name}")
    dx, dC, dW = _run(x, C, Wb, dy, G, dtype_name)
    rows = np.random.default_rng(1).choice(x.shape[0], 64, replace=False)
    rx, _, _ = oracle.layer_backward(x[rows], C, Wb, dy[rows], G)
    _check(dx[rows], rx, dtype_name, "dx")
    feats = np.random.default_rng(2).choice(C.shape[1], 6, replace=False)
    _, rC, rW = oracle.layer_backward(x[:, feats], C[:, feats], Wb[:, feats], dy, G)
    _check(dC[:, feats], rC, dtype_name, "dC")
    _check(dW[:, feats], rW, dtype_name, "dWb")
