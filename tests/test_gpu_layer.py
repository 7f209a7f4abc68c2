"""GPU parity of kan_layer_forward (fused basis + MFMA contraction + SiLU
branch) against the float64 oracle, through the C ABI.  Tolerances, normwise
max|y - ref| / max|ref|: 1e-5 in fp32, 2e-2 in bf16 (reference computed on the
same bf16-rounded tensors)."""
import numpy as np
import pytest

import oracle
from paper_2609_01956_amd import binding as kb
from paper_2609_01956_amd import workloads as wl
from gpu_common import (BF16_LAYER_TOL, F32_LAYER_TOL, device, normwise, say, to_dev,
                        to_host64, torch)

pytestmark = pytest.mark.gpu

DT = {"f32": None, "bf16": None}


def _dtype(name):
    return torch.float32 if name == "f32" else torch.bfloat16


def _tol(name):
    return F32_LAYER_TOL if name == "f32" else BF16_LAYER_TOL


def _inputs(B, n_in, n_out, G, seed, off=0.0, dtype_name="f32"):
    shape = wl.LayerShape(B, n_in, n_out, G, off_grid_frac=off)
    x, C, Wb = wl.make_layer(shape, seed)
    if dtype_name == "bf16":
        x, C, Wb = wl.round_to_bf16_f32(x), wl.round_to_bf16_f32(C), wl.round_to_bf16_f32(Wb)
    return x, C, Wb


def _gpu_layer(x, C, Wb, G, dtype_name, shape=None):
    dt = _dtype(dtype_name)
    y = kb.layer_forward(to_dev(x, dt), to_dev(C, dt), to_dev(Wb, dt), G, shape=shape)
    torch.cuda.synchronize()
    return to_host64(y)


SHAPES = [
    (1024, 2, 5, 5),      # the tiny 2 -> 5 layer, full size
    (4096, 64, 64, 5),    # the 64 -> 64 layer, full size
    (1000, 3, 37, 7),     # ragged everything, odd feature count
    (257, 33, 70, 1),     # smallest grid
    (130, 17, 300, 13),   # more than one column tile
    (64, 5, 3, 200),      # the largest swept grid, many K chunks
    (96, 2, 1, 50),       # single output
    (33, 1, 256, 10),     # single input feature
]


@pytest.mark.parametrize("dtype_name", ["f32", "bf16"])
@pytest.mark.parametrize("B,n_in,n_out,G", SHAPES)
def test_layer_matches_oracle(B, n_in, n_out, G, dtype_name):
    x, C, Wb = _inputs(B, n_in, n_out, G, seed=B + n_in + G, off=0.1, dtype_name=dtype_name)
    say(f"layer {dtype_name} B={B} in={n_in} out={n_out} G={G}")
    y = _gpu_layer(x, C, Wb, G, dtype_name)
    ref = oracle.layer(x, C, Wb, G)
    if dtype_name == "bf16":
        ref = oracle.round_bf16(ref)
    assert normwise(y, ref) <= _tol(dtype_name), normwise(y, ref)


# (rows tiles per wave, waves splitting K[, waves per workgroup[, column
# slices per tile]]) of the fused kernel; K splits need rf * nf <= 4 (nf =
# 32-column fragments a workgroup computes); eight-wave workgroups take one
# row tile per wave and no K split; column slices take rf = 1, four waves.
CFGS = ["1,1", "2,1", "1,2", "1,4", "2,2", "2,4", "1,1,8", "1,1,4,2", "1,2,4,2", "1,4,4,2"]


# bf16 with two blocks per feature (5 <= G <= 12) runs the sparse MFMA, whose
# K splits take tiles of one or two fragments (NARROW_CFGS below); G = 20 keeps
# the dense bf16 kernel under every shape.
SPARSE_CFGS = ["1,1", "2,1", "1,1,8", "1,1,4,2"]


@pytest.mark.parametrize("dtype_name,G", [("f32", 10), ("bf16", 20)] +
                         [pytest.param("bf16", 10, id="bf16-sparse")])
@pytest.mark.parametrize("cfg", CFGS)
def test_layer_every_workgroup_shape(cfg, dtype_name, G):
    # out = 45 -> two 32-column fragments per tile, so every shape is valid;
    # 9 features (odd) and 300 rows (ragged) exercise the padding paths.
    if dtype_name == "bf16" and G == 10 and cfg not in SPARSE_CFGS:
        pytest.skip("not a shape of the sparse MFMA")
    B, n_in, n_out = 300, 9, 45
    x, C, Wb = _inputs(B, n_in, n_out, G, seed=3, off=0.1, dtype_name=dtype_name)
    ref = oracle.layer(x, C, Wb, G)
    if dtype_name == "bf16":
        ref = oracle.round_bf16(ref)
    say(f"layer cfg={cfg} {dtype_name}")
    y = _gpu_layer(x, C, Wb, G, dtype_name, shape=cfg)
    assert normwise(y, ref) <= _tol(dtype_name)


WIDE = [
    # (dtype, B, in, out, G, cfg): the widest column tiles (bf16 256, fp32 128)
    ("bf16", 600, 20, 256, 20, "2,1"),
    ("bf16", 600, 20, 256, 20, "1,1"),
    ("bf16", 333, 7, 200, 50, "2,1"),
    ("bf16", 97, 3, 130, 200, "1,1"),
    ("bf16", 600, 20, 256, 10, "1,1,8"),
    ("bf16", 300, 5, 100, 50, "1,1,8"),
    # two blocks per feature (G = 7, 10; the sparse MFMA) with an odd number
    # of chunks (a padding chunk in the last unrolled pair), an odd feature
    # count and a ragged batch; and the 64-row one-wave shape of the dense
    # kernel (G = 20)
    ("bf16", 300, 18, 256, 10, "1,1,8"),
    ("bf16", 257, 17, 256, 7, "1,1,8"),
    ("bf16", 300, 18, 256, 10, "2,1,8"),
    ("bf16", 257, 17, 200, 7, "2,1,8"),
    ("bf16", 33, 1, 256, 12, "2,1,8"),
    ("bf16", 129, 5, 256, 5, "2,1,8"),   # three chunks: fewer than the unroll
    ("bf16", 260, 40, 256, 8, "2,1,8"),
    ("bf16", 257, 17, 256, 20, "2,1"),
    ("f32", 600, 20, 256, 10, "1,1"),
    ("f32", 600, 20, 256, 10, "1,4"),
    ("f32", 333, 7, 128, 50, "2,1"),
    ("f32", 97, 3, 100, 200, "1,2"),
    ("f32", 600, 20, 256, 10, "1,1,8"),
    # column slices of the widest tiles
    ("bf16", 600, 20, 256, 10, "1,1,4,2"),
    ("bf16", 333, 7, 200, 50, "1,2,4,2"),
    ("bf16", 600, 20, 256, 10, "1,1,4,4"),
    ("bf16", 97, 3, 130, 200, "1,2,4,4"),
    ("bf16", 300, 5, 100, 50, "1,4,4,4"),
    ("f32", 600, 20, 256, 10, "1,1,4,2"),
    ("f32", 333, 7, 128, 50, "1,4,4,2"),
    ("f32", 97, 3, 100, 200, "1,2,4,4"),
    ("f32", 600, 20, 256, 10, "1,4,4,4"),
]


@pytest.mark.parametrize("dtype_name,B,n_in,n_out,G,cfg", WIDE)
def test_layer_wide_tiles(dtype_name, B, n_in, n_out, G, cfg):
    x, C, Wb = _inputs(B, n_in, n_out, G, seed=B + G, off=0.1, dtype_name=dtype_name)
    ref = oracle.layer(x, C, Wb, G)
    if dtype_name == "bf16":
        ref = oracle.round_bf16(ref)
    say(f"layer wide {dtype_name} B={B} in={n_in} out={n_out} G={G} cfg={cfg}")
    y = _gpu_layer(x, C, Wb, G, dtype_name, shape=cfg)
    assert normwise(y, ref) <= _tol(dtype_name)


SPARSE_SHAPES = [
    # (B, in, out, G): two blocks per feature at G = 5, 8, 11, 12 over one,
    # two, four and eight 32-column fragments per tile, ragged batches and
    # odd feature counts
    (300, 9, 10, 5),
    (257, 17, 64, 8),
    (129, 4, 100, 11),
    (500, 33, 256, 12),
    (1000, 7, 256, 10),
]


SPARSE_256_CFGS = ["1,1,8", "2,1", "2,1,8", "1,1,4,2", "1,1,4,4"]


@pytest.mark.parametrize("cfg", SPARSE_256_CFGS)
def test_layer_bf16_sparse_mfma_256_column_shapes(cfg):
    """The shapes the sparse MFMA takes on 256-column tiles: eight 32-row
    waves, four 64-row waves (one per SIMD), eight 64-row waves on column
    halves passing each other the A of one row tile, and column slices."""
    B, n_in, n_out, G = 700, 13, 256, 10
    x, C, Wb = _inputs(B, n_in, n_out, G, seed=5, off=0.2, dtype_name="bf16")
    ref = oracle.round_bf16(oracle.layer(x, C, Wb, G))
    say(f"layer bf16 sparse 256 columns cfg={cfg}")
    y = _gpu_layer(x, C, Wb, G, "bf16", shape=cfg)
    assert normwise(y, ref) <= BF16_LAYER_TOL, normwise(y, ref)


# The sparse MFMA with a K split (tiles of one or two 32-column fragments,
# wave slices taking whole feature pairs, partial sums added through LDS):
# slices of two and four over four- and eight-wave workgroups.
NARROW_CFGS = ["1,2", "1,4", "1,2,8", "1,4,8"]
NARROW_SHAPES = [
    # (B, in, out, G): one and two fragments, odd feature counts (a phantom
    # feature), ragged batches, fewer feature pairs than K slices, one feature
    (300, 9, 10, 10),
    (257, 17, 64, 7),
    (1000, 256, 10, 10),
    (129, 3, 33, 12),
    (65, 1, 5, 5),
]


@pytest.mark.parametrize("cfg", NARROW_CFGS)
@pytest.mark.parametrize("B,n_in,n_out,G", NARROW_SHAPES)
def test_layer_bf16_sparse_k_split(B, n_in, n_out, G, cfg):
    x, C, Wb = _inputs(B, n_in, n_out, G, seed=B + n_in + G, off=0.2, dtype_name="bf16")
    ref = oracle.round_bf16(oracle.layer(x, C, Wb, G))
    say(f"layer bf16 sparse K split B={B} in={n_in} out={n_out} G={G} cfg={cfg}")
    y = _gpu_layer(x, C, Wb, G, "bf16", shape=cfg)
    assert normwise(y, ref) <= BF16_LAYER_TOL, normwise(y, ref)


STAGED_CASES = [(256, 0), (250, 0), (256, 1), (136, 3)]


@pytest.mark.parametrize("n_out,offset", STAGED_CASES)
def test_layer_shared_a_staged_epilogue(n_out, offset):
    """The shared-A shape stores y through LDS: 16-byte row segments where
    out % 8 == 0 and y is 16-byte aligned, else element stores (out = 250,
    136, or y one or three elements past an aligned address); a ragged batch
    ends inside the 256-row workgroup; nothing is written around y."""
    B, n_in, G = 300, 13, 10
    x, C, Wb = _inputs(B, n_in, n_out, G, seed=n_out + offset, off=0.1, dtype_name="bf16")
    say(f"layer shared-A epilogue out={n_out} offset={offset}")
    dt = torch.bfloat16
    p = kb.pack_layer(to_dev(C, dt), to_dev(Wb, dt), G)
    buf = torch.full((B * n_out + 64,), 3.0, dtype=dt, device=device())
    out = buf[offset:offset + B * n_out].view(B, n_out)
    kb.layer_forward_packed(to_dev(x, dt), p, out=out, shape="2,1,8")
    torch.cuda.synchronize()
    ref = oracle.round_bf16(oracle.layer(x, C, Wb, G))
    assert normwise(to_host64(out), ref) <= BF16_LAYER_TOL
    b = to_host64(buf)
    assert np.all(b[:offset] == 3.0) and np.all(b[offset + B * n_out:] == 3.0)


@pytest.mark.parametrize("B,n_in,n_out,G", SPARSE_SHAPES)
def test_layer_bf16_sparse_mfma(B, n_in, n_out, G):
    x, C, Wb = _inputs(B, n_in, n_out, G, seed=B + G, off=0.2, dtype_name="bf16")
    ref = oracle.round_bf16(oracle.layer(x, C, Wb, G))
    say(f"layer bf16 sparse B={B} in={n_in} out={n_out} G={G}")
    y = _gpu_layer(x, C, Wb, G, "bf16")
    assert normwise(y, ref) <= BF16_LAYER_TOL, normwise(y, ref)


X_WORD_CFGS = [None, "1,1", "1,1,4,2"]


@pytest.mark.parametrize("case", ["aligned", "odd_total", "x_at_odd_element"])
@pytest.mark.parametrize("cfg", X_WORD_CFGS)
def test_layer_bf16_x_word_reads_and_their_fallbacks(case, cfg):
    """With two blocks per feature (G = 10) bf16 x is read as the aligned
    32-bit word holding each element when x is 4-byte aligned and batch * in is
    even (the word then never leaves the tensor); an odd element count, or an x
    that starts at an odd element, takes 16-bit reads.  Odd feature counts give
    rows of both parities.  Every case matches the oracle."""
    B, n_in, n_out, G = {"aligned": (300, 9, 45, 10), "odd_total": (301, 9, 45, 10),
                         "x_at_odd_element": (300, 9, 45, 10)}[case]
    x, C, Wb = _inputs(B, n_in, n_out, G, seed=11, off=0.1, dtype_name="bf16")
    ref = oracle.round_bf16(oracle.layer(x, C, Wb, G))
    dt = torch.bfloat16
    if case == "x_at_odd_element":
        buf = torch.zeros(B * n_in + 1, dtype=dt, device=device())
        xd = buf[1:].view(B, n_in)
        xd.copy_(to_dev(x, dt))
        assert xd.data_ptr() % 4 == 2
    else:
        xd = to_dev(x, dt)
    say(f"layer bf16 x reads {case} cfg={cfg}")
    y = kb.layer_forward(xd, to_dev(C, dt), to_dev(Wb, dt), G, shape=cfg)
    torch.cuda.synchronize()
    assert normwise(to_host64(y), ref) <= BF16_LAYER_TOL


@pytest.mark.parametrize("dtype_name", ["f32", "bf16"])
def test_c_layer_forward_workspace_entry_point(dtype_name):
    """kan_layer_forward (packs into the caller's workspace, then the packed
    forward) called through the raw C entry point gives the same bits as pack +
    forward_packed, and a second call reusing the workspace for a smaller
    layer is right too."""
    code = kb.KAN_F32 if dtype_name == "f32" else kb.KAN_BF16
    dt = _dtype(dtype_name)
    stream = int(torch.cuda.current_stream().cuda_stream)
    ws = None
    for B, n_in, n_out, G in [(513, 31, 70, 10), (77, 9, 20, 5)]:
        x, C, Wb = _inputs(B, n_in, n_out, G, seed=9, off=0.1, dtype_name=dtype_name)
        xt, Ct, Wt = to_dev(x, dt), to_dev(C, dt), to_dev(Wb, dt)
        y = torch.empty((B, n_out), dtype=dt, device=device())
        st, need = kb.kan_layer_forward_workspace_bytes(kb.make_grid(G), code, B, n_in, n_out)
        assert st == kb.KAN_OK and need > 0
        if ws is None:
            ws = torch.empty(need, dtype=torch.uint8, device=device())
        assert ws.numel() >= need
        say(f"layer C entry point {dtype_name} B={B} in={n_in} out={n_out} G={G}")
        st = kb.kan_layer_forward(kb.make_grid(G), code, B, n_in, n_out, xt.data_ptr(),
                                  Ct.data_ptr(), Wt.data_ptr(), ws.data_ptr(), ws.numel(),
                                  y.data_ptr(), stream)
        assert st == kb.KAN_OK
        y2 = kb.layer_forward(xt, Ct, Wt, G)
        torch.cuda.synchronize()
        assert torch.equal(y, y2)
        ref = oracle.layer(x, C, Wb, G)
        if dtype_name == "bf16":
            ref = oracle.round_bf16(ref)
        assert normwise(to_host64(y), ref) <= _tol(dtype_name)


def test_packed_weights_reused_across_batches():
    B, n_in, n_out, G = 700, 12, 33, 10
    x, C, Wb = _inputs(B, n_in, n_out, G, seed=11, off=0.1)
    say("layer packed reuse")
    p = kb.pack_layer(to_dev(C, torch.float32), to_dev(Wb, torch.float32), G)
    ya = kb.layer_forward_packed(to_dev(x, torch.float32), p)
    yb = kb.layer_forward_packed(to_dev(x[:37], torch.float32), p)
    torch.cuda.synchronize()
    ref = oracle.layer(x, C, Wb, G)
    assert normwise(to_host64(ya), ref) <= F32_LAYER_TOL
    assert normwise(to_host64(yb), ref[:37]) <= F32_LAYER_TOL


def test_layer_special_cases_f32():
    B, n_in, n_out, G = 500, 11, 20, 10
    x, C, Wb = _inputs(B, n_in, n_out, G, seed=4)
    say("layer special cases")
    # partition of unity: C = 1, Wb = 0 gives y = in_features on the grid
    y = _gpu_layer(x, np.ones_like(C), np.zeros_like(Wb), G, "f32")
    np.testing.assert_allclose(y, float(n_in), rtol=1e-6)
    # base branch only: C = 0
    y = _gpu_layer(x * 3, np.zeros_like(C), Wb, G, "f32")
    ref = oracle.layer(x * 3, np.zeros_like(C), Wb, G)
    assert normwise(y, ref) <= F32_LAYER_TOL
    # spline branch only: Wb = 0, with off-grid inputs
    y = _gpu_layer(x * 3, C, np.zeros_like(Wb), G, "f32")
    ref = oracle.layer(x * 3, C, np.zeros_like(Wb), G)
    assert normwise(y, ref) <= F32_LAYER_TOL


def test_layer_nan_row_and_determinism_and_guard():
    B, n_in, n_out, G = 200, 6, 40, 5
    x, C, Wb = _inputs(B, n_in, n_out, G, seed=5)
    x[17, 3] = np.nan
    say("layer nan/determinism/guard")
    dt = torch.float32
    xt, Ct, Wt = to_dev(x, dt), to_dev(C, dt), to_dev(Wb, dt)
    buf = torch.full((B * n_out + 128,), 3.0, device=device())
    out = buf[64:64 + B * n_out].view(B, n_out)
    kb.layer_forward(xt, Ct, Wt, G, out=out)
    y1 = out.clone()
    kb.layer_forward(xt, Ct, Wt, G, out=out)
    torch.cuda.synchronize()
    assert torch.equal(y1.isnan(), out.isnan())
    assert torch.equal(torch.nan_to_num(y1), torch.nan_to_num(out))
    y = to_host64(out)
    assert np.all(np.isnan(y[17]))
    ok = np.ones(B, bool)
    ok[17] = False
    xr = x.copy()
    xr[17, 3] = 0.0
    ref = oracle.layer(xr, C, Wb, G)
    assert normwise(y[ok], ref[ok]) <= F32_LAYER_TOL
    b = to_host64(buf)
    assert np.all(b[:64] == 3.0) and np.all(b[64 + B * n_out:] == 3.0)


@pytest.mark.parametrize("n_out,cfg", [(256, "2,1,8"), (10, "1,2,8"), (256, None)])
def test_layer_bf16_sparse_nan_row(n_out, cfg):
    """A NaN input makes its whole output row NaN (through the SiLU branch) on
    the sparse MFMA shapes too: the shared-A exchange and the K split carry it
    like any other value; every other row matches the oracle."""
    B, n_in, G = 300, 18, 10
    x, C, Wb = _inputs(B, n_in, n_out, G, seed=9, off=0.2, dtype_name="bf16")
    x[17, 3] = np.nan
    say(f"layer bf16 sparse nan row out={n_out} cfg={cfg}")
    y = _gpu_layer(x, C, Wb, G, "bf16", shape=cfg)
    assert np.all(np.isnan(y[17]))
    ok = np.ones(B, bool)
    ok[17] = False
    assert not np.any(np.isnan(y[ok]))
    xr = x.copy()
    xr[17, 3] = 0.0
    ref = oracle.round_bf16(oracle.layer(xr, C, Wb, G))
    assert normwise(y[ok], ref[ok]) <= BF16_LAYER_TOL


def test_layer_empty_batch():
    say("layer empty batch")
    dt = torch.float32
    y = kb.layer_forward(torch.empty(0, 4, device=device()), torch.zeros(3, 4, 8, device=device()),
                         torch.zeros(3, 4, device=device()), 5)
    torch.cuda.synchronize()
    assert y.shape == (0, 3)


def _sample_rows(B, k, seed):
    rng = np.random.default_rng(seed)
    return np.unique(np.concatenate([rng.integers(0, B, k), [0, B - 1]]))


@pytest.mark.parametrize("name", ["c3_layer_256x256_g10_offgrid", "c4_layer_128x128_g50",
                                  "c4_layer_128x128_g100", "c4_layer_128x128_g200"])
def test_named_layer_full_size_sampled_rows(name):
    """Full-size single-layer workloads in fp32 (launch configuration of the
    benchmark), checked on sampled rows against the oracle."""
    W = wl.make_workload(name)
    x = W["x"]
    C, Wb = W["layers"][0]
    G = W["G"]
    say(f"layer full-size {name}")
    y = kb.layer_forward(to_dev(x, torch.float32), to_dev(C, torch.float32),
                         to_dev(Wb, torch.float32), G)
    torch.cuda.synchronize()
    rows = _sample_rows(x.shape[0], 256, 1)
    got = to_host64(y[torch.from_numpy(rows).to(device())])
    ref = oracle.layer(x[rows], C, Wb, G)
    assert normwise(got, ref) <= F32_LAYER_TOL, normwise(got, ref)


def _downstream_amplification(trace, layers, G, delta=1e-6, seed=0):
    """Oracle-measured normwise amplification, to the network output, of a
    relative perturbation of size delta of each layer's output (information
    for the end-to-end figures; the gate is per layer)."""
    rng = np.random.default_rng(seed)
    final = trace[-1][1]
    amps = []
    for li in range(len(layers)):
        h = trace[li][1] * (1.0 + delta * rng.standard_normal(trace[li][1].shape))
        rest = layers[li + 1:]
        out = oracle.mlp(h, rest, G, bf16=False) if rest else h
        amps.append(normwise(out, final) / delta)
    return amps


@pytest.mark.parametrize("dtype_name", ["f32", "bf16"])
def test_mlp_full_size_production_launch_per_layer(dtype_name):
    """The 3-layer 784 -> 256 -> 256 -> 10 MLP at batch 65536, launched as the
    benchmark launches it (the planner's shapes: in bf16 the shared-A shape
    with its four-stage ring over 392 chunks for 784 -> 256).  For each layer,
    the sampled rows of the GPU output are compared with the plain float64
    oracle (eq. kan_forward with exact basis and SiLU values) fed the GPU's
    own input rows of that layer, and rounded to bf16 in bf16 mode: normwise
    error <= 1e-5 (fp32) and <= 2e-2 (bf16).  End-to-end figures against the
    oracle chain are printed as information."""
    W = wl.make_workload("c5_mlp_784_256_256_10_g10")
    G = W["G"]
    dt = _dtype(dtype_name)
    bf = dtype_name == "bf16"
    B = W["x"].shape[0]
    x = wl.round_to_bf16_f32(W["x"]) if bf else W["x"]
    layers = [(wl.round_to_bf16_f32(C), wl.round_to_bf16_f32(Wb)) if bf else (C, Wb)
              for C, Wb in W["layers"]]
    code = kb.KAN_BF16 if bf else kb.KAN_F32
    want_shape = {"bf16": [(2, 1, 8, 1, 1), (2, 1, 8, 1, 1), (1, 2, 8, 1, 1)],
                  "f32": [(2, 1, 4, 1, 0), (2, 1, 4, 1, 0), (0, 4, 4, 1, 0)]}[dtype_name]
    for (C, _), want in zip(layers, want_shape):
        st, plan = kb.kan_layer_plan(kb.make_grid(G), code, B, C.shape[1], C.shape[0])
        assert st == kb.KAN_OK and plan[:5] == want and plan[5] == 1, (plan, want)
    say(f"mlp full-size production launch {dtype_name}")
    dev_layers = [(to_dev(C, dt), to_dev(Wb, dt)) for C, Wb in layers]
    xt = to_dev(x, dt)
    outs = kb.mlp_forward(xt, dev_layers, G, return_all=True)
    torch.cuda.synchronize()
    rows = _sample_rows(B, 256, 2)
    ridx = torch.from_numpy(rows).to(device())
    ins = [xt] + outs[:-1]
    for li, ((C, Wb), h_in, h_out) in enumerate(zip(layers, ins, outs)):
        xin = to_host64(h_in[ridx])
        ref = oracle.layer(xin, C, Wb, G)
        if bf:
            ref = oracle.round_bf16(ref)
        e = normwise(to_host64(h_out[ridx]), ref)
        say(f"mlp {dtype_name} layer {li + 1} on the GPU's own input: normwise {e:.3e}")
        assert e <= _tol(dtype_name), (li, e)

    # information only: the whole chain against the oracle's own chain
    got = to_host64(outs[-1][ridx])
    trace = oracle.mlp(x[rows], layers, G, bf16=bf, return_all=True)
    e2e = normwise(got, trace[-1][1])
    amps = _downstream_amplification(trace, [(C, Wb) for C, Wb in layers], G)
    info = f"mlp {dtype_name} end to end vs the oracle chain: {e2e:.3e} (amplification {amps})"
    if bf:
        ops = oracle.mlp(x[rows], layers, G, bf16=True, bf16_operands=True)
        info += f"; vs the chain with bf16 contraction operands: {normwise(got, ops):.3e}"
    say(info)


# Narrow fp32 layers (at most 16 outputs) on the vector-ALU kernel, shape
# {0, 4, 4, 1}: one row per lane, the features split over four waves and
# staged 8 at a time.  Ragged batches (one row, a partial last workgroup),
# one input feature, odd counts, partial feature chunks, grids 1 .. 58 (the
# largest it takes), x 10% off the grid.
NARROW_F32 = [
    (1, 2, 5, 5),
    (63, 1, 1, 10),
    (65, 9, 7, 10),
    (1000, 33, 10, 10),
    (130, 17, 16, 26),
    (777, 40, 11, 1),
    (300, 256, 3, 3),
    (129, 784, 13, 10),
    (150, 19, 9, 58),
]


@pytest.mark.parametrize("B,n_in,n_out,G", NARROW_F32)
def test_layer_f32_narrow_kernel(B, n_in, n_out, G):
    x, C, Wb = _inputs(B, n_in, n_out, G, seed=B + n_in + n_out + G, off=0.1)
    say(f"layer f32 narrow B={B} in={n_in} out={n_out} G={G}")
    y = _gpu_layer(x, C, Wb, G, "f32", shape="0,4")
    ref = oracle.layer(x, C, Wb, G)
    assert normwise(y, ref) <= F32_LAYER_TOL, normwise(y, ref)
    # the MFMA kernel on the same inputs: another fp32 summation order
    y2 = _gpu_layer(x, C, Wb, G, "f32", shape="1,1")
    assert normwise(y, y2) <= F32_LAYER_TOL


@pytest.mark.parametrize("n_out", list(range(1, 17)))
def test_layer_f32_narrow_every_output_count(n_out):
    """Each instantiation of the narrow kernel (outputs rounded up to even,
    LDS rows padded to four floats)."""
    B, n_in, G = 200, 21, 10
    x, C, Wb = _inputs(B, n_in, n_out, G, seed=n_out, off=0.1)
    say(f"layer f32 narrow out={n_out}")
    y = _gpu_layer(x, C, Wb, G, "f32", shape="0,4")
    ref = oracle.layer(x, C, Wb, G)
    assert normwise(y, ref) <= F32_LAYER_TOL, normwise(y, ref)


@pytest.mark.parametrize("B,n_in,n_out,G", [(16384, 19, 16, 58), (20000, 40, 5, 10)])
def test_layer_f32_narrow_planned(B, n_in, n_out, G):
    """The planner's own choice from 16384 rows on: the vector-ALU kernel,
    at the largest grid it takes and at a batch that ends inside a
    workgroup."""
    st, plan = kb.kan_layer_plan(kb.make_grid(G), kb.KAN_F32, B, n_in, n_out)
    assert st == kb.KAN_OK and plan[:4] == (0, 4, 4, 1)
    x, C, Wb = _inputs(B, n_in, n_out, G, seed=B + G, off=0.1)
    say(f"layer f32 narrow planned B={B} in={n_in} out={n_out} G={G}")
    y = _gpu_layer(x, C, Wb, G, "f32")
    ref = oracle.layer(x, C, Wb, G)
    assert normwise(y, ref) <= F32_LAYER_TOL, normwise(y, ref)


def test_layer_f32_narrow_nan_row_determinism_and_guard():
    """A NaN input makes only its own row NaN; two runs are bitwise equal;
    nothing is written around the output (a batch that ends inside a
    workgroup)."""
    B, n_in, n_out, G = 200, 37, 10, 10
    x, C, Wb = _inputs(B, n_in, n_out, G, seed=6, off=0.2)
    x[17, 30] = np.nan
    say("layer f32 narrow nan/determinism/guard")
    dt = torch.float32
    p = kb.pack_layer(to_dev(C, dt), to_dev(Wb, dt), G)
    xt = to_dev(x, dt)
    buf = torch.full((B * n_out + 128,), 3.0, device=device())
    out = buf[64:64 + B * n_out].view(B, n_out)
    kb.layer_forward_packed(xt, p, out=out, shape="0,4")
    y1 = out.clone()
    kb.layer_forward_packed(xt, p, out=out, shape="0,4")
    torch.cuda.synchronize()
    assert torch.equal(y1.isnan(), out.isnan())
    assert torch.equal(torch.nan_to_num(y1), torch.nan_to_num(out))
    y = to_host64(out)
    assert np.all(np.isnan(y[17]))
    ok = np.ones(B, bool)
    ok[17] = False
    assert not np.any(np.isnan(y[ok]))
    xr = x.copy()
    xr[17, 30] = 0.0
    ref = oracle.layer(xr, C, Wb, G)
    assert normwise(y[ok], ref[ok]) <= F32_LAYER_TOL
    b = to_host64(buf)
    assert np.all(b[:64] == 3.0) and np.all(b[64 + B * n_out:] == 3.0)


def _knot_inputs(G, dtype_name, lo=-1.0, hi=1.0):
    """Every knot t_0 .. t_{G+6} in the storage dtype, each one unit in the
    last place below and above it, lo, hi, zero and a few points past the
    outermost knots."""
    t = oracle.knots(G, lo, hi).astype(np.float32)
    if dtype_name == "bf16":
        tb = wl.round_to_bf16_f32(t)
        bits = tb.view(np.uint32)
        up = np.where(tb >= 0, bits + 0x10000, bits - 0x10000).astype(np.uint32).view(np.float32)
        dn = np.where(tb > 0, bits - 0x10000, bits + 0x10000).astype(np.uint32).view(np.float32)
        dn = np.where(tb == 0, np.float32(-2.0 ** -133), dn)
        pts = [tb, up, dn]
    else:
        pts = [t, np.nextafter(t, np.float32(np.inf)), np.nextafter(t, np.float32(-np.inf))]
    extra = np.array([lo, hi, 0.0, t[0] - 0.5, t[-1] + 0.5, 10.0, -10.0], np.float32)
    v = np.concatenate(pts + [extra]).astype(np.float32)
    return wl.round_to_bf16_f32(v) if dtype_name == "bf16" else v


KNOT_CASES = [
    # (dtype, G, in, out, shape): G = 8 (every knot exact in bf16) and G = 10
    # on the sparse bf16 shapes (shared A on 256 columns, 32-row waves, K
    # split on a narrow tile), the dense bf16 kernel (G = 16), and fp32
    ("bf16", 8, 18, 256, None), ("bf16", 8, 18, 256, "2,1,8"), ("bf16", 8, 18, 256, "1,1,8"),
    ("bf16", 8, 18, 10, "1,2,8"), ("bf16", 10, 18, 256, "2,1,8"), ("bf16", 10, 18, 10, None),
    ("bf16", 10, 17, 45, "1,1,4,2"), ("bf16", 16, 18, 256, None), ("bf16", 16, 18, 45, "1,2"),
    ("f32", 8, 18, 256, None), ("f32", 10, 18, 45, "2,1"), ("f32", 10, 17, 10, "1,4"),
    # fp32 narrow layers on the vector-ALU kernel (its own window arithmetic)
    ("f32", 8, 18, 10, "0,4"), ("f32", 10, 17, 16, "0,4"), ("f32", 26, 5, 1, "0,4"),
    ("f32", 58, 7, 16, "0,4"),
]


@pytest.mark.parametrize("dtype_name,G,n_in,n_out,cfg", KNOT_CASES)
def test_layer_inputs_on_knots(dtype_name, G, n_in, n_out, cfg):
    """Inputs exactly on every knot, one ulp either side, the grid ends, and
    past the outermost knots, through the fused layer: the span window of the
    sparse generation and the clamp (eq. bounded: exact zeros at the support
    ends) change exactly there."""
    v = _knot_inputs(G, dtype_name)
    B = 300
    rng = np.random.default_rng(G + n_in)
    x = v[rng.integers(0, v.size, (B, n_in))]
    x[: (v.size + n_in - 1) // n_in].reshape(-1)[: v.size] = v  # every point at least once
    _, C, Wb = _inputs(B, n_in, n_out, G, seed=G, dtype_name=dtype_name)
    ref = oracle.layer(x, C, Wb, G)
    if dtype_name == "bf16":
        ref = oracle.round_bf16(ref)
    say(f"layer knots {dtype_name} G={G} in={n_in} out={n_out} cfg={cfg}")
    y = _gpu_layer(x, C, Wb, G, dtype_name, shape=cfg)
    assert normwise(y, ref) <= _tol(dtype_name), normwise(y, ref)


# Small batches split the contraction across workgroups (fp32 partial sums in
# the workspace, added in a fixed order): (dtype, B, in, out, G, k), the
# planned shape, on the sparse and dense bf16 layouts, fp32 and degree 5.
K_SPLIT_CASES = [("f32", 1, 784, 64, 5, 3), ("f32", 256, 784, 64, 5, 3),
                 ("f32", 7, 300, 10, 10, 3), ("bf16", 256, 784, 64, 5, 3),
                 ("bf16", 33, 300, 256, 10, 3), ("bf16", 100, 520, 45, 16, 3),
                 ("f32", 64, 200, 40, 8, 5), ("bf16", 64, 520, 40, 8, 5)]


@pytest.mark.parametrize("dtype_name,B,n_in,n_out,G,k", K_SPLIT_CASES)
def test_layer_k_split_small_batches(dtype_name, B, n_in, n_out, G, k):
    dt = torch.float32 if dtype_name == "f32" else torch.bfloat16
    code = kb.KAN_F32 if dtype_name == "f32" else kb.KAN_BF16
    st, plan = kb.kan_layer_plan(kb.make_grid(G, spline_order=k), code, B, n_in, n_out)
    assert st == kb.KAN_OK and plan[5] > 1
    rng = np.random.default_rng(B + n_in)
    h = 2.0 / G
    x = rng.uniform(-1 - 2 * h, 1 + 2 * h, (B, n_in)).astype(np.float32)
    _, C, Wb = wl.make_layer(wl.LayerShape(B, n_in, n_out, G), B, k=k)
    if dtype_name == "bf16":
        x, C, Wb = (wl.round_to_bf16_f32(a) for a in (x, C, Wb))
    xd, Cd, Wd = to_dev(x, dt), to_dev(C, dt), to_dev(Wb, dt)
    say(f"layer K split {dtype_name} B={B} in={n_in} out={n_out} G={G} k={k} splits={plan[5]}")
    pk = kb.pack_layer(Cd, Wd, G, spline_order=k)
    y1 = kb.layer_forward_packed(xd, pk)
    y2 = kb.layer_forward_packed(xd, pk)
    y0 = kb.layer_forward_packed(xd, pk, split=False)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)  # fixed summation order
    ref = oracle.layer(x, C, Wb, G, k=k)
    tol = _tol(dtype_name)
    if dtype_name == "bf16":
        ref = oracle.round_bf16(ref)
    assert normwise(to_host64(y1), ref) <= tol
    assert normwise(to_host64(y0), ref) <= tol


def test_layer_k_split_forced_shapes():
    """The split under forced shapes: a K split inside the workgroup as well,
    and column slices."""
    B, n_in, n_out, G = 40, 257, 64, 10
    x, C, Wb = _inputs(B, n_in, n_out, G, seed=31, off=0.2, dtype_name="f32")
    ref = oracle.layer(x, C, Wb, G)
    for cfg in ("1,2", "1,4", "1,1,4,2", "2,1"):
        st, plan = kb.kan_layer_plan(kb.make_grid(G), kb.KAN_F32, B, n_in, n_out, cfg)
        assert st == kb.KAN_OK and plan[5] > 1
        say(f"layer K split forced {cfg} splits={plan[5]}")
        y = _gpu_layer(x, C, Wb, G, "f32", shape=cfg)
        assert normwise(y, ref) <= F32_LAYER_TOL, cfg


def _random_split_cases(n_per_dtype=8, seed=2026):
    """Seeded random layers (degree 1-5, grids 3-40, both dtypes) at batches
    small enough that kan_layer_plan splits the contraction."""
    rng = np.random.default_rng(seed)
    cases = {"f32": [], "bf16": []}
    while min(len(v) for v in cases.values()) < n_per_dtype:
        dtype_name = "f32" if rng.random() < 0.5 else "bf16"
        if len(cases[dtype_name]) >= n_per_dtype:
            continue
        k = int(rng.choice([3, 3, 3, 1, 2, 5]))
        G = int(rng.choice([3, 5, 8, 10, 12, 20, 40]))
        B = int(rng.integers(1, 97))
        n_in = int(rng.integers(40, 401))
        n_out = int(rng.integers(1, 129))
        code = kb.KAN_F32 if dtype_name == "f32" else kb.KAN_BF16
        st, plan = kb.kan_layer_plan(kb.make_grid(G, spline_order=k), code, B, n_in, n_out)
        if st == kb.KAN_OK and plan[5] > 1:
            cases[dtype_name].append((dtype_name, B, n_in, n_out, G, k))
    return cases["f32"] + cases["bf16"]


@pytest.mark.parametrize("dtype_name,B,n_in,n_out,G,k", _random_split_cases())
def test_layer_k_split_random_layers(dtype_name, B, n_in, n_out, G, k):
    """The split contraction on random layer sizes: within tolerance of the
    oracle, equal to the unsplit layer up to the fp32 summation order, and
    the same on a second call."""
    dt = _dtype(dtype_name)
    rng = np.random.default_rng(B * 1000 + n_in + n_out + G)
    h = 2.0 / G
    x = rng.uniform(-1 - 2 * h, 1 + 2 * h, (B, n_in)).astype(np.float32)
    _, C, Wb = wl.make_layer(wl.LayerShape(B, n_in, n_out, G), B + n_out, k=k)
    if dtype_name == "bf16":
        x, C, Wb = (wl.round_to_bf16_f32(a) for a in (x, C, Wb))
    say(f"layer K split random {dtype_name} B={B} in={n_in} out={n_out} G={G} k={k}")
    pk = kb.pack_layer(to_dev(C, dt), to_dev(Wb, dt), G, spline_order=k)
    xd = to_dev(x, dt)
    y1 = kb.layer_forward_packed(xd, pk)
    y2 = kb.layer_forward_packed(xd, pk)
    y0 = kb.layer_forward_packed(xd, pk, split=False)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)
    ref = oracle.layer(x, C, Wb, G, k=k)
    if dtype_name == "bf16":
        ref = oracle.round_bf16(ref)
    assert normwise(to_host64(y1), ref) <= _tol(dtype_name)
    assert normwise(to_host64(y1), to_host64(y0)) <= _tol(dtype_name)
