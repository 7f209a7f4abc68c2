"""Host-side shape planning of the fused layer through kan_layer_plan (no GPU):
the shapes chosen for the layers of the 784-256-256-10 MLP, which grids run
on the structured-sparse matrix instruction, that every shape the GPU parity
tests force is valid and is the one that runs, that invalid forced shapes are
rejected, and argument checks."""
import pytest

from paper_2609_01956_amd import binding as kb

import test_gpu_layer as gl

DT = {"f32": kb.KAN_F32, "bf16": kb.KAN_BF16}


def _plan(G, dtype_name, B, n_in, n_out, cfg=None):
    """(rf, wk, nw, cs, sparse) of the planned or forced shape."""
    st, plan = kb.kan_layer_plan(kb.make_grid(G), DT[dtype_name], B, n_in, n_out, cfg)
    assert st == kb.KAN_OK
    return plan[:5]


def _splits(G, dtype_name, B, n_in, n_out, cfg=None):
    st, plan = kb.kan_layer_plan(kb.make_grid(G), DT[dtype_name], B, n_in, n_out, cfg)
    assert st == kb.KAN_OK
    return plan[5]


def _rejected(G, dtype_name, B, n_in, n_out, cfg):
    st, _ = kb.kan_layer_plan(kb.make_grid(G), DT[dtype_name], B, n_in, n_out, cfg)
    return st == kb.KAN_ERR_INVALID_ARG


def _shape(cfg):
    v = [int(t) for t in cfg.split(",")]
    return tuple(v + [4, 1][len(v) - 2:])


@pytest.mark.parametrize("dtype_name,n_in,n_out,want", [
    # eight waves per workgroup: on the 256-column layers 64-row waves over
    # column halves sharing A, on the narrow layer 32-row waves in two slices
    # of the feature pairs
    ("bf16", 784, 256, (2, 1, 8, 1, 1)),
    ("bf16", 256, 256, (2, 1, 8, 1, 1)),
    ("bf16", 256, 10, (1, 2, 8, 1, 1)),
    # fp32: 64-row waves over 128-column tiles; the narrow layer on the
    # vector-ALU kernel
    ("f32", 784, 256, (2, 1, 4, 1, 0)),
    ("f32", 256, 256, (2, 1, 4, 1, 0)),
    ("f32", 256, 10, (0, 4, 4, 1, 0)),
])
def test_mlp_layers_planned_shapes(dtype_name, n_in, n_out, want):
    assert _plan(10, dtype_name, 65536, n_in, n_out) == want


@pytest.mark.parametrize("B,n_out,want", [
    # narrow sparse tiles: two K slices of eight-wave workgroups when that
    # still gives a workgroup per CU, more slices of four waves below that
    (65536, 64, (1, 2, 8, 1, 1)),
    (32768, 10, (1, 2, 8, 1, 1)),
    (16384, 10, (1, 4, 4, 1, 1)),
    # four fragments: no K split on the sparse layout's wider tiles
    (65536, 100, (1, 1, 8, 1, 1)),
])
def test_narrow_sparse_layers_planned_shapes(B, n_out, want):
    assert _plan(10, "bf16", B, 256, n_out) == want


@pytest.mark.parametrize("G,sparse", [(1, 0), (4, 0), (5, 1), (10, 1), (12, 1), (13, 0),
                                      (200, 0)])
def test_sparse_instruction_for_two_blocks_per_feature(G, sparse):
    # bf16 blocks hold 8 of a feature's G + 4 columns: two blocks for 5..12
    assert _plan(G, "bf16", 4096, 64, 64)[4] == sparse
    assert _plan(G, "f32", 4096, 64, 64)[4] == 0


def test_shared_a_shape_only_on_sparse_256_column_tiles():
    assert _plan(10, "bf16", 65536, 784, 256, "2,1,8") == (2, 1, 8, 1, 1)
    # its epilogue stores bf16 rows through LDS: it never splits the
    # contraction, also when forced on a batch that splits on other shapes
    assert _splits(10, "bf16", 64, 784, 256, "2,1,8") == 1
    assert _splits(10, "bf16", 64, 784, 256, "1,1,8") > 1
    # dense bf16, fp32 and narrower sparse tiles reject it
    for G, dt, n_out in [(20, "bf16", 256), (10, "f32", 256), (10, "bf16", 45)]:
        assert _rejected(G, dt, 65536, 784, n_out, "2,1,8")


def test_sparse_k_split_only_on_narrow_tiles():
    # waves splitting K on the sparse layout: tiles of one or two fragments;
    # eight-wave K splits are not shapes of the dense kernel
    assert _plan(10, "bf16", 65536, 256, 10, "1,4,8") == (1, 4, 8, 1, 1)
    assert _plan(10, "bf16", 65536, 256, 64, "1,2") == (1, 2, 4, 1, 1)
    for G, dt, n_out, cfg in [(10, "bf16", 256, "1,2"), (10, "bf16", 100, "1,4"),
                              (20, "bf16", 10, "1,4,8"), (10, "f32", 10, "1,2,8")]:
        assert _rejected(G, dt, 65536, 256, n_out, cfg)


def test_narrow_kernel_shape():
    """The vector-ALU kernel {0, 4, 4, 1}: fp32 cubic layers of 1 .. 16
    outputs with G <= 58, planned from batch 16384 on (below that the MFMA
    kernel's K split fills the GPU), never split."""
    assert _plan(10, "f32", 16384, 256, 10) == (0, 4, 4, 1, 0)
    assert _splits(10, "f32", 16384, 256, 10) == 1
    assert _plan(10, "f32", 16383, 256, 10)[0] != 0
    assert _plan(10, "f32", 65536, 2, 5) == (0, 4, 4, 1, 0)
    assert _plan(58, "f32", 65536, 256, 16) == (0, 4, 4, 1, 0)
    assert _plan(10, "f32", 65536, 256, 17)[0] != 0
    assert _plan(59, "f32", 65536, 256, 10)[0] != 0
    assert _plan(10, "bf16", 65536, 256, 10)[0] != 0
    # forced: any batch; the same limits
    assert _plan(10, "f32", 1, 256, 10, "0,4") == (0, 4, 4, 1, 0)
    assert _splits(10, "f32", 64, 784, 10, "0,4") == 1
    for G, dt, n_out, cfg in [(10, "bf16", 10, "0,4"), (10, "f32", 17, "0,4"),
                              (59, "f32", 10, "0,4"), (10, "f32", 10, "0,4,8"),
                              (10, "f32", 10, "0,2"), (10, "f32", 10, "0,4,4,2")]:
        assert _rejected(G, dt, 65536, 256, n_out, cfg), (G, dt, n_out, cfg)
    st, _ = kb.kan_layer_plan(kb.make_grid(10, spline_order=2), DT["f32"], 65536, 256, 10, "0,4")
    assert st == kb.KAN_ERR_INVALID_ARG


@pytest.mark.parametrize("cfg", ["3,1", "1,3", "1,1,6", "1,1,4,3", "0,1", "1,2,8"])
def test_invalid_forced_shape_is_rejected(cfg):
    assert _rejected(10, "bf16", 65536, 784, 256, cfg)
    g = kb.make_grid(10)
    # the forward rejects it on the host too (fake addresses are never touched)
    st, need = kb.kan_layer_packed_bytes(g, kb.KAN_BF16, 784, 256)
    assert kb.kan_layer_forward_packed(g, kb.KAN_BF16, 16, 784, 256, 0x100000, 0x200000000,
                                       need, 0x400000000, shape=cfg) == kb.KAN_ERR_INVALID_ARG


def _forced_cases():
    for dtype_name, G in [("f32", 10), ("bf16", 20), ("bf16", 10)]:
        for cfg in gl.CFGS:
            if dtype_name == "bf16" and G == 10 and cfg not in gl.SPARSE_CFGS:
                continue
            yield dtype_name, G, 300, 9, 45, cfg
    for dtype_name, B, n_in, n_out, G, cfg in gl.WIDE:
        yield dtype_name, G, B, n_in, n_out, cfg
    for cfg in gl.SPARSE_256_CFGS:
        yield "bf16", 10, 700, 13, 256, cfg
    for cfg in gl.X_WORD_CFGS:
        if cfg is not None:
            yield "bf16", 10, 300, 9, 45, cfg
    for B, n_in, n_out, G in gl.NARROW_SHAPES:
        for cfg in gl.NARROW_CFGS:
            yield "bf16", G, B, n_in, n_out, cfg
    for dtype_name, G, n_in, n_out, cfg in gl.KNOT_CASES:
        if cfg is not None:
            yield dtype_name, G, 300, n_in, n_out, cfg
    for B, n_in, n_out, G in gl.NARROW_F32:
        yield "f32", G, B, n_in, n_out, "0,4"
    for n_out, _ in gl.STAGED_CASES:
        yield "bf16", 10, 300, 13, n_out, "2,1,8"


@pytest.mark.parametrize("dtype_name,G,B,n_in,n_out,cfg", list(_forced_cases()))
def test_every_shape_the_gpu_tests_force_is_the_one_that_runs(dtype_name, G, B,
                                                              n_in, n_out, cfg):
    assert _plan(G, dtype_name, B, n_in, n_out, cfg)[:4] == _shape(cfg)


def test_plan_argument_checks():
    g = kb.make_grid(10)
    bad = kb.KAN_ERR_INVALID_ARG
    assert kb.kan_layer_plan(g, kb.KAN_BF16, 0, 4, 4)[0] == bad
    assert kb.kan_layer_plan(g, kb.KAN_BF16, -1, 4, 4)[0] == bad
    assert kb.kan_layer_plan(g, kb.KAN_BF16, 16, 0, 4)[0] == bad
    assert kb.kan_layer_plan(g, kb.KAN_BF16, 16, 4, 0)[0] == bad
    assert kb.kan_layer_plan(g, 2, 16, 4, 4)[0] == kb.KAN_ERR_UNSUPPORTED
    lib = kb.load_library()
    assert lib.kan_layer_plan(None, 0, 16, 4, 4, None, None) == bad
    assert lib.kan_layer_plan(g, 0, 16, 4, 4, None, None) == bad


@pytest.mark.parametrize("dtype_name", ["f32", "bf16"])
def test_k_split_only_for_small_batches(dtype_name):
    """Batches whose workgroups number fewer than 512 split the contraction
    across workgroups; the MLP's full batch and layers of few chunks never
    split."""
    for n_in, n_out in ((784, 256), (256, 256), (256, 10)):
        assert _splits(10, dtype_name, 65536, n_in, n_out) == 1
    assert _splits(10, dtype_name, 256, 784, 64) > 1
    assert _splits(10, dtype_name, 1, 784, 256) > 1
    assert _splits(10, dtype_name, 256, 2, 5) == 1   # one chunk
    # the split count falls as the batch grows
    ks = [_splits(5, dtype_name, B, 784, 64) for B in (1, 256, 4096, 65536)]
    assert ks == sorted(ks, reverse=True) and ks[-1] == 1


def test_k_split_needs_two_splits_of_four_chunks():
    """A layer splits only if its K chunks make at least two splits of 4
    chunks and 16 blocks: bf16 32 -> 10 at G = 10 (4 chunks of 8 blocks)
    never does, 64 -> 10 (8 chunks) does; bf16 256-column tiles (2 blocks per
    chunk) need 16 chunks: 32 -> 256 (16 chunks) does, 16 -> 256 (8) not."""
    for B in (1, 64, 1024):
        assert _splits(10, "bf16", B, 32, 10) == 1
        assert _splits(10, "bf16", B, 64, 10) > 1
    assert _splits(10, "bf16", 1, 32, 256) == 2
    assert _splits(10, "bf16", 1, 16, 256) == 1


@pytest.mark.parametrize("dtype_name", ["f32", "bf16"])
def test_k_split_partial_sums_bounded(dtype_name):
    """The fp32 partial sums of a split stay within 16 MiB, and the workspace
    size query covers them."""
    code = DT[dtype_name]
    for B, n_in, n_out, G in ((1, 784, 256, 10), (4096, 784, 256, 10), (8192, 784, 256, 10),
                              (2048, 2000, 512, 10), (64, 784, 64, 5)):
        ks = _splits(G, dtype_name, B, n_in, n_out)
        assert ks * B * n_out * 4 <= 16 << 20 or ks == 1
        st, n = kb.kan_layer_forward_packed_workspace_bytes(kb.make_grid(G), code, B, n_in, n_out)
        assert st == kb.KAN_OK
        assert (n == 0) == (ks == 1)
        assert n == 0 or n >= ks * B * n_out * 4
