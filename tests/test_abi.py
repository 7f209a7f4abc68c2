"""C ABI checks that need no GPU: the library loads, exports every function
declared in include/kan.h, and rejects every invalid argument on the host
with the documented status code before touching the device."""
import ctypes
import math
import os
import re

import pytest

from paper_2609_01956_amd import binding as kb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "kan.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(kan_[a-z_0-9]+)\s*\(", src)))


def test_header_declares_the_entry_points():
    names = _declared_functions()
    assert names == sorted(kb.EXPORTED_SYMBOLS)


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(kb.LIB_PATH)
    for name in _declared_functions():
        assert hasattr(lib, name), name


def test_abi_version_and_status_strings():
    assert kb.kan_abi_version() == 4
    names = ["KAN_OK", "KAN_ERR_INVALID_ARG", "KAN_ERR_UNSUPPORTED", "KAN_ERR_DEVICE",
             "KAN_ERR_SCRATCH_LIMIT"]
    for code, name in enumerate(names):
        assert kb.kan_status_string(code).startswith(name)
    assert kb.kan_status_string(99) == "unknown kan_status"


# Fake, well-aligned, non-overlapping addresses: validation must reject every
# case below on the host, so these are never dereferenced.
X, PHI, C, W, Y = 0x100000, 0x200000000, 0x300000000, 0x400000000, 0x500000000
WS, WSB = 0x700000000, 1 << 30  # a workspace large enough for every layer below


@pytest.mark.parametrize("grid,code", [
    (kb.make_grid(5, spline_order=0), kb.KAN_ERR_UNSUPPORTED),
    (kb.make_grid(5, spline_order=8), kb.KAN_ERR_UNSUPPORTED),
    (kb.make_grid(5, spline_order=-1), kb.KAN_ERR_UNSUPPORTED),
    (kb.make_grid(0), kb.KAN_ERR_INVALID_ARG),
    (kb.make_grid(-3), kb.KAN_ERR_INVALID_ARG),
    (kb.make_grid(4001), kb.KAN_ERR_INVALID_ARG),
    (kb.make_grid(5, 1.0, 1.0), kb.KAN_ERR_INVALID_ARG),
    (kb.make_grid(5, 2.0, -1.0), kb.KAN_ERR_INVALID_ARG),
    (kb.make_grid(5, math.nan, 1.0), kb.KAN_ERR_INVALID_ARG),
    (kb.make_grid(5, -1.0, math.inf), kb.KAN_ERR_INVALID_ARG),
    (kb.make_grid(5, 1e30, 1e30 * (1 + 1e-6)), kb.KAN_ERR_INVALID_ARG),  # lo/h beyond 2^22
])
def test_bad_grid(grid, code):
    assert kb.kan_basis_eval(grid, kb.KAN_F32, X, 16, PHI) == code
    assert kb.kan_layer_forward(grid, kb.KAN_F32, 16, 4, 4, X, C, W, WS, WSB, Y) == code


def test_null_grid_and_bad_dtype():
    lib = kb.load_library()
    assert lib.kan_basis_eval(None, 0, X, 16, PHI, None) == kb.KAN_ERR_INVALID_ARG
    assert lib.kan_layer_forward(None, 0, 16, 4, 4, X, C, W, WS, WSB, Y, None) == kb.KAN_ERR_INVALID_ARG
    g = kb.make_grid(5)
    assert kb.kan_basis_eval(g, 2, X, 16, PHI) == kb.KAN_ERR_UNSUPPORTED
    assert kb.kan_basis_eval(g, -1, X, 16, PHI) == kb.KAN_ERR_UNSUPPORTED


def test_basis_argument_checks():
    g = kb.make_grid(5)
    f32, bf = kb.KAN_F32, kb.KAN_BF16
    assert kb.kan_basis_eval(g, f32, X, -1, PHI) == kb.KAN_ERR_INVALID_ARG
    assert kb.kan_basis_eval(g, f32, 0, 16, PHI) == kb.KAN_ERR_INVALID_ARG
    assert kb.kan_basis_eval(g, f32, X, 16, 0) == kb.KAN_ERR_INVALID_ARG
    assert kb.kan_basis_eval(g, f32, X + 2, 16, PHI) == kb.KAN_ERR_INVALID_ARG   # misaligned f32
    assert kb.kan_basis_eval(g, f32, X, 16, PHI + 1) == kb.KAN_ERR_INVALID_ARG
    assert kb.kan_basis_eval(g, bf, X + 1, 16, PHI) == kb.KAN_ERR_INVALID_ARG    # misaligned bf16
    # output overlapping the input
    assert kb.kan_basis_eval(g, f32, X, 16, X + 32) == kb.KAN_ERR_INVALID_ARG
    assert kb.kan_basis_eval(g, f32, X + 64, 16, X) == kb.KAN_ERR_INVALID_ARG
    # n * (G + 3) overflowing
    assert kb.kan_basis_eval(g, f32, X, 2 ** 62, PHI) == kb.KAN_ERR_INVALID_ARG
    # empty problem: OK, launches nothing, pointers unchecked
    assert kb.kan_basis_eval(g, f32, 0, 0, 0) == kb.KAN_OK
    assert kb.kan_basis_eval(g, bf, 0, 0, 0) == kb.KAN_OK


def test_layer_argument_checks():
    g = kb.make_grid(10)
    f32 = kb.KAN_F32
    bad = kb.KAN_ERR_INVALID_ARG
    assert kb.kan_layer_forward(g, f32, -1, 4, 4, X, C, W, WS, WSB, Y) == bad
    assert kb.kan_layer_forward(g, f32, 16, 0, 4, X, C, W, WS, WSB, Y) == bad
    assert kb.kan_layer_forward(g, f32, 16, 4, 0, X, C, W, WS, WSB, Y) == bad
    assert kb.kan_layer_forward(g, f32, 16, 2 ** 30, 4, X, C, W, WS, WSB, Y) == bad  # in * (G + 4) >= 2^31
    assert kb.kan_layer_forward(g, f32, 16, 4, 4, 0, C, W, WS, WSB, Y) == bad
    assert kb.kan_layer_forward(g, f32, 16, 4, 4, X, 0, W, WS, WSB, Y) == bad
    assert kb.kan_layer_forward(g, f32, 16, 4, 4, X, C, 0, WS, WSB, Y) == bad
    assert kb.kan_layer_forward(g, f32, 16, 4, 4, X, C, W, WS, WSB, 0) == bad
    assert kb.kan_layer_forward(g, f32, 16, 4, 4, X, C + 2, W, WS, WSB, Y) == bad
    assert kb.kan_layer_forward(g, f32, 16, 4, 4, X, C, W, WS, WSB, Y + 2) == bad
    # y overlapping each input
    assert kb.kan_layer_forward(g, f32, 16, 4, 4, X, C, W, WS, WSB, X + 8) == bad
    assert kb.kan_layer_forward(g, f32, 16, 4, 4, X, C, W, WS, WSB, C + 8) == bad
    assert kb.kan_layer_forward(g, f32, 16, 4, 4, X, C, W, WS, WSB, W) == bad
    # x byte offsets of a workgroup are 32-bit: 256 rows x in x 4 bytes must
    # stay below 2^32 (in both dtypes)
    g1 = kb.make_grid(1)
    for dt in (f32, kb.KAN_BF16):
        assert kb.kan_layer_forward(g1, dt, 16, 2 ** 22, 1, X, C, W, WS, WSB, Y) == bad
        assert kb.kan_layer_forward_packed(g1, dt, 16, 2 ** 22, 1, X, C, WSB, Y) == bad
        assert kb.kan_layer_plan(g1, dt, 16, 2 ** 22, 1)[0] == bad
        assert kb.kan_layer_packed_bytes(g1, dt, 2 ** 22, 1)[0] == bad
        assert kb.kan_layer_packed_bytes(g1, dt, 2 ** 22 - 1, 1)[0] == kb.KAN_OK
    # workspace: null, misaligned (16 bytes), short, overlapping any tensor
    # (16 rows of 784 -> 4: the packed weights, then the partial sums of the
    # split contraction; the packed weights' size is the least accepted)
    need = kb.kan_layer_forward_workspace_bytes(g, f32, 16, 784, 4)[1]
    packed = kb.kan_layer_packed_bytes(g, f32, 784, 4)[1]
    assert need > packed
    assert kb.kan_layer_forward(g, f32, 16, 784, 4, X, C, W, 0, need, Y) == bad
    assert kb.kan_layer_forward(g, f32, 16, 784, 4, X, C, W, WS + 8, need, Y) == bad
    assert kb.kan_layer_forward(g, f32, 16, 784, 4, X, C, W, WS, packed - 1, Y) == bad
    for p in (X, C, W, Y):
        assert kb.kan_layer_forward(g, f32, 16, 784, 4, X, C, W, p - 16, need, Y) == bad
    # empty batch: OK without launching
    assert kb.kan_layer_forward(g, f32, 0, 4, 4, 0, 0, 0, 0, 0, 0) == kb.KAN_OK


def _expected_packed_bytes(G, bf16, n_in, n_out):
    """Size of the packed weights: per tile of 32 * nf output columns, per pair of
    features, per block of kj columns, kj weights for each of 2 * 32 * nf
    (feature, column) slots; the blocks of a tile are padded to whole chunks of
    min(8, 16 KiB / block bytes) blocks."""
    kj, es, nfmax = (8, 2, 8) if bf16 else (2, 4, 4)
    nsb = -(-(G + 4) // kj)
    npairs = -(-n_in // 2)
    nf = 1
    while nf < nfmax and 32 * nf < n_out:
        nf *= 2
    ntiles = -(-n_out // (32 * nf))
    blk_bytes = 2 * 32 * nf * kj * es
    kb = min(8, 16384 // blk_bytes)
    nblk_pad = -(-(npairs * nsb) // kb) * kb
    return ntiles * nblk_pad * blk_bytes


@pytest.mark.parametrize("G,n_in,n_out", [(10, 784, 256), (10, 256, 10), (5, 2, 5), (200, 128, 128),
                                          (7, 3, 300), (1, 1, 1), (50, 129, 65)])
@pytest.mark.parametrize("bf16", [False, True])
def test_packed_bytes(G, n_in, n_out, bf16):
    st, n = kb.kan_layer_packed_bytes(kb.make_grid(G), kb.KAN_BF16 if bf16 else kb.KAN_F32,
                                      n_in, n_out)
    assert st == kb.KAN_OK
    assert n == _expected_packed_bytes(G, bf16, n_in, n_out)
    # 784 -> 256, G = 10 in bf16: 392 pairs x 2 blocks x 8 KiB
    if (G, n_in, n_out, bf16) == (10, 784, 256, True):
        assert n == 392 * 2 * 8192


def test_workspace_bytes_checks():
    g = kb.make_grid(10)
    bad = kb.KAN_ERR_INVALID_ARG
    lib = kb.load_library()
    assert lib.kan_layer_forward_workspace_bytes(ctypes.byref(g), 0, 16, 4, 4, None) == bad
    assert kb.kan_layer_forward_workspace_bytes(g, kb.KAN_F32, -1, 4, 4)[0] == bad
    assert kb.kan_layer_forward_workspace_bytes(g, kb.KAN_F32, 16, 0, 4)[0] == bad
    assert kb.kan_layer_forward_workspace_bytes(kb.make_grid(10, spline_order=8), kb.KAN_F32,
                                                16, 4, 4)[0] == kb.KAN_ERR_UNSUPPORTED
    # the packed weights, plus the split contraction's fp32 partial sums for
    # batches too small to fill the GPU
    for B in (0, 65536):
        st, n = kb.kan_layer_forward_workspace_bytes(g, kb.KAN_BF16, B, 784, 256)
        assert st == kb.KAN_OK and n == 392 * 2 * 8192
    st, n = kb.kan_layer_forward_workspace_bytes(g, kb.KAN_BF16, 1, 784, 256)
    st2, ks = kb.kan_layer_plan(g, kb.KAN_BF16, 1, 784, 256)
    assert st == st2 == kb.KAN_OK and ks[5] > 1
    assert n == 392 * 2 * 8192 + -(-ks[5] * 1 * 256 * 4 // 256) * 256


def test_packed_entry_point_checks():
    g = kb.make_grid(10)
    f32, bad = kb.KAN_F32, kb.KAN_ERR_INVALID_ARG
    P = 0x600000000
    lib = kb.load_library()
    assert lib.kan_layer_packed_bytes(ctypes.byref(g), f32, 4, 4, None) == bad
    assert kb.kan_layer_packed_bytes(g, f32, 0, 4)[0] == bad
    assert kb.kan_layer_packed_bytes(g, f32, 4, 0)[0] == bad
    assert kb.kan_layer_packed_bytes(kb.make_grid(10, spline_order=9), f32, 4, 4)[0] == \
        kb.KAN_ERR_UNSUPPORTED
    need = kb.kan_layer_packed_bytes(g, f32, 4, 4)[1]
    # pack: null, misaligned (16 bytes for the packed buffer), short, overlapping
    assert kb.kan_layer_pack(g, f32, 4, 4, 0, W, P, need) == bad
    assert kb.kan_layer_pack(g, f32, 4, 4, C, 0, P, need) == bad
    assert kb.kan_layer_pack(g, f32, 4, 4, C, W, 0, need) == bad
    assert kb.kan_layer_pack(g, f32, 4, 4, C, W, P + 8, need) == bad
    assert kb.kan_layer_pack(g, f32, 4, 4, C, W, P, need - 1) == bad
    assert kb.kan_layer_pack(g, f32, 4, 4, C, W, C, need) == bad
    assert kb.kan_layer_pack(g, f32, 4, 4, C, W, W - 16, need) == bad
    # forward_packed: null, misaligned, short, overlapping, negative / empty batch
    assert kb.kan_layer_forward_packed(g, f32, 16, 4, 4, 0, P, need, Y) == bad
    assert kb.kan_layer_forward_packed(g, f32, 16, 4, 4, X, 0, need, Y) == bad
    assert kb.kan_layer_forward_packed(g, f32, 16, 4, 4, X, P, need, 0) == bad
    assert kb.kan_layer_forward_packed(g, f32, 16, 4, 4, X, P + 4, need, Y) == bad
    assert kb.kan_layer_forward_packed(g, f32, 16, 4, 4, X, P, need - 16, Y) == bad
    assert kb.kan_layer_forward_packed(g, f32, 16, 4, 4, X, P, need, P + 16) == bad
    assert kb.kan_layer_forward_packed(g, f32, 16, 4, 4, X, P, need, X + 4) == bad
    assert kb.kan_layer_forward_packed(g, f32, -1, 4, 4, X, P, need, Y) == bad
    assert kb.kan_layer_forward_packed(g, f32, 0, 4, 4, 0, 0, 0, 0) == kb.KAN_OK


def test_check_maps_codes_to_exceptions():
    kb.check(kb.KAN_OK)
    with pytest.raises(ValueError):
        kb.check(kb.KAN_ERR_INVALID_ARG)
    with pytest.raises(NotImplementedError):
        kb.check(kb.KAN_ERR_UNSUPPORTED)
    with pytest.raises(kb.KanError):
        kb.check(kb.KAN_ERR_DEVICE)


def test_torch_wrappers_reject_host_tensors():
    import torch
    x = torch.zeros(4, 3)
    with pytest.raises(ValueError):
        kb.basis(x, 5)
    with pytest.raises(ValueError):
        kb.layer_forward(x, torch.zeros(2, 3, 8), torch.zeros(2, 3), 5)


def test_product_path_does_not_touch_the_oracle():
    """The binding and the HIP sources never import, load or name the oracle."""
    pkg = os.path.join(ROOT, "paper_2609_01956_amd")
    for dirpath, _, files in os.walk(pkg):
        for fn in files:
            if fn.endswith((".py", ".hip", ".cpp", ".h")):
                text = open(os.path.join(dirpath, fn)).read()
                assert "oracle" not in text.lower(), os.path.join(dirpath, fn)


def test_noalloc_entry_point_host_checks():
    """kan_layer_forward_noalloc rejects, on the host and before any HIP call,
    the same invalid arguments as kan_layer_forward, and a layer whose packed
    weights exceed its fixed 16 MiB scratch with KAN_ERR_SCRATCH_LIMIT."""
    f32, bad = kb.KAN_F32, kb.KAN_ERR_INVALID_ARG
    g = kb.make_grid(10)
    assert kb.kan_layer_forward_noalloc(g, f32, -1, 4, 4, X, C, W, Y) == bad
    assert kb.kan_layer_forward_noalloc(g, f32, 16, 4, 4, 0, C, W, Y) == bad
    assert kb.kan_layer_forward_noalloc(g, f32, 16, 4, 4, X, C, W, X + 8) == bad
    assert kb.kan_layer_forward_noalloc(kb.make_grid(10, spline_order=0), f32, 16, 4, 4, X, C, W,
                                        Y) == kb.KAN_ERR_UNSUPPORTED
    assert kb.kan_layer_forward_noalloc(g, f32, 0, 4, 4, 0, 0, 0, 0) == kb.KAN_OK
    # 256 -> 128 at G = 200 in fp32: 26.7 MB of packed weights
    g200 = kb.make_grid(200)
    assert kb.kan_layer_packed_bytes(g200, f32, 256, 128)[1] > kb.KAN_NOALLOC_SCRATCH_BYTES
    assert kb.kan_layer_forward_noalloc(g200, f32, 16, 256, 128, X, C, W, Y) == \
        kb.KAN_ERR_SCRATCH_LIMIT
    # the largest configured layers fit: 784 -> 256 at G = 10, 128 -> 128 at G = 200
    for G, n_in, n_out in [(10, 784, 256), (200, 128, 128)]:
        for dt in (kb.KAN_F32, kb.KAN_BF16):
            assert kb.kan_layer_packed_bytes(kb.make_grid(G), dt, n_in, n_out)[1] <= \
                kb.KAN_NOALLOC_SCRATCH_BYTES
    with pytest.raises(ValueError):
        kb.check(kb.KAN_ERR_SCRATCH_LIMIT)


def test_backward_host_checks():
    """kan_layer_backward rejects invalid arguments on the host, before any
    HIP call (fake addresses, never dereferenced)."""
    g = kb.make_grid(10)
    f32, bad = kb.KAN_F32, kb.KAN_ERR_INVALID_ARG
    DY, DX, DC, DW = 0x800000000, 0x900000000, 0xA00000000, 0xB00000000
    st, need = kb.kan_layer_backward_workspace_bytes(g, f32, 16, 4, 4)
    assert st == kb.KAN_OK and need > 0
    call = lambda *a: kb.kan_layer_backward(g, f32, 16, 4, 4, *a)
    assert call(X, C, W, 0, DX, DC, DW, WS, need) == bad               # no dy
    assert call(X, C, W, DY, DX, DC, 0, WS, need) == bad               # one weight gradient only
    assert call(X, C, W, DY, DX, 0, DW, WS, need) == bad
    assert call(X, C, W, DY, 0, 0, 0, WS, need) == bad                 # nothing requested
    assert call(X, 0, W, DY, DX, DC, DW, WS, need) == bad              # dx needs the weights
    assert call(X, C, W, DY, DX, DC, DW, WS, need - 1) == bad          # short workspace
    assert call(X, C, W, DY, DX, DC, DW, WS + 8, need) == bad          # misaligned workspace
    assert call(X, C, W, DY, DX + 2, DC, DW, WS, need) == bad          # misaligned dx
    assert call(X, C, W, DY, X + 16, DC, DW, WS, need) == bad          # dx over x
    assert call(X, C, W, DY, DX, DY, DW, WS, need) == bad              # dcoef over dy
    assert call(X, C, W, DY, DX, DC, DC + 16, WS, need) == bad         # outputs overlapping
    assert call(X, C, W, DY, DX, DC, DW, DX - 16, need) == bad         # workspace over dx
    assert kb.kan_layer_backward(g, f32, -1, 4, 4, X, C, W, DY, DX, DC, DW, WS, need) == bad
    # the backward is cubic only
    for k in (1, 2, 4, 7):
        assert kb.kan_layer_backward(kb.make_grid(10, spline_order=k), f32, 16, 4, 4, X, C, W, DY,
                                     DX, DC, DW, WS, need) == kb.KAN_ERR_UNSUPPORTED
        assert kb.kan_layer_backward_workspace_bytes(kb.make_grid(10, spline_order=k), f32, 16,
                                                     4, 4)[0] == kb.KAN_ERR_UNSUPPORTED
    # an empty batch needing only dx: nothing to do
    assert kb.kan_layer_backward(g, f32, 0, 4, 4, 0, C, W, 0, DX, 0, 0, WS, need) == kb.KAN_OK
    lib = kb.load_library()
    assert lib.kan_layer_backward_workspace_bytes(ctypes.byref(g), 0, 16, 4, 4, None) == bad
    assert kb.kan_layer_backward_workspace_bytes(g, f32, -1, 4, 4)[0] == bad


@pytest.mark.parametrize("G,n_in,n_out,B,bf16", [(10, 784, 256, 65536, True),
                                                 (10, 784, 256, 65536, False),
                                                 (200, 128, 128, 8192, False),
                                                 (5, 2, 5, 1024, False)])
def test_backward_workspace_bytes(G, n_in, n_out, B, bf16):
    """The workspace holds the packed weights of the dx contraction, dy
    transposed (padded to 32 outputs and 32 rows) and the fp32 partial weight
    gradients of at most 256 batch splits' worth of workgroups."""
    dt = kb.KAN_BF16 if bf16 else kb.KAN_F32
    st, n = kb.kan_layer_backward_workspace_bytes(kb.make_grid(G), dt, B, n_in, n_out)
    assert st == kb.KAN_OK
    es = 2 if bf16 else 4
    out32 = -(-n_out // 32) * 32
    bpad = -(-B // 32) * 32
    assert n >= out32 * bpad * es
    cp = 16 if G + 4 <= 16 else 32 * -(-(G + 4) // 32)
    kr = 32 * ((n_in + 1) // 2 if cp == 16 else n_in * cp // 32)
    assert n >= kr * n_out * es  # packed weights
    assert n < out32 * bpad * es + 300 * out32 * kr * 4 + kr * 256 * 4 + (1 << 20)


def test_backward_workspace_holds_the_narrow_dx_table():
    """Layers of at most 16 outputs take dx on the vector-ALU kernel from
    16384 rows on; its weight table [in rounded up to 8][G + 7 rounded down
    to even][out rounded up to even, then to a multiple of 4] (fp32 weights,
    or bf16 weights in pairs) takes the place of the packed weights (for
    256 -> 10 at G = 10, 256 x 16 x 12 elements: 192 KiB in fp32, within the
    256 KiB of packed fp32 weights; 96 KiB in bf16, within their 128 KiB), and
    only when a feature's table (columns x row elements) fits 256."""
    g = kb.make_grid(10)
    for dt in (kb.KAN_BF16, kb.KAN_F32):
        st, small = kb.kan_layer_backward_workspace_bytes(g, dt, 16383, 256, 10)
        st2, big = kb.kan_layer_backward_workspace_bytes(g, dt, 16384, 256, 10)
        assert st == st2 == kb.KAN_OK
        es = 2 if dt == kb.KAN_BF16 else 4
        grow = big - small  # the new row's share of dy^T and x^T, plus the table
        table = 256 * 16 * 12 * es
        packed = 128 * (1 if dt == kb.KAN_BF16 else 2) * 1024
        assert table < packed
        assert grow < 4096 * es, (dt, grow)
    # 17 outputs, or a grid whose table rows pass 256 floats: the MFMA kernel
    for n_out, G in [(17, 10), (16, 12)]:
        a = kb.kan_layer_backward_workspace_bytes(kb.make_grid(G), kb.KAN_BF16, 16383, 256, n_out)[1]
        b = kb.kan_layer_backward_workspace_bytes(kb.make_grid(G), kb.KAN_BF16, 16384, 256, n_out)[1]
        assert b - a < 8192


@pytest.mark.parametrize("k", [1, 2, 4, 5, 6, 7])
def test_other_degrees_accepted(k):
    """Degrees 1..7 (eq. general_truncated): G + k bases; the fused layer runs
    one workgroup shape (the run-time degree build), never the structured-sparse
    instruction, and a forced other shape is rejected."""
    g = kb.make_grid(10, spline_order=k)
    assert kb.kan_basis_eval(g, kb.KAN_F32, X, 0, PHI) == kb.KAN_OK
    for dt in (kb.KAN_F32, kb.KAN_BF16):
        st, plan = kb.kan_layer_plan(g, dt, 65536, 784, 256)
        assert st == kb.KAN_OK and plan == (1, 1, 4, 1, 0, 1)
        assert kb.kan_layer_plan(g, dt, 65536, 784, 256, "2,1")[0] == kb.KAN_ERR_INVALID_ARG
        st, n = kb.kan_layer_packed_bytes(g, dt, 5, 7)
        assert st == kb.KAN_OK
        kj = 8 if dt == kb.KAN_BF16 else 2
        assert n % (2 * 32 * kj * (2 if dt == kb.KAN_BF16 else 4)) == 0


def test_cdb_basis_host_checks():
    g = kb.make_grid(10)
    f32, bad = kb.KAN_F32, kb.KAN_ERR_INVALID_ARG
    assert kb.kan_basis_eval_cdb(g, f32, X, -1, PHI) == bad
    assert kb.kan_basis_eval_cdb(g, f32, 0, 16, PHI) == bad
    assert kb.kan_basis_eval_cdb(g, f32, X + 2, 16, PHI) == bad
    assert kb.kan_basis_eval_cdb(g, f32, X, 16, X + 32) == bad
    assert kb.kan_basis_eval_cdb(kb.make_grid(10, spline_order=8), f32, X, 16, PHI) == \
        kb.KAN_ERR_UNSUPPORTED
    assert kb.kan_basis_eval_cdb(g, f32, 0, 0, 0) == kb.KAN_OK


def test_span_forward_host_checks():
    """kan_layer_forward_span rejects invalid arguments on the host (fake
    addresses, never dereferenced) and grids too wide for its LDS tile."""
    g = kb.make_grid(100)
    f32, bad = kb.KAN_F32, kb.KAN_ERR_INVALID_ARG
    WS = 0xC00000000
    st, need = kb.kan_layer_forward_span_workspace_bytes(g, f32, 300, 13, 45)
    assert st == kb.KAN_OK and need > 0
    call = lambda *a: kb.kan_layer_forward_span(g, f32, 300, 13, 45, *a)
    assert call(X, C, W, WS, need - 1, Y) == bad            # short workspace
    assert call(X, C, W, 0, need, Y) == bad                 # no workspace
    assert call(X, C, W, WS + 8, need, Y) == bad            # misaligned workspace
    assert call(X, C, W, Y - 16, need, Y) == bad            # workspace over y
    assert call(X, C, W, WS, need, X + 16) == bad           # y over x
    assert call(X, 0, W, WS, need, Y) == bad                # no coefficients
    assert call(X + 2, C, W, WS, need, Y) == bad            # misaligned x
    assert kb.kan_layer_forward_span(g, f32, -1, 13, 45, X, C, W, WS, need, Y) == bad
    assert kb.kan_layer_forward_span(g, f32, 0, 13, 45, 0, 0, 0, 0, 0, 0) == kb.KAN_OK
    # G + k + 1 = 512 columns fit one feature's weight tile, 513 do not
    assert kb.kan_layer_forward_span_workspace_bytes(kb.make_grid(508), f32, 16, 3, 40)[0] == \
        kb.KAN_OK
    wide = kb.make_grid(509)
    assert kb.kan_layer_forward_span_workspace_bytes(wide, f32, 16, 3, 40)[0] == \
        kb.KAN_ERR_UNSUPPORTED
    assert kb.kan_layer_forward_span(wide, f32, 16, 3, 40, X, C, W, WS, 1 << 30, Y) == \
        kb.KAN_ERR_UNSUPPORTED
    assert kb.kan_layer_forward_span_workspace_bytes(kb.make_grid(10, spline_order=7), f32, 16,
                                                     3, 40)[0] == kb.KAN_OK


@pytest.mark.parametrize("G,n_in,n_out,B", [(50, 128, 128, 8192), (200, 128, 128, 8192),
                                            (100, 13, 45, 300), (5, 2, 5, 1024)])
def test_span_workspace_bytes(G, n_in, n_out, B):
    """The workspace holds the fp32 weights transposed per feature and padded
    to the output tile (16, 32 or 64), plus fp32 partial sums for at most 512
    feature splits when the row blocks do not fill the chip."""
    for dt in (kb.KAN_F32, kb.KAN_BF16):
        st, n = kb.kan_layer_forward_span_workspace_bytes(kb.make_grid(G), dt, B, n_in, n_out)
        assert st == kb.KAN_OK
        w = n_in * (G + 4) * n_out * 4
        assert w <= n <= n_in * (G + 4) * (n_out + 63) * 4 + 512 * B * n_out * 4 + 512


def test_packed_forward_workspace_host_checks():
    """kan_layer_forward_packed's workspace (the split contraction's partial
    sums of small batches): the size query, and a workspace that would be
    used is checked for alignment and overlap on the host."""
    g = kb.make_grid(10)
    f32, bad = kb.KAN_F32, kb.KAN_ERR_INVALID_ARG
    P, WS = 0x600000000, 0x700000000
    pk = kb.kan_layer_packed_bytes(g, f32, 784, 64)[1]
    st, need = kb.kan_layer_forward_packed_workspace_bytes(g, f32, 256, 784, 64)
    st2, plan = kb.kan_layer_plan(g, f32, 256, 784, 64)
    assert st == st2 == kb.KAN_OK and plan[5] > 1
    assert need == -(-plan[5] * 256 * 64 * 4 // 256) * 256
    # no split for a full batch, nor for an empty one
    assert kb.kan_layer_forward_packed_workspace_bytes(g, f32, 65536, 784, 64) == (kb.KAN_OK, 0)
    assert kb.kan_layer_forward_packed_workspace_bytes(g, f32, 0, 784, 64) == (kb.KAN_OK, 0)
    assert kb.kan_layer_forward_packed_workspace_bytes(g, f32, -1, 784, 64)[0] == bad
    lib = kb.load_library()
    assert lib.kan_layer_forward_packed_workspace_bytes(ctypes.byref(g), 0, 256, 784, 64, None,
                                                        None) == bad
    call = lambda ws, nb, y=Y: kb.kan_layer_forward_packed(g, f32, 256, 784, 64, X, P, pk, y,
                                                           workspace=ws, workspace_bytes=nb)
    assert call(WS + 8, need) == bad                  # misaligned, would be used
    assert call(X - 16, need) == bad                  # over x
    assert call(P + 64, need) == bad                  # over the packed weights
    assert call(Y - 16, need) == bad                  # over y
