"""GPU parity of kan_basis_eval against the float64 oracle (truncated power +
clamp), called through the C ABI.  Tolerances: basis max-abs <= 1e-6 in fp32,
partition-of-unity error <= 1e-5 for G up to 200, exact zeros off support."""
import numpy as np
import pytest

import oracle
from paper_2609_01956_amd import binding as kb
from paper_2609_01956_amd import workloads as wl
from gpu_common import (F32_BASIS_TOL, PU_TOL, device, say, to_dev, to_host64, torch)

pytestmark = pytest.mark.gpu


def _edge_points(G, lo=-1.0, hi=1.0):
    t = oracle.knots(G, lo, hi).astype(np.float32)
    ups = np.nextafter(t, np.float32(np.inf))
    downs = np.nextafter(t, np.float32(-np.inf))
    mids = ((t[:-1].astype(np.float64) + t[1:]) / 2).astype(np.float32)
    extra = np.array([0.0, -0.0, lo, hi, 4.0, -4.0, 1e4, -1e4, 3.9999, -3.9999], dtype=np.float32)
    return np.concatenate([t, ups, downs, mids, extra]).astype(np.float32)


def _off_support(x, G, lo=-1.0, hi=1.0):
    """[n, G+3] mask of inputs strictly outside basis j's support.  (The
    oracle's literal five-term sum cancels to exactly 0 within ~1e-14 of the
    support's right end, so exact zeros are located from the knots instead.)"""
    t = oracle.knots(G, lo, hi)
    xd = np.asarray(x, np.float64)[:, None]
    margin = 1e-12 * (hi - lo)
    return (xd < t[None, :G + 3] - margin) | (xd > t[None, 4:G + 7] + margin)


def _run_basis(x32: np.ndarray, G: int, dtype=None):
    dtype = dtype or torch.float32
    xt = to_dev(x32, dtype)
    phi = kb.basis(xt, G)
    torch.cuda.synchronize()
    return phi


@pytest.mark.parametrize("G", [1, 2, 3, 5, 10, 32, 50, 64, 100, 200, 1000])
def test_basis_f32_matches_oracle(G):
    rng = np.random.default_rng(100 + G)
    x = np.concatenate([rng.uniform(-1.6, 1.6, 20011).astype(np.float32), _edge_points(G)])
    say(f"basis f32 G={G} n={x.size}")
    phi = to_host64(_run_basis(x, G))
    ref = oracle.basis_tp(x.astype(np.float64), G)
    err = np.abs(phi - ref)
    assert err.max() <= F32_BASIS_TOL, (G, err.max())
    # the clamp makes every value off the support [t_j, t_{j+4}] exactly zero
    assert np.all(phi[_off_support(x, G)] == 0.0)


@pytest.mark.parametrize("G", [5, 10, 32, 50, 64, 100, 200])
def test_partition_of_unity(G):
    x = np.concatenate([np.linspace(-1, 1, 2001, dtype=np.float32),
                        np.random.default_rng(G).uniform(-1, 1, 100000).astype(np.float32)])
    say(f"basis PU G={G}")
    phi = _run_basis(x, G).to(torch.float64)
    pu = float((phi.sum(dim=1) - 1.0).abs().max())
    assert pu <= PU_TOL, (G, pu)


@pytest.mark.parametrize("G", [5, 10, 100])
def test_basis_bf16_matches_oracle(G):
    rng = np.random.default_rng(7 + G)
    x = wl.round_to_bf16_f32(np.concatenate([rng.uniform(-1.5, 1.5, 9999).astype(np.float32),
                                              _edge_points(G)]))
    say(f"basis bf16 G={G}")
    phi = to_host64(_run_basis(x, G, torch.bfloat16))
    ref = oracle.basis_tp(x.astype(np.float64), G)
    # one bf16 rounding of a value within 1e-6 of the reference
    assert np.all(np.abs(phi - ref) <= 2.0 ** -8 * np.abs(ref) + 2e-6)
    assert np.all(phi[_off_support(x, G)] == 0.0)


def test_basis_special_values():
    x = np.array([np.nan, np.inf, -np.inf, 1e30, -1e30, 0.25], dtype=np.float32)
    say("basis special values")
    phi = to_host64(_run_basis(x, 5))
    assert np.all(np.isnan(phi[0]))
    assert np.all(phi[1:5] == 0.0)
    np.testing.assert_allclose(phi[5], oracle.basis_tp(np.array([0.25]), 5)[0], atol=F32_BASIS_TOL)


@pytest.mark.parametrize("n", [1, 2, 7, 255, 256, 257, 4097])
@pytest.mark.parametrize("dtype_name", ["f32", "bf16"])
def test_basis_ragged_unaligned_and_guarded(n, dtype_name):
    """Odd lengths, an output that starts one element past a 16-byte boundary
    (scalar store path) and canaries on both sides of the output."""
    dtype = torch.float32 if dtype_name == "f32" else torch.bfloat16
    G = 10
    nb = G + 3
    x = wl.round_to_bf16_f32(np.random.default_rng(n).uniform(-1.3, 1.3, n).astype(np.float32))
    ref = oracle.basis_tp(x.astype(np.float64), G)
    say(f"basis ragged n={n} {dtype_name}")
    xt = to_dev(x, dtype)
    for offset in (0, 1):
        buf = torch.full((n * nb + 64,), 7.0, dtype=dtype, device=device())
        out = buf[offset:offset + n * nb].view(n, nb)
        kb.basis(xt, G, out=out)
        torch.cuda.synchronize()
        got = to_host64(out)
        tol = F32_BASIS_TOL if dtype == torch.float32 else None
        if tol is not None:
            assert np.abs(got - ref).max() <= tol
        else:
            assert np.all(np.abs(got - ref) <= 2.0 ** -8 * np.abs(ref) + 2e-6)
        b = to_host64(buf)
        assert np.all(b[:offset] == 7.0) and np.all(b[offset + n * nb:] == 7.0)


def test_basis_empty():
    say("basis empty")
    phi = kb.basis(torch.empty(0, device=device()), 5)
    torch.cuda.synchronize()
    assert phi.shape == (0, 8)


@pytest.mark.parametrize("dtype_name", ["f32", "bf16"])
def test_basis_full_size_mlp_input_sampled(dtype_name):
    """The 65536 x 784 input of the 3-layer MLP workload (G = 10) at full size:
    sampled elements against the oracle, partition of unity over every
    in-grid element, exact zeros over every off-support element count."""
    dtype = torch.float32 if dtype_name == "f32" else torch.bfloat16
    W = wl.make_workload("c5_mlp_784_256_256_10_g10")
    x = W["x"] if dtype == torch.float32 else wl.round_to_bf16_f32(W["x"])
    G = W["G"]
    say(f"basis full-size 65536x784 G={G} {dtype_name}")
    xt = to_dev(x, dtype)
    phi = kb.basis(xt, G)
    torch.cuda.synchronize()
    flat = phi.view(-1, G + 3)
    rng = np.random.default_rng(5)
    idx = np.unique(np.concatenate([rng.integers(0, x.size, 20000),
                                    np.arange(784 * 3), [x.size - 1]]))
    got = to_host64(flat[torch.from_numpy(idx).to(device())])
    ref = oracle.basis_tp(x.reshape(-1)[idx].astype(np.float64), G)
    if dtype == torch.float32:
        assert np.abs(got - ref).max() <= F32_BASIS_TOL
    else:
        assert np.all(np.abs(got - ref) <= 2.0 ** -8 * np.abs(ref) + 2e-6)
    pu = (flat.to(torch.float32).sum(dim=1, dtype=torch.float64) - 1.0).abs().max()
    tol = PU_TOL if dtype == torch.float32 else 4 * 2.0 ** -8
    assert float(pu) <= tol
