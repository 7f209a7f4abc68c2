"""GPU parity of kan_basis_eval_cdb (the Cox-de Boor recursion of eq. cdb0 /
eq. cdbk over every knot interval) against the float64 oracle's Cox-de Boor
route and against the truncated-power kernel, through the C ABI: max-abs
<= 1e-6 in fp32, the same exact zeros off support, NaN and infinities as
kan_basis_eval."""
import numpy as np
import pytest

import oracle
from paper_2609_01956_amd import binding as kb
from paper_2609_01956_amd import workloads as wl
from gpu_common import F32_BASIS_TOL, say, to_dev, to_host64, torch

pytestmark = pytest.mark.gpu


def _points(G, k, n=20000, seed=0):
    rng = np.random.default_rng(seed)
    h = 2.0 / G
    t = oracle.knots(G, k=k).astype(np.float32)
    x = rng.uniform(-1 - (k + 1.5) * h, 1 + (k + 1.5) * h, n).astype(np.float32)
    return np.concatenate([x, t, np.nextafter(t, np.float32(np.inf)),
                           np.nextafter(t, np.float32(-np.inf))]).astype(np.float32)


# G + 2k intervals: up to 16 and 32 in registers, the wider ones in LDS rows
@pytest.mark.parametrize("k,G", [(3, 5), (3, 10), (3, 26), (3, 50), (3, 200), (1, 10), (2, 20),
                                 (4, 8), (5, 40), (7, 12)])
def test_cdb_matches_oracle_and_truncated_power(k, G):
    x = _points(G, k, seed=G + k)
    say(f"basis cdb k={k} G={G}")
    xt = to_dev(x, torch.float32)
    cdb = to_host64(kb.basis(xt, G, spline_order=k, method="cdb"))
    tp = to_host64(kb.basis(xt, G, spline_order=k))
    torch.cuda.synchronize()
    ref = oracle.basis_cdb(x, G, k=k)
    assert np.abs(cdb - ref).max() <= F32_BASIS_TOL, np.abs(cdb - ref).max()
    assert np.abs(cdb - tp).max() <= 2 * F32_BASIS_TOL
    # off every support exactly 0, beyond the rounding of the coordinate that
    # picks the interval (one fp32 rounding at the magnitude G + 2k, in units
    # of h)
    t = oracle.knots(G, k=k)
    xd = x.astype(np.float64)[:, None]
    m = 4 * 2.0 ** -24 * (G + 2 * k) * (2.0 / G)
    off = (xd < t[None, :G + k] - m) | (xd > t[None, k + 1:G + 2 * k + 1] + m)
    assert np.all(cdb[off] == 0.0)


def test_cdb_nan_inf_and_bf16():
    G = 10
    x = np.array([np.nan, np.inf, -np.inf, 0.25, -0.7], np.float32)
    say("basis cdb nan/inf")
    got = to_host64(kb.basis(to_dev(x, torch.float32), G, method="cdb"))
    torch.cuda.synchronize()
    assert np.all(np.isnan(got[0])) and np.all(got[1:3] == 0.0)
    np.testing.assert_allclose(got[3:], oracle.basis_cdb(x[3:], G), atol=F32_BASIS_TOL)
    # bf16 storage: the values rounded to bf16
    xb = wl.round_to_bf16_f32(np.random.default_rng(1).uniform(-1.3, 1.3, 5000).astype(np.float32))
    got = to_host64(kb.basis(to_dev(xb, torch.bfloat16), G, method="cdb"))
    torch.cuda.synchronize()
    ref = oracle.basis_cdb(xb, G)
    assert np.abs(got - ref).max() <= 2.0 ** -8 * 0.7 + 1e-6
