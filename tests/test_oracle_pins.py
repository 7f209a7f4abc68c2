"""Pins of the float64 oracle against facts fixed outside it.

Every test here runs on the CPU.  None re-types the oracle's own formula:
each compares it with a value the paper prints (golden files under
tests/golden/, each citing its passage), a library routine (scipy's B-spline
basis elements, numpy matmul, scipy's expit, torch's bfloat16 conversion), a
closed form, an invariant of B-splines, or a second independent route.
"""
import math
import os

import numpy as np
import pytest
import scipy.special
from scipy.interpolate import BSpline

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append([float(v) for v in line.split()])
    return np.array(rows)


def _scipy_basis(x, G, lo, hi, k=3):
    """Basis matrix [len(x), G+k] from scipy's B-spline basis elements on the
    knots t_j = lo + (j - k) h (the grid convention under test)."""
    h = (hi - lo) / G
    t = lo + (np.arange(G + 2 * k + 1) - k) * h
    out = np.zeros((len(x), G + k))
    for j in range(G + k):
        b = BSpline.basis_element(t[j:j + k + 2], extrapolate=False)
        v = b(x)
        out[:, j] = np.nan_to_num(v, nan=0.0)
    return out


def _test_points(G, lo, hi, n=2000, seed=0):
    rng = np.random.default_rng(seed)
    h = (hi - lo) / G
    t = lo + (np.arange(G + 7) - 3) * h
    pts = [rng.uniform(lo - 4 * h, hi + 4 * h, n), t, t + 1e-9 * h, t - 1e-9 * h,
           (t[:-1] + t[1:]) / 2, [lo, hi, 0.0]]
    return np.concatenate([np.asarray(p, dtype=np.float64) for p in pts])


# ------------------------------------------------------------------ knots

@pytest.mark.parametrize("G,lo,hi", [(5, -1.0, 1.0), (10, -3.0, 3.0), (200, -1.0, 1.0), (7, 0.25, 2.0)])
def test_knots_grid_convention(G, lo, hi):
    t = oracle.knots(G, lo, hi)
    assert t.shape == (G + 7,)
    h = (hi - lo) / G
    assert t[3] == pytest.approx(lo, abs=1e-15)
    assert t[G + 3] == pytest.approx(hi, abs=1e-13)
    np.testing.assert_allclose(np.diff(t), h, rtol=1e-12)


# ----------------------------------------------------- closed forms (paper)

@pytest.mark.parametrize("route", ["tp", "cdb", "seg"])
@pytest.mark.parametrize("G", [5, 10, 200])
def test_closed_form_values(route, G):
    """N(u) at integer and half-integer u equals the values of eq. truncated."""
    tab = _golden("cubic_closed_form.txt")
    lo, hi = -1.0, 1.0
    h = (hi - lo) / G
    t = oracle.knots(G, lo, hi)
    fn = {"tp": oracle.basis_tp, "cdb": oracle.basis_cdb, "seg": oracle.basis_seg}[route]
    for j in [0, 1, G // 2, G + 2]:
        x = t[j] + tab[:, 0] * h
        got = fn(x, G, lo, hi)[:, j]
        want = tab[:, 1] / tab[:, 2]
        np.testing.assert_allclose(got, want, atol=1e-12, rtol=0)


def test_segment_values_match_paper_matrix():
    """On every knot span the four nonzero TP and Cox-de Boor bases equal
    [1 tau tau^2 tau^3] M_B-spline with the matrix printed in eq. bspline_matrix."""
    M = _golden("bspline_matrix.txt") / 6.0
    G, lo, hi = 9, -1.0, 1.0
    h = (hi - lo) / G
    t = oracle.knots(G, lo, hi)
    rng = np.random.default_rng(1)
    for m in range(3, G + 3):  # spans inside [lo, hi)
        tau = rng.uniform(0, 1, 64)
        x = t[m] + tau * h
        T = np.stack([np.ones_like(tau), tau, tau ** 2, tau ** 3], axis=1)
        want = T @ M  # columns: N_{m-3}, N_{m-2}, N_{m-1}, N_m
        for fn in (oracle.basis_tp, oracle.basis_cdb, oracle.basis_seg):
            phi = fn(x, G, lo, hi)
            np.testing.assert_allclose(phi[:, m - 3:m + 1], want, atol=1e-13, rtol=0)
            others = np.delete(phi, np.arange(m - 3, m + 1), axis=1)
            assert np.all(np.abs(others) < 1e-14)


# ------------------------------------------------------ library routine pin

@pytest.mark.parametrize("G,lo,hi", [(1, -1.0, 1.0), (2, -1.0, 1.0), (5, -1.0, 1.0),
                                     (10, -3.0, 3.0), (50, -1.0, 1.0), (13, 0.5, 4.0)])
@pytest.mark.parametrize("route", ["tp", "cdb", "seg"])
def test_cubic_basis_matches_scipy(G, lo, hi, route):
    x = _test_points(G, lo, hi, n=600)
    # scipy's basis element is closed at the right end of its support; the
    # value there is 0 in every convention, so compare away from the far end.
    want = _scipy_basis(x, G, lo, hi)
    fn = {"tp": oracle.basis_tp, "cdb": oracle.basis_cdb, "seg": oracle.basis_seg}[route]
    got = fn(x, G, lo, hi)
    np.testing.assert_allclose(got, want, atol=1e-12, rtol=0)


@pytest.mark.parametrize("k", [1, 2, 4, 5])
@pytest.mark.parametrize("route", ["tp", "cdb"])
def test_general_degree_matches_scipy(k, route):
    """eq. general_truncated (any degree, clamp to [0, k+1]) and eq. cdbk."""
    G, lo, hi = 6, -1.0, 1.0
    x = _test_points(G, lo, hi, n=400, seed=k)
    want = _scipy_basis(x, G, lo, hi, k=k)
    fn = oracle.basis_tp if route == "tp" else oracle.basis_cdb
    got = fn(x, G, lo, hi, k=k)
    np.testing.assert_allclose(got, want, atol=1e-11, rtol=0)


# ---------------------------------------------------------- three routes

@pytest.mark.parametrize("G", [1, 5, 10, 50, 100, 200])
def test_routes_agree(G):
    """TP + clamp, Cox-de Boor and the segment form compute one function."""
    lo, hi = -1.0, 1.0
    x = _test_points(G, lo, hi, n=3000, seed=G)
    a = oracle.basis_tp(x, G, lo, hi)
    b = oracle.basis_cdb(x, G, lo, hi)
    c = oracle.basis_seg(x, G, lo, hi)
    np.testing.assert_allclose(a, b, atol=1e-13, rtol=0)
    np.testing.assert_allclose(a, c, atol=1e-13, rtol=0)


# -------------------------------------------------------------- invariants

@pytest.mark.parametrize("G", [1, 5, 10, 32, 64, 100, 200])
def test_partition_of_unity_and_support(G):
    lo, hi = -1.0, 1.0
    h = (hi - lo) / G
    t = oracle.knots(G, lo, hi)
    x_in = np.concatenate([np.linspace(lo, hi, 2001),
                           np.random.default_rng(G).uniform(lo, hi, 5000)])
    phi = oracle.basis_tp(x_in, G, lo, hi)
    assert np.max(np.abs(phi.sum(1) - 1.0)) < 1e-13
    # nonnegative up to the cancellation of five terms of size <= 64 near u = 4
    assert np.all(phi >= -64 * 8 * np.finfo(float).eps)
    # strictly partial sum between t_0 and lo, and exactly zero beyond t_0
    x_left = np.linspace(t[0] + 1e-3 * h, lo - 1e-3 * h, 101)
    assert np.all(oracle.basis_tp(x_left, G, lo, hi).sum(1) < 1.0)
    x_far = np.array([t[0] - 1e-9, t[0] - h, t[-1], t[-1] + h, 1e4, -1e4, np.inf, -np.inf])
    assert np.all(oracle.basis_tp(x_far, G, lo, hi) == 0.0)
    assert np.all(oracle.basis_cdb(x_far[np.isfinite(x_far)], G, lo, hi) == 0.0)
    # every basis is exactly zero off [t_j, t_{j+4}] (the clamp, eq. bounded)
    x = _test_points(G, lo, hi, n=1000)
    phi = oracle.basis_tp(x, G, lo, hi)
    for j in range(G + 3):
        off = (x < t[j]) | (x > t[j + 4])
        assert np.all(phi[off, j] == 0.0)


@pytest.mark.parametrize("G", [5, 50])
def test_symmetry(G):
    """N(u) = N(4 - u): the stencil {1, -4, 6, -4, 1} is symmetric."""
    lo, hi = -1.0, 1.0
    h = (hi - lo) / G
    t = oracle.knots(G, lo, hi)
    u = np.random.default_rng(3).uniform(-1, 5, 500)
    j = G // 2
    a = oracle.basis_tp(t[j] + u * h, G, lo, hi)[:, j]
    b = oracle.basis_tp(t[j] + (4 - u) * h, G, lo, hi)[:, j]
    np.testing.assert_allclose(a, b, atol=1e-13, rtol=0)


def test_c2_continuity_at_knots():
    """Cubic B-splines on simple knots are C^2 across interior knots (Sec. 2,
    Step 3): one-sided difference quotients of N, N', N'' agree at each knot,
    while the third derivative jumps."""
    G, lo, hi = 5, -1.0, 1.0
    h = (hi - lo) / G
    t = oracle.knots(G, lo, hi)
    j = 3
    d = 1e-4 * h

    def derivs(x0, side):
        # value and first three derivatives from one side by polynomial fit
        s = side * d * np.arange(1, 7)
        vals = oracle.basis_tp(x0 + s, G, lo, hi)[:, j]
        coef = np.polyfit(s, vals, 3)
        return coef[3], coef[2], 2 * coef[1], 6 * coef[0]

    for m in range(j + 1, j + 4):
        L = derivs(t[m], -1)
        R = derivs(t[m], +1)
        assert abs(L[0] - R[0]) < 1e-9
        assert abs(L[1] - R[1]) < 1e-5 / h
        assert abs(L[2] - R[2]) < 1e-3 / h ** 2
        assert abs(L[3] - R[3]) > 0.5 / h ** 3  # the cubic pieces differ


@pytest.mark.parametrize("G,lo,hi", [(5, -1.0, 1.0), (10, -3.0, 3.0), (100, -1.0, 1.0)])
def test_linear_precision(G, lo, hi):
    """Greville abscissae xi_j = (t_{j+1} + t_{j+2} + t_{j+3}) / 3 reproduce x
    on [lo, hi] (textbook B-spline property, de Boor)."""
    t = oracle.knots(G, lo, hi)
    xi = (t[1:G + 4] + t[2:G + 5] + t[3:G + 6]) / 3.0
    x = np.random.default_rng(5).uniform(lo, hi, 3000)
    phi = oracle.basis_tp(x, G, lo, hi)
    np.testing.assert_allclose(phi @ xi, x, atol=1e-12 * max(1.0, abs(lo), abs(hi)), rtol=0)


def test_cardinal_spline_is_fourfold_box_convolution():
    """The uniform cubic B-spline is the 4-fold convolution of the unit box
    (independent definition, evaluated numerically on a fine grid)."""
    n = 2000
    step = 1.0 / n
    box = np.ones(n)
    conv = box
    for _ in range(3):
        conv = np.convolve(conv, box) * step
    # conv[m] approximates M(u) at u = (m + 2) * step (midpoint offsets of 4 boxes)
    u = (np.arange(conv.size) + 2.0) * step
    sel = slice(0, conv.size, 97)
    G, lo, hi = 5, -1.0, 1.0
    h = (hi - lo) / G
    t = oracle.knots(G, lo, hi)
    got = oracle.basis_tp(t[2] + u[sel] * h, G, lo, hi)[:, 2]
    np.testing.assert_allclose(got, conv[sel], atol=5e-3)


def test_unclamped_form_cancels_off_support():
    """Without the clamp the five truncated powers still sum to zero beyond the
    support (a dropped or mis-signed term would leave a cubic there); in double
    the cancellation residual stays near eps * u^3."""
    G, lo, hi = 5, -1.0, 1.0
    h = (hi - lo) / G
    t = oracle.knots(G, lo, hi)
    u = np.linspace(4.0, 12.0, 81)
    v = oracle.basis_tp(t[0] + u * h, G, lo, hi, clamp=False)[:, 0]
    assert np.all(np.abs(v) <= 64 * np.finfo(float).eps * u ** 3)
    u_in = np.random.default_rng(7).uniform(0, 4, 500)
    a = oracle.basis_tp(t[0] + u_in * h, G, lo, hi, clamp=False)[:, 0]
    b = oracle.basis_tp(t[0] + u_in * h, G, lo, hi, clamp=True)[:, 0]
    np.testing.assert_allclose(a, b, atol=1e-13, rtol=0)


def test_nan_propagates():
    x = np.array([0.1, np.nan, -0.3])
    for fn in (oracle.basis_tp, oracle.basis_cdb, oracle.basis_seg):
        phi = fn(x, 5, -1.0, 1.0)
        assert np.all(np.isnan(phi[1])) and not np.any(np.isnan(phi[[0, 2]]))


# ---------------------------------------------------- fp32 stability table

def test_table2_order_of_magnitude_with_fp32_emulation():
    """A float32 evaluation of the literal five-term sum on the oracle's knots
    reproduces the magnitudes of Table 2 (a check of the knot convention, not a
    parity target): unclamped out-of-support residual within 2x, clamped PU
    error within 3x, unclamped PU error within 5x."""
    tab = _golden("table2_stability.txt")
    f32 = np.float32
    for G, oos_nc, pu_nc, _oos_c, pu_c in tab:
        G = int(G)
        t = oracle.knots(G).astype(f32)
        h = f32(f32(2.0) / f32(G))
        x = np.linspace(-1, 1, 2001).astype(f32)
        tt = oracle.knots(G)

        def ev(clamp):
            u = ((x[:, None] - t[None, :G + 3]) / h).astype(f32)
            if clamp:
                u = np.clip(u, f32(0), f32(4))

            def c3(z):
                z = np.maximum(z, f32(0))
                return z * z * z
            return ((c3(u) - f32(4) * c3(u - f32(1)) + f32(6) * c3(u - f32(2))
                     - f32(4) * c3(u - f32(3)) + c3(u - f32(4))) / f32(6)).astype(f32)

        off = (x[:, None].astype(float) < tt[None, :G + 3]) | (x[:, None].astype(float) > tt[None, 4:G + 7])
        Nn, Nc = ev(False), ev(True)
        pu_c_e = np.abs(Nc.astype(float).sum(1) - 1).max()
        assert pu_c / 3 <= pu_c_e <= pu_c * 3, (G, pu_c_e)
        if not np.isnan(oos_nc):
            oos_e = np.abs(Nn[off]).max()
            pu_e = np.abs(Nn.astype(float).sum(1) - 1).max()
            assert oos_nc / 2 <= oos_e <= oos_nc * 2, (G, oos_e)
            assert pu_nc / 5 <= pu_e <= pu_nc * 5, (G, pu_e)


# ------------------------------------------------------------------- layer

def test_silu_matches_scipy():
    x = np.concatenate([np.linspace(-30, 30, 601), [0.0, -0.0]])
    np.testing.assert_allclose(oracle.silu(x), x * scipy.special.expit(x), rtol=1e-15, atol=1e-300)


def _rand_layer(B, n_in, n_out, G, seed=0, lo=-1.0, hi=1.0):
    rng = np.random.default_rng(seed)
    x = rng.uniform(lo, hi, (B, n_in))
    C = rng.normal(0, 0.3, (n_out, n_in, G + 3))
    Wb = rng.normal(0, 0.5, (n_out, n_in))
    return x, C, Wb


def test_layer_partition_of_unity_gives_fan_in():
    x, C, Wb = _rand_layer(33, 7, 5, 10)
    y = oracle.layer(x, np.ones_like(C), np.zeros_like(Wb), 10)
    np.testing.assert_allclose(y, 7.0, atol=1e-12)


def test_layer_linear_precision_sums_inputs():
    G, lo, hi = 10, -1.0, 1.0
    x, C, Wb = _rand_layer(40, 6, 3, G)
    t = oracle.knots(G, lo, hi)
    xi = (t[1:G + 4] + t[2:G + 5] + t[3:G + 6]) / 3.0
    Cg = np.broadcast_to(xi, C.shape).copy()
    y = oracle.layer(x, Cg, np.zeros_like(Wb), G, lo, hi)
    np.testing.assert_allclose(y, np.repeat(x.sum(1, keepdims=True), 3, axis=1), atol=1e-12)


def test_layer_base_branch_matches_matmul():
    x, C, Wb = _rand_layer(50, 9, 4, 5)
    x = x * 3.0  # include off-grid values: the spline branch is zero-weighted anyway
    y = oracle.layer(x, np.zeros_like(C), Wb, 5)
    want = (x * scipy.special.expit(x)) @ Wb.T
    np.testing.assert_allclose(y, want, rtol=1e-13, atol=1e-13)


def test_layer_one_hot_coefficients_select_single_basis():
    G, lo, hi = 5, -1.0, 1.0
    B, n_in, n_out = 20, 3, 8
    x, _, _ = _rand_layer(B, n_in, n_out, G, seed=9)
    C = np.zeros((n_out, n_in, G + 3))
    for o in range(n_out):
        C[o, :, o] = 1.0  # output o sums basis j = o over the inputs
    y = oracle.layer(x, C, np.zeros((n_out, n_in)), G, lo, hi)
    sc = _scipy_basis(x.ravel(), G, lo, hi).reshape(B, n_in, G + 3)
    np.testing.assert_allclose(y, sc.sum(1)[:, :n_out], atol=1e-12)


def test_layer_brute_force_tiny():
    """Pure-Python loops over scipy basis values and math.exp, B<=3, in<=2, out<=2."""
    G, lo, hi = 5, -1.0, 1.0
    for seed, (B, n_in, n_out) in enumerate([(1, 1, 1), (3, 2, 2), (2, 1, 2), (3, 2, 1)]):
        x, C, Wb = _rand_layer(B, n_in, n_out, G, seed=seed, lo=-1.6, hi=1.6)
        want = np.zeros((B, n_out))
        for b in range(B):
            for o in range(n_out):
                s = 0.0
                for i in range(n_in):
                    xv = float(x[b, i])
                    row = _scipy_basis(np.array([xv]), G, lo, hi)[0]
                    for j in range(G + 3):
                        s += float(C[o, i, j]) * float(row[j])
                    s += float(Wb[o, i]) * xv / (1.0 + math.exp(-xv))
                want[b, o] = s
        for route in ("tp", "cdb"):
            got = oracle.layer(x, C, Wb, G, lo, hi, basis=route)
            np.testing.assert_allclose(got, want, atol=1e-12, rtol=1e-12)


def test_layer_transposed_operands_are_caught():
    """Shapes that only fit when C or Wb is transposed are rejected, and a
    non-square layer distinguishes [out, in] from [in, out]."""
    x, C, Wb = _rand_layer(4, 3, 2, 5)
    with pytest.raises(ValueError):
        oracle.layer(x, C.transpose(1, 0, 2), Wb, 5)
    with pytest.raises(ValueError):
        oracle.layer(x, C, Wb.T, 5)


# -------------------------------------------------------------------- bf16

def test_round_bf16_matches_torch_and_ties_to_even():
    import torch
    rng = np.random.default_rng(11)
    v = np.concatenate([rng.normal(0, 1, 20000), rng.normal(0, 1e-30, 200),
                        rng.normal(0, 1e30, 200), [0.0, -0.0, 1e-40, -3e38, 3.4e38]]).astype(np.float32)
    want = torch.from_numpy(v).to(torch.bfloat16).to(torch.float64).numpy()
    got = oracle.round_bf16(v.astype(np.float64))
    np.testing.assert_array_equal(got, want)
    # exact ties: 1 + 2^-8 lies halfway between 1 and 1 + 2^-7 -> even (1);
    # 1 + 3*2^-8 lies halfway between 1 + 2^-7 and 1 + 2^-6 -> even (1 + 2^-6)
    got = oracle.round_bf16(np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, 1 + 2 ** -8 + 2 ** -30]))
    np.testing.assert_array_equal(got, [1.0, 1 + 2 ** -6, 1 + 2 ** -7])
    assert np.isnan(oracle.round_bf16(np.array([np.nan]))[0])
    assert np.isinf(oracle.round_bf16(np.array([1e39]))[0])


def test_mlp_chains_layers_and_rounds_storage():
    G = 5
    x, C1, W1 = _rand_layer(16, 4, 3, G, seed=1)
    _, C2, W2 = _rand_layer(16, 3, 2, G, seed=2)
    y = oracle.mlp(x, [(C1, W1), (C2, W2)], G)
    want = oracle.layer(oracle.layer(x, C1, W1, G), C2, W2, G)
    np.testing.assert_array_equal(y, want)
    yb = oracle.mlp(x, [(C1, W1), (C2, W2)], G, bf16=True)
    r = oracle.round_bf16
    h1 = r(oracle.layer(r(x), r(C1), r(W1), G))
    np.testing.assert_array_equal(yb, r(oracle.layer(h1, r(C2), r(W2), G)))


def test_mlp_matches_pure_python_chain():
    """A two-layer chain evaluated in pure Python: scalar loops over scipy's
    B-spline basis elements, math.exp for SiLU, and, in bf16 mode, torch's
    bfloat16 conversion of the input, the weights and each layer's output (the
    storage of eq. kan_forward's tensors in bf16).  None of the oracle's
    routines takes part."""
    import torch
    G, lo, hi = 5, -1.0, 1.0
    rng = np.random.default_rng(31)
    x = rng.uniform(-1.3, 1.3, (3, 3))
    C1 = rng.normal(0, 0.5, (2, 3, G + 3))
    W1 = rng.normal(0, 0.7, (2, 3))
    C2 = rng.normal(0, 0.5, (2, 2, G + 3))
    W2 = rng.normal(0, 0.7, (2, 2))
    h = (hi - lo) / G
    t = [lo + (j - 3) * h for j in range(G + 7)]
    elems = [BSpline.basis_element(t[j:j + 5], extrapolate=False) for j in range(G + 3)]

    def bf(v):
        return float(torch.tensor(v, dtype=torch.float64).to(torch.bfloat16).to(torch.float64))

    def layer(xs, C, Wb, rnd):
        out = []
        for row in xs:
            ys = []
            for o in range(len(Wb)):
                acc = 0.0
                for i, v in enumerate(row):
                    for j in range(G + 3):
                        b = float(elems[j](v))
                        acc += rnd(C[o][i][j]) * (0.0 if math.isnan(b) else b)
                    acc += rnd(Wb[o][i]) * v / (1.0 + math.exp(-v))
                ys.append(rnd(acc))
            out.append(ys)
        return out

    for bf16, rnd in [(False, float), (True, bf)]:
        xs = [[rnd(v) for v in row] for row in x.tolist()]
        want = layer(layer(xs, C1.tolist(), W1.tolist(), rnd), C2.tolist(), W2.tolist(), rnd)
        got = oracle.mlp(x, [(C1, W1), (C2, W2)], G, lo, hi, bf16=bf16)
        if bf16:
            # the same bf16 values (a double sum differing in its last bit could
            # only move a value lying within 1e-16 of a rounding tie)
            np.testing.assert_allclose(got, want, rtol=2 ** -8, atol=0)
            assert np.mean(got == np.array(want)) == 1.0
        else:
            np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-14)


def test_layer_bf16_operands_matches_rounded_matmul():
    """bf16-operand mode equals numpy matmuls of bf16-rounded scipy basis values
    and SiLU values, and the rounding agrees with torch's bfloat16 conversion."""
    import torch
    G = 10
    x, C, Wb = _rand_layer(37, 5, 6, G, seed=12, lo=-1.5, hi=1.5)
    y = oracle.layer(x, C, Wb, G, bf16_operands=True)
    phi = _scipy_basis(x.ravel(), G, -1.0, 1.0).reshape(37, 5, G + 3)
    want = (oracle.round_bf16(phi).reshape(37, -1) @ C.reshape(6, -1).T
            + oracle.round_bf16(x * scipy.special.expit(x)) @ Wb.T)
    np.testing.assert_allclose(y, want, rtol=1e-12, atol=1e-12)
    v = phi.astype(np.float32).astype(np.float64)
    tb = torch.from_numpy(v.astype(np.float32)).to(torch.bfloat16).double().numpy()
    np.testing.assert_array_equal(oracle.round_bf16(v), tb)
    assert not np.allclose(y, oracle.layer(x, C, Wb, G), rtol=1e-6, atol=0)
