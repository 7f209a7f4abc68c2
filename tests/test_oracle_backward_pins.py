"""Pins of the oracle's backward (gradients of eq. kan_forward) against facts
fixed outside it, all on the CPU: hand-evaluated closed forms of the cubic
derivative (tests/golden/cubic_derivative_closed_form.txt), scipy's B-spline
derivatives for degrees 1..5, the derivative of the partition of unity,
central finite differences of the oracle's forward (a separate routine),
numpy matmuls of scipy basis values for dC and dWb, and a pure-Python brute
force on tiny inputs."""
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


def _scipy_elems(G, lo, hi, k, deriv=0):
    h = (hi - lo) / G
    t = lo + (np.arange(G + 2 * k + 1) - k) * h
    out = []
    for j in range(G + k):
        b = BSpline.basis_element(t[j:j + k + 2], extrapolate=False)
        out.append(b.derivative(deriv) if deriv else b)
    return out


def _scipy_matrix(x, elems):
    m = np.zeros((len(x), len(elems)))
    for j, b in enumerate(elems):
        m[:, j] = np.nan_to_num(b(x), nan=0.0)
    return m


def _off_knot_points(G, lo, hi, k, n=3000, seed=0):
    """Random points over the whole knot range and beyond, kept at least
    1e-6 h away from every knot (where a degree-1 derivative jumps)."""
    rng = np.random.default_rng(seed)
    h = (hi - lo) / G
    x = rng.uniform(lo - (k + 1.5) * h, hi + (k + 1.5) * h, n)
    frac = (x - lo) / h - np.floor((x - lo) / h)
    return x[(frac > 1e-6) & (frac < 1 - 1e-6)]


@pytest.mark.parametrize("G", [5, 10, 200])
def test_cubic_derivative_closed_forms(G):
    tab = _golden("cubic_derivative_closed_form.txt")
    lo, hi = -1.0, 1.0
    h = (hi - lo) / G
    t = oracle.knots(G, lo, hi)
    for j in [0, 1, G // 2, G + 2]:
        x = t[j] + tab[:, 0] * h
        got = oracle.basis_tp_deriv(x, G, lo, hi)[:, j]
        want = tab[:, 1] / tab[:, 2] / h
        np.testing.assert_allclose(got, want, rtol=0, atol=1e-12 / h)


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
@pytest.mark.parametrize("G,lo,hi", [(5, -1.0, 1.0), (12, -2.5, 0.5)])
def test_derivative_matches_scipy(k, G, lo, hi):
    x = _off_knot_points(G, lo, hi, k, seed=k + G)
    want = _scipy_matrix(x, _scipy_elems(G, lo, hi, k, deriv=1))
    got = oracle.basis_tp_deriv(x, G, lo, hi, k=k)
    h = (hi - lo) / G
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-10 / h)


@pytest.mark.parametrize("G", [5, 32, 200])
def test_derivative_of_partition_of_unity_vanishes(G):
    x = np.linspace(-1, 1, 2001)
    d = oracle.basis_tp_deriv(x, G)
    assert np.abs(d.sum(axis=1)).max() <= 1e-9 * G
    # and it is not trivially zero
    assert np.abs(d).max() > 0.1 * G


def test_derivative_zero_off_support_and_nan():
    G = 7
    t = oracle.knots(G)
    x = np.array([t[0] - 0.3, t[-1] + 0.3, -50.0, 50.0])
    assert np.all(oracle.basis_tp_deriv(x, G) == 0.0)
    assert np.all(np.isnan(oracle.basis_tp_deriv(np.array([np.nan]), G)))


def test_silu_derivative_matches_expit():
    x = np.concatenate([np.linspace(-30, 30, 6001), [0.0, 1e-8, -1e-8]])
    s = scipy.special.expit(x)
    np.testing.assert_allclose(oracle.silu_deriv(x), s * (1 + x * (1 - s)), rtol=1e-13,
                               atol=1e-15)


def _rand(B, n_in, n_out, G, seed, lo=-1.0, hi=1.0, spread=1.3):
    rng = np.random.default_rng(seed)
    x = rng.uniform(lo * spread, hi * spread, (B, n_in))
    C = rng.normal(0, 0.5, (n_out, n_in, G + 3))
    Wb = rng.normal(0, 0.5, (n_out, n_in))
    dy = rng.normal(0, 1.0, (B, n_out))
    return x, C, Wb, dy


def _loss(x, C, Wb, dy, G):
    return float(np.sum(dy * oracle.layer(x, C, Wb, G)))


def test_gradients_match_central_differences_of_the_forward():
    """L = sum(dy * layer(x, C, Wb)); each gradient entry against a central
    difference of the oracle's forward routine."""
    G = 6
    x, C, Wb, dy = _rand(5, 3, 4, G, seed=3)
    dx, dC, dW = oracle.layer_backward(x, C, Wb, dy, G)
    e = 1e-6
    for idx in np.ndindex(*x.shape):
        xp, xm = x.copy(), x.copy()
        xp[idx] += e
        xm[idx] -= e
        fd = (_loss(xp, C, Wb, dy, G) - _loss(xm, C, Wb, dy, G)) / (2 * e)
        assert abs(fd - dx[idx]) <= 1e-6 * max(1.0, abs(fd)), (idx, fd, dx[idx])
    for idx in list(np.ndindex(*C.shape))[::5]:
        Cp, Cm = C.copy(), C.copy()
        Cp[idx] += e
        Cm[idx] -= e
        fd = (_loss(x, Cp, Wb, dy, G) - _loss(x, Cm, Wb, dy, G)) / (2 * e)
        assert abs(fd - dC[idx]) <= 1e-7 * max(1.0, abs(fd)), (idx, fd, dC[idx])
    for idx in np.ndindex(*Wb.shape):
        Wp, Wm = Wb.copy(), Wb.copy()
        Wp[idx] += e
        Wm[idx] -= e
        fd = (_loss(x, C, Wp, dy, G) - _loss(x, C, Wm, dy, G)) / (2 * e)
        assert abs(fd - dW[idx]) <= 1e-7 * max(1.0, abs(fd)), (idx, fd, dW[idx])


def test_weight_gradients_are_matmuls_of_scipy_values():
    """dC = dy^T Phi(x) and dWb = dy^T silu(x): numpy matmuls of scipy's basis
    values and scipy's expit."""
    G, lo, hi = 10, -1.0, 1.0
    x, C, Wb, dy = _rand(200, 5, 7, G, seed=8)
    dx, dC, dW = oracle.layer_backward(x, C, Wb, dy, G, lo, hi)
    elems = _scipy_elems(G, lo, hi, 3)
    for i in range(x.shape[1]):
        phi = _scipy_matrix(x[:, i], elems)
        np.testing.assert_allclose(dC[:, i, :], dy.T @ phi, rtol=1e-11, atol=1e-12)
    silu = x * scipy.special.expit(x)
    np.testing.assert_allclose(dW, dy.T @ silu, rtol=1e-11, atol=1e-12)


def test_input_gradient_brute_force_tiny():
    """dx from scalar Python loops over scipy's derivative elements and
    math.exp, on a 2 x 2 -> 3 layer."""
    G, lo, hi = 5, -1.0, 1.0
    x, C, Wb, dy = _rand(2, 2, 3, G, seed=21)
    dx, _, _ = oracle.layer_backward(x, C, Wb, dy, G, lo, hi)
    der = _scipy_elems(G, lo, hi, 3, deriv=1)
    for b in range(2):
        for i in range(2):
            v = float(x[b, i])
            s = 1.0 / (1.0 + math.exp(-v))
            sd = s + v * s * (1.0 - s)
            tot = 0.0
            for o in range(3):
                t = sum(float(C[o, i, j]) * float(np.nan_to_num(der[j](v), nan=0.0))
                        for j in range(G + 3))
                tot += float(dy[b, o]) * (t + float(Wb[o, i]) * sd)
            assert abs(tot - dx[b, i]) <= 1e-12 * max(1.0, abs(tot))


def test_backward_special_cases():
    """C = 1, Wb = 0: dx = sum_o dy (the derivative of the partition of unity
    is 0, so dx = 0 on the grid); C = 0: dx = sigma'(x) (dy Wb)."""
    G = 8
    x, C, Wb, dy = _rand(50, 4, 3, G, seed=5, spread=0.99)
    dx, _, _ = oracle.layer_backward(x, np.ones_like(C), np.zeros_like(Wb), dy, G)
    assert np.abs(dx).max() <= 1e-10
    dx, dC, dW = oracle.layer_backward(x, np.zeros_like(C), Wb, dy, G)
    np.testing.assert_allclose(dx, oracle.silu_deriv(x) * (dy @ Wb), rtol=1e-12, atol=1e-13)
    # the weight gradients do not depend on the weights
    _, dC2, dW2 = oracle.layer_backward(x, C, Wb, dy, G)
    np.testing.assert_array_equal(dC, dC2)
    np.testing.assert_array_equal(dW, dW2)
