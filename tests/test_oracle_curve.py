"""Pins of the accuracy-curve extrapolation oracle (oracle/curve.py): the
non-negative least-squares solver against its optimality conditions, exact
solutions and an independent library routine (scipy.optimize.nnls); the curve
fit against noiseless curves of known parameters; the cost extrapolation
against its closed form."""
import numpy as np
import pytest

from oracle import curve


def _kkt(A, b, x, tol=1e-9):
    """Karush-Kuhn-Tucker conditions of min ||Ax - b||, x >= 0: x >= 0; the
    negative gradient w = A^T (b - Ax) is <= 0 everywhere and 0 where x > 0."""
    w = A.T @ (b - A @ x)
    scale = np.abs(A.T @ b).max() + 1e-300
    assert np.all(x >= 0)
    assert np.all(w <= tol * scale), w
    assert np.all(np.abs(w[x > 0]) <= tol * scale), w


@pytest.mark.parametrize("m,n,seed", [(8, 4, 0), (20, 6, 1), (5, 8, 2), (40, 3, 3), (3, 3, 4)])
def test_nnls_satisfies_kkt(m, n, seed):
    rng = np.random.default_rng(seed)
    A = rng.standard_normal((m, n))
    b = rng.standard_normal(m)
    x, r = curve.nnls(A, b)
    _kkt(A, b, x)
    assert abs(r - np.linalg.norm(A @ x - b)) < 1e-12


@pytest.mark.parametrize("seed", range(6))
def test_nnls_matches_scipy(seed):
    from scipy.optimize import nnls as scipy_nnls
    rng = np.random.default_rng(100 + seed)
    m, n = rng.integers(3, 30), rng.integers(1, 10)
    A = rng.standard_normal((m, n))
    b = rng.standard_normal(m)
    x, r = curve.nnls(A, b)
    xs, rs = scipy_nnls(A, b)
    assert abs(r - rs) <= 1e-10 * max(1.0, rs)
    np.testing.assert_allclose(x, xs, atol=1e-9)


def test_nnls_recovers_exact_nonnegative_solution():
    rng = np.random.default_rng(7)
    A = rng.standard_normal((12, 5))
    xt = np.array([0.0, 1.5, 0.0, 2.25, 0.5])
    x, r = curve.nnls(A, A @ xt)
    np.testing.assert_allclose(x, xt, atol=1e-10)
    assert r < 1e-10


def test_nnls_zero_when_every_direction_increases_the_residual():
    A = np.eye(3)
    x, r = curve.nnls(A, np.array([-1.0, -2.0, -0.5]))
    assert np.all(x == 0)
    assert abs(r - np.linalg.norm([1.0, 2.0, 0.5])) < 1e-12


@pytest.mark.parametrize("b0,b1,b2", [(8.0, 2.0, 0.1), (2.0, 1.25, 0.05), (20.0, 1.05, 0.3)])
def test_curve_recovers_noiseless_optimus_curve(b0, b1, b2):
    """Points of e(x) = 1 / (b0 x + b1) + b2 at the passes of a 5-epoch run on
    10% of the window: the fit returns the parameters and predicts the error
    at 10 full passes."""
    xs = 0.1 * np.arange(1, 6)
    acc = 1.0 - (1.0 / (b0 * xs + b1) + b2)
    c = curve.fit_accuracy_curve(xs, acc)
    assert c.rss < 1e-16
    np.testing.assert_allclose([c.b0, c.b1, c.b2], [b0, b1, b2], rtol=1e-5, atol=1e-8)
    np.testing.assert_allclose(c.accuracy(10.0), 1.0 - (1.0 / (10 * b0 + b1) + b2), atol=1e-8)


def test_curve_is_monotone_and_bounded_on_noisy_points():
    rng = np.random.default_rng(3)
    xs = 0.05 * np.arange(1, 6)
    acc = 1.0 - (1.0 / (10 * xs + 1.5) + 0.12) + 0.01 * rng.standard_normal(5)
    c = curve.fit_accuracy_curve(xs, acc)
    grid = np.linspace(0.01, 20, 200)
    a = c.accuracy(grid)
    assert np.all(np.diff(a) >= -1e-15) and np.all((a >= 0) & (a <= 1))
    assert min(c.b0, c.b1, c.b2) >= 0
    # the fit is at least as good as the best constant
    assert c.rss <= np.sum((acc - acc.mean()) ** 2) + 1e-15


def test_curve_with_a_perfect_point_reaches_full_accuracy():
    c = curve.fit_accuracy_curve([0.1, 0.2, 0.3], [0.5, 0.9, 1.0])
    assert c.b2 == 0.0
    assert c.accuracy(100.0) > 0.99


def test_extrapolate_cost_scales_by_steps_and_epochs():
    """Per-epoch cost is deterministic (section 4.3): 200 of 4000 frames at
    batch 64 is 4 steps an epoch, the whole window 63; 10 epochs."""
    c, acc, sec = curve.extrapolate([0.4, 0.6], [0.002, 0.0022], 200, 4000, 64, 10)
    assert abs(sec - 0.0021 * 63 / 4 * 10) < 1e-12
    assert abs(acc - float(c.accuracy(10.0))) < 1e-15
    assert 0.0 <= acc <= 1.0
