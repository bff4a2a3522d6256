"""Pins of the oracle's ridge fit (Eq. Wstar with centring, Sec. 3.1).

The map's weights come from this closed form.  It is checked by exact
recovery of a planted affine map, by its normal equations, by convergence to
ordinary least squares as lambda -> 0, by the textbook expected-error formula
of OLS, and by agreement of the Cholesky and SVD routes.
"""

import numpy as np
import pytest

from oracle import kvx_oracle as O


def _planted(seed, N=400, p=12, q=5, noise=0.0):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((N, p)) * rng.uniform(0.5, 2.0, size=p) + rng.standard_normal(p)
    W = rng.standard_normal((p, q))
    b = rng.standard_normal(q)
    Y = X @ W + b + noise * rng.standard_normal((N, q))
    return X, Y, W, b


@pytest.mark.parametrize("fit", [O.ridge_fit, O.ridge_fit_svd])
def test_noise_free_recovery(fit):
    X, Y, W, b = _planted(0)
    Wh, bh = fit(X, Y, lam=0.0)
    np.testing.assert_allclose(Wh, W, atol=1e-10)
    np.testing.assert_allclose(bh, b, atol=1e-10)


def test_normal_equations_hold():
    """(Xc^T Xc + lam I) W = Xc^T Yc and the residual of the centred fit has zero mean."""
    X, Y, _, _ = _planted(1, noise=0.3)
    lam = 0.7
    W, b = O.ridge_fit(X, Y, lam)
    Xc, Yc = X - X.mean(0), Y - Y.mean(0)
    np.testing.assert_allclose(Xc.T @ (Yc - Xc @ W), lam * W, atol=1e-9)
    np.testing.assert_allclose((Y - X @ W - b).mean(0), 0.0, atol=1e-12)


def test_cholesky_and_svd_routes_agree():
    X, Y, _, _ = _planted(2, noise=0.5)
    for lam in (0.0, 0.01, 10.0):
        W1, b1 = O.ridge_fit(X, Y, lam)
        W2, b2 = O.ridge_fit_svd(X, Y, lam)
        np.testing.assert_allclose(W1, W2, atol=1e-10)
        np.testing.assert_allclose(b1, b2, atol=1e-10)


def test_lambda_to_zero_tends_to_least_squares_linearly():
    X, Y, _, _ = _planted(3, noise=0.5)
    A = np.column_stack([X, np.ones(len(X))])
    sol = np.linalg.lstsq(A, Y, rcond=None)[0]
    W0, b0 = sol[:-1], sol[-1]
    gaps = []
    for lam in (1.0, 1e-2, 1e-4, 1e-6):
        W, b = O.ridge_fit(X, Y, lam)
        gaps.append(np.linalg.norm(W - W0) + np.linalg.norm(b - b0))
    ratios = [gaps[i] / gaps[i + 1] for i in range(len(gaps) - 1)]
    for r in ratios:
        assert 80 < r < 120          # gap shrinks in proportion to lambda
    assert gaps[-1] < 1e-6


def test_expected_error_matches_ols_formula():
    """At lambda = 0, E||W_hat - W||_F^2 = sigma^2 * q * tr((Xc^T Xc)^-1)."""
    rng = np.random.default_rng(4)
    N, p, q, sigma = 200, 6, 4, 0.3
    X = rng.standard_normal((N, p))
    W = rng.standard_normal((p, q))
    Xc = X - X.mean(0)
    want = sigma ** 2 * q * np.trace(np.linalg.inv(Xc.T @ Xc))
    errs = []
    for _ in range(400):
        Y = X @ W + 1.5 + sigma * rng.standard_normal((N, q))
        Wh, _ = O.ridge_fit(X, Y, 0.0)
        errs.append(np.sum((Wh - W) ** 2))
    assert abs(np.mean(errs) / want - 1.0) < 0.1


def test_ridge_shrinks_towards_zero():
    X, Y, _, _ = _planted(5, noise=0.5)
    norms = [np.linalg.norm(O.ridge_fit(X, Y, lam)[0]) for lam in (0.0, 10.0, 1e3, 1e5)]
    assert all(a > b for a, b in zip(norms, norms[1:]))
