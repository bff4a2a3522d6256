"""Pins of the oracle's whole-mapper fit (Sec. 3.1 Fitting, Sec. 3.3).

fit_cache builds every (target layer, head, K|V) design from the selected
source layers and fits it by ridge.  It is pinned by exact recovery of a
planted mapper pushed through the (separately pinned) map itself, with
different RoPE bases and layouts on the two sides, by the statistical error
of OLS under noise, and by the ridge shrinkage towards zero."""

import math

import numpy as np
import pytest

from oracle import kvx_oracle as O


def _planted(seed, L_s=5, L_t=3, H=2, N=80, d=8, k=2, style=0, th_s=1e4, th_t=1e4,
             factor=1.0):
    rng = np.random.default_rng(seed)
    src = rng.standard_normal((L_s, 2, H, N, d)) * rng.uniform(0.5, 2.0, size=d) + 0.3
    idx = np.stack([rng.choice(L_s, k, replace=False) for _ in range(L_t)])
    W_K = rng.standard_normal((L_t, H, k * d, d)) / math.sqrt(k * d)
    W_V = rng.standard_normal((L_t, H, k * d, d)) / math.sqrt(k * d)
    b_K = rng.standard_normal((L_t, H, d))
    b_V = rng.standard_normal((L_t, H, d))
    pos = rng.integers(0, 30000, size=N)
    rs = O.Rope(th_s, style=style, factor=factor)
    rt = O.Rope(th_t, style=style, factor=factor)
    return src, idx, (W_K, W_V, b_K, b_V), rs, rt, pos


@pytest.mark.parametrize("style", [0, 1])
@pytest.mark.parametrize("bases", [(1e4, 1e4), (1e4, 1e6), (5e5, 5e5)])
def test_recovers_a_planted_mapper(style, bases):
    """Target caches made by the map from a known mapper: the fit at lambda = 0
    returns that mapper (keys are fitted after stripping the target RoPE)."""
    src, idx, (W_K, W_V, b_K, b_V), rs, rt, pos = _planted(
        7, style=style, th_s=bases[0], th_t=bases[1], factor=8.0 if bases[0] == 5e5 else 1.0)
    tgt = O.map_cache(src, idx, W_K, W_V, b_K, b_V, rs, rt, pos)
    fK, fV, gK, gV = O.fit_cache(src, idx, tgt, rs, rt, pos, lam=0.0)
    for got, want in ((fK, W_K), (fV, W_V), (gK, b_K), (gV, b_V)):
        np.testing.assert_allclose(got, want, atol=1e-9)
    # and mapping with the fitted mapper reproduces the target caches
    again = O.map_cache(src, idx, fK, fV, gK, gV, rs, rt, pos)
    np.testing.assert_allclose(again, tgt, atol=1e-9)


def test_index_order_follows_the_lists():
    """Permuting a target layer's index list permutes the fitted row blocks."""
    src, idx, (W_K, W_V, b_K, b_V), rs, rt, pos = _planted(8, k=3, L_s=6)
    tgt = O.map_cache(src, idx, W_K, W_V, b_K, b_V, rs, rt, pos)
    perm = idx[:, ::-1].copy()
    fK, fV, _, _ = O.fit_cache(src, perm, tgt, rs, rt, pos, lam=0.0)
    d = src.shape[-1]
    rev = np.concatenate([np.arange(i * d, (i + 1) * d) for i in (2, 1, 0)])
    np.testing.assert_allclose(fK, W_K[:, :, rev, :], atol=1e-9)
    np.testing.assert_allclose(fV, W_V[:, :, rev, :], atol=1e-9)


def test_noise_error_matches_ols():
    """With Gaussian noise on the target values, the fitted map's error has the
    OLS expectation sigma^2 * d * tr((Xc^T Xc)^-1) (values: no rotations)."""
    rng = np.random.default_rng(9)
    src, idx, (W_K, W_V, b_K, b_V), rs, rt, pos = _planted(9, L_t=1, H=1, N=120, k=1)
    clean = O.map_cache(src, idx, W_K, W_V, b_K, b_V, rs, rt, pos)
    X = src[idx[0, 0], 1, 0]
    Xc = X - X.mean(0)
    d, sigma = X.shape[1], 0.2
    want = sigma ** 2 * d * np.trace(np.linalg.inv(Xc.T @ Xc))
    errs = []
    for _ in range(200):
        tgt = clean.copy()
        tgt[:, 1] += sigma * rng.standard_normal(tgt[:, 1].shape)
        _, fV, _, _ = O.fit_cache(src, idx, tgt, rs, rt, pos, lam=0.0)
        errs.append(np.sum((fV - W_V) ** 2))
    assert abs(np.mean(errs) / want - 1.0) < 0.15


def test_ridge_term_shrinks_the_fit():
    src, idx, (W_K, W_V, b_K, b_V), rs, rt, pos = _planted(10)
    tgt = O.map_cache(src, idx, W_K, W_V, b_K, b_V, rs, rt, pos)
    n0 = np.linalg.norm(O.fit_cache(src, idx, tgt, rs, rt, pos, lam=0.0)[1])
    n1 = np.linalg.norm(O.fit_cache(src, idx, tgt, rs, rt, pos, lam=1e3)[1])
    assert n1 < n0
