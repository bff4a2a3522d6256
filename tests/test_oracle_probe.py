"""Pins of the oracle's single-source probe and top-k selection (Sec. 2.3,
Eq. single_source_ols; Sec. 3.2).

ols_r2 is checked against scikit-learn's least squares and its
variance-weighted R^2, against the squared Pearson correlation for one
regressor and one response, and against exact and independent cases;
probe_r2 against planted layer-to-layer maps with different RoPE on the two
sides; select_topk against a brute-force ranking with ties."""

import math

import numpy as np
import pytest

from oracle import kvx_oracle as O


def test_ols_r2_matches_sklearn():
    lm = pytest.importorskip("sklearn.linear_model")
    met = pytest.importorskip("sklearn.metrics")
    rng = np.random.default_rng(1)
    X = rng.standard_normal((300, 6)) + 2.0
    Y = X @ rng.standard_normal((6, 4)) + rng.standard_normal((300, 4)) * [0.5, 1.0, 2.0, 4.0]
    pred = lm.LinearRegression().fit(X, Y).predict(X)
    want = met.r2_score(Y, pred, multioutput="variance_weighted")
    assert abs(O.ols_r2(X, Y) - want) < 1e-12


def test_ols_r2_one_regressor_is_squared_correlation():
    rng = np.random.default_rng(2)
    x = rng.standard_normal(500)
    y = 0.6 * x + rng.standard_normal(500)
    r = np.corrcoef(x, y)[0, 1]
    assert abs(O.ols_r2(x[:, None], y[:, None]) - r * r) < 1e-12


def test_ols_r2_exact_and_independent():
    rng = np.random.default_rng(3)
    X = rng.standard_normal((400, 5))
    assert abs(O.ols_r2(X, X @ rng.standard_normal((5, 3)) + 7.0) - 1.0) < 1e-12
    # independent response: R^2 is the fraction p / (N - 1) on average
    vals = [O.ols_r2(X, rng.standard_normal((400, 3))) for _ in range(200)]
    assert abs(np.mean(vals) - 5 / 399) < 0.004


@pytest.mark.parametrize("style", [0, 1])
def test_probe_finds_planted_layer_maps(style):
    """Target layer l is made from source layer s(l) by an invertible linear map
    in the stripped (content) space plus noise elsewhere: R2 is 1 exactly at
    (s(l), l) for keys and values and below 1 elsewhere."""
    rng = np.random.default_rng(4)
    L_s, L_t, H, N, d = 4, 3, 2, 90, 8
    rs, rt = O.Rope(1e4, style=style), O.Rope(1e6, style=style)
    pos = rng.integers(0, 20000, size=N)
    src = rng.standard_normal((L_s, 2, H, N, d))
    tgt = np.zeros((L_t, 2, H, N, d))
    planted = [2, 0, 3]
    for l, s in enumerate(planted):
        for h in range(H):
            M = rng.standard_normal((d, d)) + 3 * np.eye(d)
            content = O.rope_rotate(src[s, 0, h], pos, rs, inverse=True) @ M + 0.5
            tgt[l, 0, h] = O.rope_rotate(content, pos, rt)
            tgt[l, 1, h] = src[s, 1, h] @ M - 1.0
    r2 = O.probe_r2(src, tgt, rs, rt, pos)
    assert r2.shape == (L_s, L_t, H, 2)
    for l, s in enumerate(planted):
        np.testing.assert_allclose(r2[s, l], 1.0, atol=1e-12)
        others = [t for t in range(L_s) if t != s]
        assert (r2[others, l] < 0.9).all()
    np.testing.assert_array_equal(O.select_topk(r2, 1)[:, 0], planted)


def test_select_topk_brute_force_and_ties():
    rng = np.random.default_rng(5)
    r2 = rng.uniform(-0.2, 1.0, size=(7, 5, 3, 2))
    got = O.select_topk(r2, 3)
    for l in range(5):
        score = [r2[s, l].mean() for s in range(7)]
        best = sorted(range(7), key=lambda s: score[s], reverse=True)[:3]
        assert list(got[l]) == sorted(best)
    # equal scores: the lower source index wins
    r2 = np.zeros((6, 2, 1, 2))
    r2[[1, 4], 0] = 0.5
    r2[[2, 5], 0] = 0.3
    assert list(O.select_topk(r2, 3)[0]) == [1, 2, 4]
    assert list(O.select_topk(r2, 2)[1]) == [0, 1]      # all equal: lowest indices
