"""Pins of the oracle's MLP mapper (Sec. 4.4, Appendix F).

With every ReLU input positive the network is the affine map x W1 W2 W3 +
(b1 W2 W3 + b2 W3 + b3), so it must equal the (separately pinned) ridge-form
map with that W and b, RoPE handling included; with the first layer dead it
returns the last bias (rotated by the target RoPE for keys); and a ReLU that
cuts a pre-activation is checked on a small hand-built case."""

import math

import numpy as np
import pytest

from oracle import kvx_oracle as O


def _mlp(rng, L_t, H, kd, F, d, b1_shift=0.0):
    return (rng.standard_normal((L_t, H, kd, F)) / math.sqrt(kd),
            rng.standard_normal((L_t, H, F)) + b1_shift,
            rng.standard_normal((L_t, H, F, F)) / math.sqrt(F),
            rng.standard_normal((L_t, H, F)) + b1_shift,
            rng.standard_normal((L_t, H, F, d)) / math.sqrt(F),
            rng.standard_normal((L_t, H, d)))


def _inputs(seed, L_s=4, L_t=2, H=2, T=9, d=8, k=2, style=0):
    rng = np.random.default_rng(seed)
    src = rng.standard_normal((L_s, 2, H, T, d))
    idx = np.stack([rng.choice(L_s, k, replace=False) for _ in range(L_t)])
    pos = rng.integers(0, 40000, size=T)
    return rng, src, idx, pos, O.Rope(1e4, style=style), O.Rope(1e6, style=style)


@pytest.mark.parametrize("style", [0, 1])
def test_all_positive_reduces_to_the_affine_map(style):
    rng, src, idx, pos, rs, rt = _inputs(1, style=style)
    L_t, H, d, k, F = 2, 2, 8, 2, 16
    # large positive biases and a non-negative middle layer keep every
    # pre-activation positive
    def positive(m):
        W1, b1, W2, b2, W3, b3 = m
        return W1, b1, np.abs(W2), b2, W3, b3
    mK = positive(_mlp(rng, L_t, H, k * d, F, d, b1_shift=50.0))
    mV = positive(_mlp(rng, L_t, H, k * d, F, d, b1_shift=50.0))
    got = O.mlp_map_cache(src, idx, mK, mV, rs, rt, pos)

    def affine(m):
        W1, b1, W2, b2, W3, b3 = m
        W = W1 @ W2 @ W3
        b = np.einsum("lhf,lhfd->lhd", np.einsum("lhf,lhfg->lhg", b1, W2), W3) \
            + np.einsum("lhf,lhfd->lhd", b2, W3) + b3
        return W, b
    WK, bK = affine(mK)
    WV, bV = affine(mV)
    want = O.map_cache(src, idx, WK, WV, bK, bV, rs, rt, pos)
    np.testing.assert_allclose(got, want, rtol=1e-10, atol=1e-9)


def test_dead_first_layer_returns_the_last_bias():
    rng, src, idx, pos, rs, rt = _inputs(2)
    L_t, H, d, k, F = 2, 2, 8, 2, 16
    mK, mV = _mlp(rng, L_t, H, k * d, F, d, b1_shift=-80.0), _mlp(rng, L_t, H, k * d, F, d, b1_shift=-80.0)
    got = O.mlp_map_cache(src, idx, mK, mV, rs, rt, pos)
    T = src.shape[3]
    for l in range(L_t):
        for h in range(H):
            np.testing.assert_allclose(got[l, 1, h], np.broadcast_to(mV[5][l, h], (T, d)), atol=1e-12)
            want_k = O.rope_rotate(np.broadcast_to(mK[5][l, h], (T, d)), pos, rt)
            np.testing.assert_allclose(got[l, 0, h], want_k, atol=1e-12)


def test_relu_cut_by_hand():
    """One token, one head, k = 1, d = 2, F = 2 with hand-picked weights; values
    (no rotation): x = (1, -2).  Layer 1: pre = x W1 + b1 = (1*1 + -2*0 + 0,
    1*0 + -2*1 + 0.5) = (1, -1.5) -> ReLU (1, 0).  Layer 2: (1, 0) W2 + b2 =
    (2, -3) + (0, 1) = (2, -2) -> ReLU (2, 0).  Layer 3: (2, 0) W3 + b3 =
    (2*3, 2*-1) + (0.25, 0) = (6.25, -2)."""
    src = np.zeros((1, 2, 1, 1, 2))
    src[0, 1, 0, 0] = [1.0, -2.0]
    one = lambda a: np.asarray(a, dtype=np.float64)[None, None]
    m = (one([[1.0, 0.0], [0.0, 1.0]]), one([0.0, 0.5]), one([[2.0, -3.0], [5.0, 7.0]]),
         one([0.0, 1.0]), one([[3.0, -1.0], [11.0, 13.0]]), one([0.25, 0.0]))
    zero = tuple(np.zeros_like(t) for t in m)
    got = O.mlp_map_cache(src, np.array([[0]]), zero, m, O.Rope(1e4), O.Rope(1e4), np.array([5]))
    np.testing.assert_allclose(got[0, 1, 0, 0], [6.25, -2.0], atol=1e-15)
