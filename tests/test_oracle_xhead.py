"""Pins of the oracle's cross-head map (Sec. 3.2 features with Eq. ridge_kv).

The cross-head form is checked against the per-head form (itself pinned in
test_oracle_map.py) through its block-diagonal special case, against a
selection map whose answer is a stored source head, against a dense-matrix
evaluation with explicitly built rotation matrices, against the reordering
of source heads, and against a scalar-loop evaluation that decodes every
feature index on its own.
"""

import math

import numpy as np
import pytest

from oracle import kvx_oracle as O


def _problem(seed, L_s=5, L_t=3, H_s=3, H_t=2, T=6, d_s=8, d_t=8, k=2, bias=True, style=0,
             th_s=1e4, th_t=1e4):
    rng = np.random.default_rng(seed)
    F = k * H_s * d_s
    return dict(
        src_kv=rng.standard_normal((L_s, 2, H_s, T, d_s)),
        idx=np.stack([rng.choice(L_s, k, replace=False) for _ in range(L_t)]),
        W_K=rng.standard_normal((L_t, H_t, F, d_t)) / math.sqrt(F),
        W_V=rng.standard_normal((L_t, H_t, F, d_t)) / math.sqrt(F),
        b_K=rng.standard_normal((L_t, H_t, d_t)) if bias else None,
        b_V=rng.standard_normal((L_t, H_t, d_t)) if bias else None,
        rope_src=O.Rope(th_s, style=style), rope_tgt=O.Rope(th_t, style=style),
        positions=rng.integers(0, 50000, size=T))


@pytest.mark.parametrize("style", [0, 1])
def test_block_diagonal_equals_per_head(style):
    """With W^{l,h} zero outside the rows of source head h (H_s = H_t, d_s = d_t),
    the cross-head form is the per-head form: row (i*H + h)*d + c of the
    cross-head map is row i*d + c of the per-head map of head h."""
    rng = np.random.default_rng(3)
    L_s, L_t, H, T, d, k = 6, 3, 3, 5, 8, 3
    p = _problem(4, L_s=L_s, L_t=L_t, H_s=H, H_t=H, T=T, d_s=d, d_t=d, k=k, style=style,
                 th_s=1e4, th_t=5e5)
    WK_ph = rng.standard_normal((L_t, H, k * d, d))
    WV_ph = rng.standard_normal((L_t, H, k * d, d))
    WK_x = np.zeros((L_t, H, k * H * d, d))
    WV_x = np.zeros((L_t, H, k * H * d, d))
    for h in range(H):
        for i in range(k):
            rows = slice((i * H + h) * d, (i * H + h + 1) * d)
            WK_x[:, h, rows] = WK_ph[:, h, i * d:(i + 1) * d]
            WV_x[:, h, rows] = WV_ph[:, h, i * d:(i + 1) * d]
    common = {n: p[n] for n in ("src_kv", "idx", "b_K", "b_V", "rope_src", "rope_tgt",
                                 "positions")}
    want = O.map_cache(W_K=WK_ph, W_V=WV_ph, **common)
    got = O.map_cache_xhead(W_K=WK_x, W_V=WV_x, **common)
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-12)


@pytest.mark.parametrize("style", [0, 1])
def test_selection_map_copies_a_source_head(style):
    """W^{l,h} = a 0/1 matrix picking source head g(h) of selected layer i(h)
    (d_s = d_t), equal RoPE on both sides, bias b: keys come out as the stored
    source keys plus the bias rotated to each token, values as the stored
    values plus the bias (strip and re-apply cancel, Sec. 3.3)."""
    L_s, L_t, H_s, H_t, T, d, k = 5, 2, 3, 4, 6, 8, 2
    p = _problem(5, L_s=L_s, L_t=L_t, H_s=H_s, H_t=H_t, T=T, d_s=d, d_t=d, k=k, style=style)
    pick = {(l, h): ((l + h) % k, (2 * h + l) % H_s) for l in range(L_t) for h in range(H_t)}
    F = k * H_s * d
    W = np.zeros((L_t, H_t, F, d))
    for (l, h), (i, g) in pick.items():
        W[l, h, (i * H_s + g) * d:(i * H_s + g + 1) * d] = np.eye(d)
    p["W_K"], p["W_V"] = W, W.copy()
    out = O.map_cache_xhead(**p)
    bias_rot = O.rope_rotate(np.broadcast_to(p["b_K"][:, :, None, :], (L_t, H_t, T, d)),
                             p["positions"], p["rope_tgt"])
    for (l, h), (i, g) in pick.items():
        s = p["idx"][l, i]
        np.testing.assert_allclose(out[l, 0, h], p["src_kv"][s, 0, g] + bias_rot[l, h],
                                   atol=1e-12)
        np.testing.assert_allclose(out[l, 1, h], p["src_kv"][s, 1, g] + p["b_V"][l, h],
                                   atol=1e-12)


def _rot_matrix(pos, w, d, style):
    """Block rotation matrix of one token built plane by plane (column vectors)."""
    R = np.zeros((d, d))
    for j in range(d // 2):
        u, v = (j, j + d // 2) if style == 0 else (2 * j, 2 * j + 1)
        a = pos * w[j]
        R[u, u], R[u, v] = math.cos(a), -math.sin(a)
        R[v, u], R[v, v] = math.sin(a), math.cos(a)
    return R


@pytest.mark.parametrize("style", [0, 1])
def test_dense_matrix_evaluation_with_different_head_dims(style):
    """d_s != d_t and H_s != H_t: per token, build the feature vector with
    numerically inverted rotation matrices, multiply, add, rotate."""
    p = _problem(6, H_s=2, H_t=3, T=4, d_s=8, d_t=4, k=2, style=style, th_s=1e4, th_t=1e6)
    src, idx, pos = p["src_kv"], p["idx"], p["positions"]
    ws = O.rope_inv_freq(p["rope_src"], 8)
    wt = O.rope_inv_freq(p["rope_tgt"], 4)
    got = O.map_cache_xhead(**p)
    L_t, H_t = idx.shape[0], 3
    for l in range(L_t):
        for t in range(len(pos)):
            Rinv = np.linalg.inv(_rot_matrix(pos[t], ws, 8, style))
            xk = np.concatenate([Rinv @ src[s, 0, g, t] for s in idx[l] for g in range(2)])
            xv = np.concatenate([src[s, 1, g, t] for s in idx[l] for g in range(2)])
            Rt = _rot_matrix(pos[t], wt, 4, style)
            for h in range(H_t):
                yk = Rt @ (xk @ p["W_K"][l, h] + p["b_K"][l, h])
                yv = xv @ p["W_V"][l, h] + p["b_V"][l, h]
                np.testing.assert_allclose(got[l, 0, h, t], yk, atol=1e-11)
                np.testing.assert_allclose(got[l, 1, h, t], yv, atol=1e-11)


def test_source_head_reordering():
    """Permuting the source heads together with the matching W rows leaves the
    result unchanged; permuting only the heads changes it."""
    p = _problem(7, H_s=4, H_t=2, k=2)
    perm = np.array([2, 0, 3, 1])
    k, H_s, d = 2, 4, 8
    rows = np.concatenate([np.arange((i * H_s + perm[g]) * d, (i * H_s + perm[g] + 1) * d)
                           for i in range(k) for g in range(H_s)])
    q = dict(p)
    q["src_kv"] = p["src_kv"][:, :, perm]
    q["W_K"], q["W_V"] = p["W_K"][:, :, rows], p["W_V"][:, :, rows]
    np.testing.assert_allclose(O.map_cache_xhead(**q), O.map_cache_xhead(**p), atol=1e-12)
    r = dict(p)
    r["src_kv"] = q["src_kv"]
    assert np.abs(O.map_cache_xhead(**r) - O.map_cache_xhead(**p)).max() > 1e-3


@pytest.mark.parametrize("style,bias", [(0, True), (1, False)])
def test_loops_match_vectorised(style, bias):
    p = _problem(8, H_s=3, H_t=2, T=3, d_s=8, d_t=6, k=2, style=style, bias=bias,
                 th_s=1e4, th_t=5e5)
    np.testing.assert_allclose(O.map_cache_xhead_loops(**p), O.map_cache_xhead(**p),
                               rtol=0, atol=1e-13)
