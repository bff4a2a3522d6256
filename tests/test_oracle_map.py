"""Pins of the oracle's whole map (Eq. ridge_kv, Sec. 3.2 and Sec. 3.3).

The oracle is checked against special cases with known answers (identity
map, bias only, RoPE re-basing), against an independent dense-matrix
evaluation of the paper's formula with numerically inverted rotations,
against structural properties (block order, linearity, head and K/V
independence, token locality) and against a scalar-loop evaluation.
"""

import math

import numpy as np
import pytest

from oracle import kvx_oracle as O


def _problem(seed, L_s=5, L_t=3, H=2, T=7, d=8, k=2, bias=True, style=0,
             th_s=1e4, th_t=1e4, factor=1.0):
    rng = np.random.default_rng(seed)
    src = rng.standard_normal((L_s, 2, H, T, d))
    idx = np.stack([rng.choice(L_s, k, replace=False) for _ in range(L_t)])
    W_K = rng.standard_normal((L_t, H, k * d, d)) / math.sqrt(k * d)
    W_V = rng.standard_normal((L_t, H, k * d, d)) / math.sqrt(k * d)
    b_K = rng.standard_normal((L_t, H, d)) if bias else None
    b_V = rng.standard_normal((L_t, H, d)) if bias else None
    pos = rng.integers(0, 50000, size=T)
    rs = O.Rope(th_s, style=style, factor=factor)
    rt = O.Rope(th_t, style=style, factor=factor)
    return dict(src_kv=src, idx=idx, W_K=W_K, W_V=W_V, b_K=b_K, b_V=b_V,
                rope_src=rs, rope_tgt=rt, positions=pos)


def _eye_problem(seed, style=0, th_s=1e4, th_t=1e4):
    p = _problem(seed, k=1, bias=False, style=style, th_s=th_s, th_t=th_t)
    L_t, H, kd, d = p["W_K"].shape
    eye = np.broadcast_to(np.eye(d), (L_t, H, d, d)).copy()
    p["W_K"], p["W_V"] = eye, eye.copy()
    return p


@pytest.mark.parametrize("style", [0, 1])
def test_identity_map_returns_selected_source_layer(style):
    """k = 1, W = I, b = 0, equal RoPE on both sides: output = source layer idx[l,0]."""
    p = _eye_problem(10, style=style)
    out = O.map_cache(**p)
    for l in range(out.shape[0]):
        s = p["idx"][l, 0]
        np.testing.assert_allclose(out[l], p["src_kv"][s], atol=1e-12)


@pytest.mark.parametrize("style", [0, 1])
def test_bias_only(style):
    """W = 0: keys become the bias rotated by the target RoPE, values the bias."""
    p = _problem(11, style=style)
    p["W_K"] = np.zeros_like(p["W_K"])
    p["W_V"] = np.zeros_like(p["W_V"])
    out = O.map_cache(**p)
    T = len(p["positions"])
    for l in range(out.shape[0]):
        for h in range(out.shape[2]):
            bk = np.broadcast_to(p["b_K"][l, h], (T, p["b_K"].shape[-1]))
            np.testing.assert_allclose(out[l, 0, h],
                                       O.rope_rotate(bk, p["positions"], p["rope_tgt"]),
                                       atol=1e-13)
            np.testing.assert_allclose(out[l, 1, h], np.broadcast_to(p["b_V"][l, h], (T, bk.shape[1])),
                                       atol=1e-15)


def test_rebasing_between_thetas():
    """k = 1, W = I, b = 0, theta_s != theta_t: each key plane turns by
    p * (w_t - w_s) in the complex form; values pass through."""
    th_s, th_t = 1e4, 1e6
    p = _eye_problem(12, th_s=th_s, th_t=th_t)
    out = O.map_cache(**p)
    d = p["src_kv"].shape[-1]
    j = np.arange(d // 2)
    dw = th_t ** (-2.0 * j / d) - th_s ** (-2.0 * j / d)
    pos = p["positions"]
    for l in range(out.shape[0]):
        x = p["src_kv"][p["idx"][l, 0], 0]            # [H, T, d]
        z = (x[..., : d // 2] + 1j * x[..., d // 2:]) * np.exp(1j * pos[:, None] * dw)
        want = np.concatenate([z.real, z.imag], axis=-1)
        np.testing.assert_allclose(out[l, 0], want, atol=1e-9)
        np.testing.assert_allclose(out[l, 1], p["src_kv"][p["idx"][l, 0], 1], atol=0)


def _dense_R(pos, w, d, style):
    R = np.zeros((d, d))
    for j in range(d // 2):
        a, b = (j, j + d // 2) if style == 0 else (2 * j, 2 * j + 1)
        c, s = math.cos(pos * w[j]), math.sin(pos * w[j])
        R[a, a], R[a, b], R[b, a], R[b, b] = c, -s, s, c
    return R


@pytest.mark.parametrize("style,th_s,th_t", [(0, 1e4, 1e4), (0, 1e4, 1e6), (1, 1e6, 5e5)])
def test_dense_matrix_evaluation(style, th_s, th_t):
    """Evaluate the paper's content-space formula token by token with dense
    rotation matrices, numerically inverted for the strip (column-vector form:
    x_i = R_s(t)^-1 k_i, y = W^T [x_1; ...; x_k] + b, k_hat = R_t(t) y)."""
    p = _problem(13, L_s=4, L_t=3, H=2, T=5, d=8, k=3, style=style,
                 th_s=th_s, th_t=th_t)
    out = O.map_cache(**p)
    d = 8
    ws = np.array([th_s ** (-(2.0 * j) / d) for j in range(d // 2)])
    wt = np.array([th_t ** (-(2.0 * j) / d) for j in range(d // 2)])
    for l in range(3):
        for h in range(2):
            for t in range(5):
                pos = int(p["positions"][t])
                Rs_inv = np.linalg.inv(_dense_R(pos, ws, d, style))
                Rt = _dense_R(pos, wt, d, style)
                xk = np.concatenate([Rs_inv @ p["src_kv"][s, 0, h, t] for s in p["idx"][l]])
                xv = np.concatenate([p["src_kv"][s, 1, h, t] for s in p["idx"][l]])
                yk = p["W_K"][l, h].T @ xk + p["b_K"][l, h]
                yv = p["W_V"][l, h].T @ xv + p["b_V"][l, h]
                np.testing.assert_allclose(out[l, 0, h, t], Rt @ yk, atol=1e-12)
                np.testing.assert_allclose(out[l, 1, h, t], yv, atol=1e-12)


def test_block_order_invariance():
    """Permuting a layer's index list together with W's row blocks changes nothing."""
    p = _problem(14, k=3)
    out = O.map_cache(**p)
    q = dict(p)
    L_t, H, kd, d = p["W_K"].shape
    perm = np.array([2, 0, 1])
    q["idx"] = p["idx"][:, perm]
    blocks = lambda W: W.reshape(L_t, H, 3, d, d)[:, :, perm].reshape(L_t, H, kd, d)
    q["W_K"], q["W_V"] = blocks(p["W_K"]), blocks(p["W_V"])
    np.testing.assert_allclose(O.map_cache(**q), out, atol=1e-12)


def test_block_order_matters_without_permuting_W():
    """Reordering the index list alone must change the result (concat order is real)."""
    p = _problem(15, k=2)
    q = dict(p)
    q["idx"] = p["idx"][:, ::-1].copy()
    assert np.max(np.abs(O.map_cache(**q) - O.map_cache(**p))) > 1e-3


def test_linearity():
    """The map is linear in (W, b) jointly and linear in the source when b = 0."""
    p1 = _problem(16)
    p2 = _problem(17)
    p2["src_kv"], p2["idx"], p2["positions"] = p1["src_kv"], p1["idx"], p1["positions"]
    s = dict(p1)
    for key in ("W_K", "W_V", "b_K", "b_V"):
        s[key] = 2.0 * p1[key] - 0.5 * p2[key]
    np.testing.assert_allclose(O.map_cache(**s),
                               2.0 * O.map_cache(**p1) - 0.5 * O.map_cache(**p2), atol=1e-11)
    a = _problem(18, bias=False)
    b = dict(a)
    b["src_kv"] = _problem(19)["src_kv"]
    c = dict(a)
    c["src_kv"] = 3.0 * a["src_kv"] + b["src_kv"]
    np.testing.assert_allclose(O.map_cache(**c), 3.0 * O.map_cache(**a) + O.map_cache(**b),
                               atol=1e-11)


def test_head_and_kv_independence():
    """Perturbing one head's key map changes exactly that (layer, head, K) tensor."""
    p = _problem(20, L_t=3, H=3)
    out = O.map_cache(**p)
    q = dict(p)
    q["W_K"] = p["W_K"].copy()
    q["W_K"][1, 2] += 0.1
    diff = np.abs(O.map_cache(**q) - out).reshape(3, 2, 3, -1).max(axis=-1)
    changed = diff > 1e-12
    assert changed[1, 0, 2]
    assert changed.sum() == 1


def test_loops_match_vectorised():
    p = _problem(21, L_s=3, L_t=2, H=2, T=4, d=8, k=2, style=0, th_s=1e4, th_t=5e5)
    np.testing.assert_allclose(O.map_cache_loops(**p), O.map_cache(**p), atol=1e-12)
    p = _problem(22, L_s=3, L_t=2, H=1, T=3, d=8, k=2, style=1, factor=8.0)
    np.testing.assert_allclose(O.map_cache_loops(**p), O.map_cache(**p), atol=1e-12)


def test_token_locality_chunks_and_permutation():
    """Row t depends only on source row t and position t: mapping in chunks, or
    in permuted order, gives the same rows."""
    p = _problem(23, T=13)
    full = O.map_cache(**p)
    parts = []
    for a, b in [(0, 5), (5, 6), (6, 13)]:
        q = dict(p)
        q["src_kv"] = p["src_kv"][:, :, :, a:b]
        q["positions"] = p["positions"][a:b]
        parts.append(O.map_cache(**q))
    np.testing.assert_allclose(np.concatenate(parts, axis=3), full, atol=1e-13)
    perm = np.random.default_rng(0).permutation(13)
    q = dict(p)
    q["src_kv"] = p["src_kv"][:, :, :, perm]
    q["positions"] = p["positions"][perm]
    np.testing.assert_allclose(O.map_cache(**q), full[:, :, :, perm], atol=1e-13)


def test_map_layer_matches_map_cache():
    p = _problem(24)
    full = O.map_cache(**p)
    for l in range(full.shape[0]):
        one = O.map_layer(p["src_kv"], p["idx"][l], p["W_K"][l], p["W_V"][l],
                          p["b_K"][l], p["b_V"][l], p["rope_src"], p["rope_tgt"],
                          p["positions"])
        np.testing.assert_array_equal(one, full[l])


def test_none_bias_equals_zero_bias():
    p = _problem(25)
    q = dict(p)
    q["b_K"] = np.zeros_like(p["b_K"])
    q["b_V"] = np.zeros_like(p["b_V"])
    r = dict(p)
    r["b_K"] = r["b_V"] = None
    np.testing.assert_array_equal(O.map_cache(**q), O.map_cache(**r))


def test_duplicate_indices_are_well_defined():
    """A repeated source layer contributes twice, each block through its own W rows."""
    p = _problem(26, k=2, bias=False)
    p["idx"] = np.array([[1, 1]] * p["idx"].shape[0])
    d = p["src_kv"].shape[-1]
    L_t, H = p["W_K"].shape[:2]
    q = dict(p)
    q["idx"] = np.array([[1]] * L_t)
    q["W_K"] = p["W_K"][:, :, :d] + p["W_K"][:, :, d:]
    q["W_V"] = p["W_V"][:, :, :d] + p["W_V"][:, :, d:]
    np.testing.assert_allclose(O.map_cache(**p), O.map_cache(**q), atol=1e-12)


def test_scatter_rows_paged_layout():
    """Rows land in their slots; every other slot keeps its old contents; an
    identity slot map reproduces the dense layout."""
    rng = np.random.default_rng(27)
    rows = rng.standard_normal((2, 2, 3, 5, 4))
    pool = np.full((2, 2, 3, 16, 4), -7.0)
    slots = np.array([9, 2, 15, 0, 4])
    out = O.scatter_rows(pool, rows, slots)
    np.testing.assert_array_equal(out[:, :, :, slots], rows)
    rest = np.setdiff1d(np.arange(16), slots)
    assert np.all(out[:, :, :, rest] == -7.0)
    dense = O.scatter_rows(np.zeros((2, 2, 3, 5, 4)), rows, np.arange(5))
    np.testing.assert_array_equal(dense, rows)
