"""fp64 CPU oracle for cross-model KV cache mapping (TEST INFRASTRUCTURE).

This module is the checker, not the product.  Only the test suite, the smoke
entry point and the benchmark's CPU-baseline leg may import it.  It shares no
code with the HIP path: it does its own RoPE, its own gather, its own
contraction, and it imports nothing but NumPy.

What it computes (paper: "Cross-Model KV Cache Transfer in LLM Families: A
Closed-Form Linear Mapping for Prefill Reuse"):

* Eq. (ridge_kv), Sec. 3.1 -- the per-head affine map
  ``K_hat = X_K W_K + b_K`` and ``V_hat = X_V W_V + b_V``;
* Sec. 3.2 (cross-layer source selection) -- X is the concatenation, in the
  order of the selected-layer list, of the source features of the k selected
  source layers.  This oracle implements the per-head form, in which the
  block taken from each selected layer is that layer's head ``h`` only, so
  ``W`` is ``[k*d, d]`` (the paper's cross-head form concatenates all KV heads
  of each layer; the per-head form is that W restricted to be block-diagonal
  over heads);
* Sec. 3.3 (content-space mapping) -- keys are stripped of the source RoPE
  before the map, the bias is added in content space, and the target RoPE is
  applied afterwards at the same positions:
  ``K_hat = (K_s R_src^{-1}(t) W_K + b_K) R_tgt(t)``; values carry no RoPE;
* Eq. (Wstar), Sec. 3.1 -- the closed-form ridge fit on centred data with the
  bias recovered as ``b = mean(Y) - mean(X) W``;
* Sec. 3.2 with Eq. (ridge_kv) in the cross-head form -- ``map_layer_xhead``:
  the input of each target head concatenates every KV head of every selected
  source layer, W^{l,h} is ``[k*H_s*d_s, d_t]``, and source and target may
  differ in head count and head dimension;
* Appendix D (serving cost) -- the mapper parameter count;
* Sec. 3.1 (Fitting) with Sec. 3.3 -- ``fit_cache``: the whole per-head
  mapper fitted from two models' caches of the same calibration tokens, the
  keys of both sides stripped of their RoPE before the fit;
* Sec. 2.3, Eq. (single_source_ols), and Sec. 3.2 -- ``probe_r2`` /
  ``select_topk``: the single-source OLS coefficient of determination of
  every (source layer, target layer, head) for stripped keys and values, and
  the top-k source layers of each target layer by its head average;
* Sec. 4.4 with Appendix F (Run information) -- ``mlp_map_layer``: the MLP
  mapper (two 1024-unit ReLU hidden layers per target layer, head, K|V) as
  a drop-in for the ridge map, with the same strip and re-apply of RoPE.

Everything is evaluated in float64 on inputs that are upcast exactly from
their stored precision.  There is no blocking, fusion or reordering beyond
the definition: a reader can check each function against the paper by eye.

Readings taken where the paper is silent (each is listed in the design notes):
RoPE pairs are the half-split ("rotate-half") layout by default, with the
interleaved layout as an option; frequencies are ``theta^(-2j/d)`` over the
full head dimension; the optional Llama-3 frequency rescaling follows the
published Llama 3.1 rule; index lists are 0-based and their order fixes the
order of W's row blocks; a missing bias means zero.
"""

from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

__all__ = [
    "Rope",
    "rope_inv_freq",
    "rope_angles",
    "rope_rotate",
    "map_layer",
    "map_cache",
    "map_cache_loops",
    "scatter_rows",
    "ridge_fit",
    "ridge_fit_svd",
    "mapper_params",
    "rel_fro",
    "fit_cache",
    "ols_r2",
    "probe_r2",
    "select_topk",
    "mlp_map_layer",
    "mlp_map_cache",
]

HALF_SPLIT = 0
INTERLEAVED = 1


@dataclass(frozen=True)
class Rope:
    """RoPE parameters of one model (Sec. 3.3).

    ``style`` 0 pairs channel j with channel j + d/2 (rotate-half layout);
    ``style`` 1 pairs channel 2j with channel 2j + 1.
    ``factor`` == 1 disables the Llama-3 frequency rescaling; otherwise
    ``low_freq_factor``, ``high_freq_factor`` and ``original_max_pos`` are the
    published Llama 3.1 rescaling parameters.
    """

    theta: float
    style: int = HALF_SPLIT
    factor: float = 1.0
    low_freq_factor: float = 1.0
    high_freq_factor: float = 4.0
    original_max_pos: int = 8192

    @staticmethod
    def from_dict(p: dict) -> "Rope":
        return Rope(
            theta=float(p["theta"]),
            style=int(p.get("style", 0)),
            factor=float(p.get("factor", 1.0)),
            low_freq_factor=float(p.get("low_freq_factor", 1.0)),
            high_freq_factor=float(p.get("high_freq_factor", 4.0)),
            original_max_pos=int(p.get("original_max_pos", 8192)),
        )


def _as_rope(r) -> Rope:
    return r if isinstance(r, Rope) else Rope.from_dict(r)


def rope_inv_freq(rope, d: int) -> np.ndarray:
    """Angular frequency of each of the d/2 rotation planes, float64 [d/2].

    Base rule (RoPE, as cited in Sec. 3.3): omega_j = theta^(-2j/d).
    Optional Llama-3 rescaling, applied per frequency with wavelength
    lambda_j = 2*pi/omega_j and original context length C:
      lambda_j < C/high_freq_factor  -> omega_j unchanged,
      lambda_j > C/low_freq_factor   -> omega_j / factor,
      otherwise                      -> (1-s)*omega_j/factor + s*omega_j,
                                        s = (C/lambda_j - low)/(high - low).
    """
    rope = _as_rope(rope)
    if d % 2:
        raise ValueError("head dimension must be even")
    j = np.arange(d // 2, dtype=np.float64)
    omega = rope.theta ** (-2.0 * j / d)
    if rope.factor == 1.0:
        return omega
    ctx = float(rope.original_max_pos)
    lo, hi = rope.low_freq_factor, rope.high_freq_factor
    out = np.empty_like(omega)
    for n, w in enumerate(omega):
        wavelen = 2.0 * math.pi / w
        if wavelen < ctx / hi:
            out[n] = w
        elif wavelen > ctx / lo:
            out[n] = w / rope.factor
        else:
            s = (ctx / wavelen - lo) / (hi - lo)
            out[n] = (1.0 - s) * w / rope.factor + s * w
    return out


def rope_angles(positions, rope, d: int) -> np.ndarray:
    """Rotation angle a[t, j] = positions[t] * omega_j, float64 [T, d/2]."""
    pos = np.asarray(positions, dtype=np.float64)
    return pos[:, None] * rope_inv_freq(rope, d)[None, :]


def _planes(d: int, style: int):
    """Channel indices (first, second) of each rotation plane."""
    j = np.arange(d // 2)
    if style == HALF_SPLIT:
        return j, j + d // 2
    if style == INTERLEAVED:
        return 2 * j, 2 * j + 1
    raise ValueError(f"unknown RoPE style {style}")


def rope_rotate(x, positions, rope, inverse: bool = False) -> np.ndarray:
    """Apply R_Theta(t) (or its inverse) to every d-dim row of x.

    x has shape [..., T, d] and row t is rotated at positions[t].  Each plane
    (u, v) turns by angle a:  u' = u cos a - v sin a,  v' = v cos a + u sin a;
    the inverse turns by -a (R is orthogonal, Sec. 3.3).
    """
    rope = _as_rope(rope)
    x = np.asarray(x, dtype=np.float64)
    d = x.shape[-1]
    a = rope_angles(positions, rope, d)
    if inverse:
        a = -a
    c, s = np.cos(a), np.sin(a)
    first, second = _planes(d, rope.style)
    u, v = x[..., first], x[..., second]
    out = np.empty_like(x)
    out[..., first] = u * c - v * s
    out[..., second] = v * c + u * s
    return out


def map_layer(src_kv, idx_row, W_K_l, W_V_l, b_K_l, b_V_l, rope_src, rope_tgt,
              positions) -> np.ndarray:
    """Mapped target KV of one target layer, float64 [2, H, T, d].

    src_kv   [L_s, 2, H, T, d]  stored source cache (keys carry source RoPE)
    idx_row  [k]                selected source layers, 0-based; list order is
                                the order of W's row blocks
    W_K_l    [H, k*d, d]        per-head key map; row block i <-> idx_row[i]
    W_V_l    [H, k*d, d]        per-head value map
    b_K_l    [H, d] or None     key bias (content space), None means zero
    b_V_l    [H, d] or None     value bias
    """
    idx_row = [int(i) for i in idx_row]
    # Only the selected layers are upcast, so a large cache is never copied whole.
    def layer(s, kv):
        return np.asarray(src_kv[s, kv], dtype=np.float64)  # [H, T, d]
    # Sec. 3.3: strip the source rotation from each selected layer's keys.
    xk = np.concatenate(
        [rope_rotate(layer(s, 0), positions, rope_src, inverse=True) for s in idx_row],
        axis=-1)                                            # [H, T, k*d]
    xv = np.concatenate([layer(s, 1) for s in idx_row], axis=-1)
    # Eq. (ridge_kv): one affine map per head.
    yk = np.matmul(xk, np.asarray(W_K_l, dtype=np.float64))  # [H, T, d]
    yv = np.matmul(xv, np.asarray(W_V_l, dtype=np.float64))
    if b_K_l is not None:
        yk = yk + np.asarray(b_K_l, dtype=np.float64)[:, None, :]
    if b_V_l is not None:
        yv = yv + np.asarray(b_V_l, dtype=np.float64)[:, None, :]
    # Sec. 3.3: re-encode keys with the target rotation at the same positions.
    yk = rope_rotate(yk, positions, rope_tgt, inverse=False)
    return np.stack([yk, yv], axis=0)


def map_cache(src_kv, idx, W_K, W_V, b_K, b_V, rope_src, rope_tgt,
              positions) -> np.ndarray:
    """Mapped target cache, float64 [L_t, 2, H, T, d].

    idx [L_t, k]; W_K, W_V [L_t, H, k*d, d]; b_K, b_V [L_t, H, d] or None.
    """
    idx = np.asarray(idx)
    L_t = idx.shape[0]
    out = []
    for l in range(L_t):
        out.append(map_layer(
            src_kv, idx[l], W_K[l], W_V[l],
            None if b_K is None else b_K[l], None if b_V is None else b_V[l],
            rope_src, rope_tgt, positions))
    return np.stack(out, axis=0)


def map_cache_loops(src_kv, idx, W_K, W_V, b_K, b_V, rope_src, rope_tgt,
                    positions) -> np.ndarray:
    """Scalar-loop evaluation of the same map, for tiny inputs only.

    Written element by element from the formula in Sec. 3.3 so that an index
    slip in the vectorised path shows up as a disagreement.
    """
    rs, rt = _as_rope(rope_src), _as_rope(rope_tgt)
    src = np.asarray(src_kv, dtype=np.float64)
    L_s, _, H, T, d = src.shape
    idx = np.asarray(idx)
    L_t, k = idx.shape
    ws = rope_inv_freq(rs, d)
    wt = rope_inv_freq(rt, d)
    fs, ss = _planes(d, rs.style)
    ft, st = _planes(d, rt.style)
    out = np.zeros((L_t, 2, H, T, d))
    for l in range(L_t):
        for h in range(H):
            for t in range(T):
                p = float(positions[t])
                x_k = [0.0] * (k * d)
                x_v = [0.0] * (k * d)
                for i in range(k):
                    s = int(idx[l, i])
                    row = src[s, 0, h, t]
                    for j in range(d // 2):
                        a = -p * ws[j]
                        u, v = row[fs[j]], row[ss[j]]
                        x_k[i * d + fs[j]] = u * math.cos(a) - v * math.sin(a)
                        x_k[i * d + ss[j]] = v * math.cos(a) + u * math.sin(a)
                    for c in range(d):
                        x_v[i * d + c] = src[s, 1, h, t, c]
                y_k = [0.0] * d
                y_v = [0.0] * d
                for c in range(d):
                    acc_k = 0.0 if b_K is None else float(b_K[l, h, c])
                    acc_v = 0.0 if b_V is None else float(b_V[l, h, c])
                    for r in range(k * d):
                        acc_k += x_k[r] * float(W_K[l, h, r, c])
                        acc_v += x_v[r] * float(W_V[l, h, r, c])
                    y_k[c] = acc_k
                    y_v[c] = acc_v
                for j in range(d // 2):
                    a = p * wt[j]
                    u, v = y_k[ft[j]], y_k[st[j]]
                    out[l, 0, h, t, ft[j]] = u * math.cos(a) - v * math.sin(a)
                    out[l, 0, h, t, st[j]] = v * math.cos(a) + u * math.sin(a)
                out[l, 1, h, t, :] = y_v
    return out


def map_layer_xhead(src_kv, idx_row, W_K_l, W_V_l, b_K_l, b_V_l, rope_src, rope_tgt,
                    positions) -> np.ndarray:
    """Cross-head form of one target layer, float64 [2, H_t, T, d_t].

    Eq. (ridge_kv) with the features of Sec. 3.2: for every selected source
    layer (in list order) the keys, or values, of ALL its KV heads are
    concatenated (head 0 first), and those per-layer blocks are concatenated
    in turn, so the input of target head h has k*H_s*d_s features and
    W^{l,h} is [k*H_s*d_s, d_t].  Keys are stripped of the source rotation
    before, and given the target rotation after, the map (Sec. 3.3).

    src_kv   [L_s, 2, H_s, T, d_s]
    idx_row  [k]                     selected source layers, 0-based
    W_K_l    [H_t, k*H_s*d_s, d_t]   row (i*H_s + g)*d_s + c multiplies
                                     channel c of source head g of layer
                                     idx_row[i]
    W_V_l    [H_t, k*H_s*d_s, d_t]
    b_K_l    [H_t, d_t] or None      content-space bias (None means zero)
    b_V_l    [H_t, d_t] or None
    """
    idx_row = [int(i) for i in idx_row]

    def layer(s, kv):
        return np.asarray(src_kv[s, kv], dtype=np.float64)  # [H_s, T, d_s]

    def heads_side_by_side(x):
        # [H_s, T, d_s] -> [T, H_s*d_s], head g in columns g*d_s .. g*d_s+d_s-1
        return np.concatenate(list(x), axis=-1)

    xk = np.concatenate(
        [heads_side_by_side(rope_rotate(layer(s, 0), positions, rope_src, inverse=True))
         for s in idx_row], axis=-1)                        # [T, k*H_s*d_s]
    xv = np.concatenate([heads_side_by_side(layer(s, 1)) for s in idx_row], axis=-1)
    yk = np.matmul(xk[None], np.asarray(W_K_l, dtype=np.float64))  # [H_t, T, d_t]
    yv = np.matmul(xv[None], np.asarray(W_V_l, dtype=np.float64))
    if b_K_l is not None:
        yk = yk + np.asarray(b_K_l, dtype=np.float64)[:, None, :]
    if b_V_l is not None:
        yv = yv + np.asarray(b_V_l, dtype=np.float64)[:, None, :]
    yk = rope_rotate(yk, positions, rope_tgt, inverse=False)
    return np.stack([yk, yv], axis=0)


def map_cache_xhead(src_kv, idx, W_K, W_V, b_K, b_V, rope_src, rope_tgt,
                    positions) -> np.ndarray:
    """Cross-head form of the whole cache, float64 [L_t, 2, H_t, T, d_t].

    idx [L_t, k]; W_K, W_V [L_t, H_t, k*H_s*d_s, d_t]; b_K, b_V [L_t, H_t, d_t]
    or None.
    """
    idx = np.asarray(idx)
    return np.stack([
        map_layer_xhead(src_kv, idx[l], W_K[l], W_V[l],
                        None if b_K is None else b_K[l], None if b_V is None else b_V[l],
                        rope_src, rope_tgt, positions)
        for l in range(idx.shape[0])], axis=0)


def map_cache_xhead_loops(src_kv, idx, W_K, W_V, b_K, b_V, rope_src, rope_tgt,
                          positions) -> np.ndarray:
    """Scalar-loop evaluation of the cross-head form, for tiny inputs only.

    Each feature index r is decoded into (selected layer i, source head g,
    channel c) by integer division, the reverse of how the vectorised form
    builds its concatenation, so a layout slip in either shows up.
    """
    rs, rt = _as_rope(rope_src), _as_rope(rope_tgt)
    src = np.asarray(src_kv, dtype=np.float64)
    L_s, _, H_s, T, d_s = src.shape
    idx = np.asarray(idx)
    L_t, k = idx.shape
    H_t, F, d_t = np.asarray(W_K).shape[1:]
    assert F == k * H_s * d_s
    ws, wt = rope_inv_freq(rs, d_s), rope_inv_freq(rt, d_t)
    fs, ss = _planes(d_s, rs.style)
    ft, st = _planes(d_t, rt.style)
    # partner channel and sign of the plane each source channel belongs to
    part = [0] * d_s
    plane = [0] * d_s
    first = [False] * d_s
    for j in range(d_s // 2):
        part[fs[j]], part[ss[j]] = ss[j], fs[j]
        plane[fs[j]] = plane[ss[j]] = j
        first[fs[j]] = True
    out = np.zeros((L_t, 2, H_t, T, d_t))
    for l in range(L_t):
        for t in range(T):
            p = float(positions[t])
            xk = [0.0] * F
            xv = [0.0] * F
            for r in range(F):
                i, rem = divmod(r, H_s * d_s)
                g, c = divmod(rem, d_s)
                s = int(idx[l, i])
                a = -p * ws[plane[c]]          # inverse rotation
                u = src[s, 0, g, t, c]
                v = src[s, 0, g, t, part[c]]
                if first[c]:
                    xk[r] = u * math.cos(a) - v * math.sin(a)
                else:
                    xk[r] = u * math.cos(a) + v * math.sin(a)
                xv[r] = src[s, 1, g, t, c]
            for h in range(H_t):
                yk = [0.0] * d_t
                for c in range(d_t):
                    acc_k = 0.0 if b_K is None else float(b_K[l, h, c])
                    acc_v = 0.0 if b_V is None else float(b_V[l, h, c])
                    for r in range(F):
                        acc_k += xk[r] * float(W_K[l, h, r, c])
                        acc_v += xv[r] * float(W_V[l, h, r, c])
                    yk[c] = acc_k
                    out[l, 1, h, t, c] = acc_v
                for j in range(d_t // 2):
                    a = p * wt[j]
                    u, v = yk[ft[j]], yk[st[j]]
                    out[l, 0, h, t, ft[j]] = u * math.cos(a) - v * math.sin(a)
                    out[l, 0, h, t, st[j]] = v * math.cos(a) + u * math.sin(a)
    return out


def scatter_rows(pool, rows, slot_mapping) -> np.ndarray:
    """Write mapped rows into a slot-addressed target pool (paged layout).

    pool [L_t, 2, H, S, d] (any dtype, returned as a copy), rows
    [L_t, 2, H, T, d], slot_mapping [T]: row t lands in slot slot_mapping[t];
    slots not named in slot_mapping keep their previous contents.
    """
    out = np.array(pool, copy=True)
    out[:, :, :, np.asarray(slot_mapping, dtype=np.int64), :] = rows
    return out


def ridge_fit(X, Y, lam: float = 0.01):
    """Closed-form ridge fit of Eq. (Wstar) with centring (Sec. 3.1).

    X [N, p], Y [N, q].  Centre both, solve (Xc^T Xc + lam I) W = Xc^T Yc by
    Cholesky, recover b = mean(Y) - mean(X) W.  Returns (W [p, q], b [q]).
    """
    X = np.asarray(X, dtype=np.float64)
    Y = np.asarray(Y, dtype=np.float64)
    xm, ym = X.mean(axis=0), Y.mean(axis=0)
    Xc, Yc = X - xm, Y - ym
    A = Xc.T @ Xc + lam * np.eye(X.shape[1])
    L = np.linalg.cholesky(A)
    Z = np.linalg.solve(L, Xc.T @ Yc)
    W = np.linalg.solve(L.T, Z)
    b = ym - xm @ W
    return W, b


def ridge_fit_svd(X, Y, lam: float = 0.01):
    """Same fit through the SVD of the centred design: W = V diag(s/(s^2+lam)) U^T Yc."""
    X = np.asarray(X, dtype=np.float64)
    Y = np.asarray(Y, dtype=np.float64)
    xm, ym = X.mean(axis=0), Y.mean(axis=0)
    Xc, Yc = X - xm, Y - ym
    U, s, Vt = np.linalg.svd(Xc, full_matrices=False)
    W = Vt.T @ ((s / (s * s + lam))[:, None] * (U.T @ Yc))
    b = ym - xm @ W
    return W, b


def mapper_params(L_t: int, H_t: int, k: int, H_s: int, d_s: int, d_t: int) -> int:
    """Mapper parameter count for K and V together (Appendix D, serving cost).

    Each of the L_t * H_t target heads has a K map and a V map with
    k*H_s*d_s input features and d_t outputs (cross-head form).  The per-head
    form used on the hot path is the case H_s = 1 in the feature count.
    """
    return 2 * L_t * H_t * (k * H_s * d_s) * d_t


def rel_fro(x, ref) -> float:
    """||x - ref||_F / ||ref||_F (absolute error when ref is all zero)."""
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    num = float(np.linalg.norm((x - ref).ravel()))
    den = float(np.linalg.norm(ref.ravel()))
    return num if den == 0.0 else num / den


def _plane(cache, layer, kv, h):
    """One (layer, K|V, head) plane of a cache as float64 [N, d]."""
    return np.asarray(cache[layer, kv, h], dtype=np.float64)


def fit_cache(src_kv, idx, tgt_kv, rope_src, rope_tgt, positions, lam: float = 0.01):
    """Fit the whole per-head mapper from calibration caches (Sec. 3.1, Fitting).

    src_kv [L_s, 2, H, N, d] and tgt_kv [L_t, 2, H, N, d] hold the source and
    the target model's caches of the same N calibration tokens, at
    ``positions`` [N].  For target layer l and head h the design matrix
    concatenates, in the order of idx[l], the selected source layers' keys
    stripped of the source RoPE (values as stored), and the response is the
    target's keys stripped of the target RoPE (Sec. 3.3: the map is fitted in
    the position-free space) or its values.  Each (l, h, K|V) is one
    ridge_fit.  Returns W_K, W_V [L_t, H, k*d, d] and b_K, b_V [L_t, H, d]
    (float64), the arguments map_cache takes.
    """
    idx = np.asarray(idx)
    L_t, k = idx.shape
    H, d = np.asarray(src_kv[0, 0]).shape[0], np.asarray(src_kv[0, 0]).shape[-1]
    W = np.zeros((2, L_t, H, k * d, d))
    b = np.zeros((2, L_t, H, d))
    for l in range(L_t):
        for h in range(H):
            for kv in range(2):
                blocks = []
                for s in idx[l]:
                    x = _plane(src_kv, int(s), kv, h)
                    if kv == 0:
                        x = rope_rotate(x, positions, rope_src, inverse=True)
                    blocks.append(x)
                X = np.concatenate(blocks, axis=1)
                Y = _plane(tgt_kv, l, kv, h)
                if kv == 0:
                    Y = rope_rotate(Y, positions, rope_tgt, inverse=True)
                W[kv, l, h], b[kv, l, h] = ridge_fit(X, Y, lam)
    return W[0], W[1], b[0], b[1]


def ols_r2(X, Y) -> float:
    """Coefficient of determination of the ordinary least-squares fit
    Y ~ X W + b (Eq. single_source_ols), pooled over the output dimensions:
    1 - sum ||Y - X W - b||^2 / sum ||Y - mean(Y)||^2.  The fit is lstsq on
    the centred data (no regularisation)."""
    X = np.asarray(X, dtype=np.float64)
    Y = np.asarray(Y, dtype=np.float64)
    Xc, Yc = X - X.mean(axis=0), Y - Y.mean(axis=0)
    W = np.linalg.lstsq(Xc, Yc, rcond=None)[0]
    res = Yc - Xc @ W
    return 1.0 - float(np.sum(res * res)) / float(np.sum(Yc * Yc))


def probe_r2(src_kv, tgt_kv, rope_src, rope_tgt, positions) -> np.ndarray:
    """Single-source linear probe of Sec. 2.3: R2[l', l, h, c] for every source
    layer l', target layer l and KV head h, for c = 0 the keys of both sides
    stripped of their RoPE (K_stripped) and c = 1 the values, each one OLS fit
    of the target's per-token head features on the source's (Eq.
    single_source_ols).  float64 [L_s, L_t, H, 2]."""
    src = np.asarray(src_kv)
    tgt = np.asarray(tgt_kv)
    L_s, _, H = src.shape[:3]
    L_t = tgt.shape[0]
    out = np.zeros((L_s, L_t, H, 2))
    for h in range(H):
        xs = [[rope_rotate(_plane(src, s, 0, h), positions, rope_src, inverse=True),
               _plane(src, s, 1, h)] for s in range(L_s)]
        ys = [[rope_rotate(_plane(tgt, l, 0, h), positions, rope_tgt, inverse=True),
               _plane(tgt, l, 1, h)] for l in range(L_t)]
        for s in range(L_s):
            for l in range(L_t):
                for c in range(2):
                    out[s, l, h, c] = ols_r2(xs[s][c], ys[l][c])
    return out


def select_topk(r2, k: int) -> np.ndarray:
    """Top-k source layers of each target layer (Sec. 3.2): rank the source
    layers by R2 averaged over heads and over stripped keys and values, take
    the k best (an equal score goes to the lower source index) and list them
    in ascending order.  r2 [L_s, L_t, H, 2] -> int32 [L_t, k]."""
    r2 = np.asarray(r2, dtype=np.float64)
    L_s, L_t = r2.shape[:2]
    score = r2.mean(axis=(2, 3))                    # [L_s, L_t]
    out = np.zeros((L_t, k), dtype=np.int32)
    for l in range(L_t):
        order = sorted(range(L_s), key=lambda s: (-score[s, l], s))
        out[l] = sorted(order[:k])
    return out


def mlp_map_layer(src_kv, idx_row, mlp_K, mlp_V, rope_src, rope_tgt, positions) -> np.ndarray:
    """The MLP mapper of one target layer (Sec. 4.4), float64 [2, H, T, d].

    The input features are those of the ridge map (stripped keys or values of
    the selected source layers, concatenated in list order), and each
    (head, K|V) has its own network Linear(k*d, F) -> ReLU -> Linear(F, F) ->
    ReLU -> Linear(F, d) (Appendix F: F = 1024).  Keys are re-encoded with the
    target RoPE afterwards, as for the ridge map (Sec. 3.3).
    mlp_K, mlp_V: tuples (W1 [H, k*d, F], b1 [H, F], W2 [H, F, F], b2 [H, F],
    W3 [H, F, d], b3 [H, d]), rows = inputs (x @ W + b).
    """
    idx_row = [int(i) for i in idx_row]

    def layer(s, kv):
        return np.asarray(src_kv[s, kv], dtype=np.float64)   # [H, T, d]
    xk = np.concatenate([rope_rotate(layer(s, 0), positions, rope_src, inverse=True)
                         for s in idx_row], axis=-1)            # [H, T, k*d]
    xv = np.concatenate([layer(s, 1) for s in idx_row], axis=-1)

    def net(x, p):
        W1, b1, W2, b2, W3, b3 = (np.asarray(t, dtype=np.float64) for t in p)
        h1 = np.maximum(np.matmul(x, W1) + b1[:, None, :], 0.0)
        h2 = np.maximum(np.matmul(h1, W2) + b2[:, None, :], 0.0)
        return np.matmul(h2, W3) + b3[:, None, :]
    yk = rope_rotate(net(xk, mlp_K), positions, rope_tgt, inverse=False)
    yv = net(xv, mlp_V)
    return np.stack([yk, yv], axis=0)


def mlp_map_cache(src_kv, idx, mlp_K, mlp_V, rope_src, rope_tgt, positions) -> np.ndarray:
    """MLP mapper of the whole cache, float64 [L_t, 2, H, T, d]; mlp_K / mlp_V
    are tuples of per-layer arrays (W1 [L_t, H, k*d, F], b1 [L_t, H, F], W2
    [L_t, H, F, F], b2 [L_t, H, F], W3 [L_t, H, F, d], b3 [L_t, H, d])."""
    idx = np.asarray(idx)
    return np.stack([
        mlp_map_layer(src_kv, idx[l], tuple(t[l] for t in mlp_K), tuple(t[l] for t in mlp_V),
                      rope_src, rope_tgt, positions)
        for l in range(idx.shape[0])], axis=0)
