"""Shared helpers for the GPU parity tests: run the HIP path through the C ABI
and compare with the fp64 oracle tensor by tensor."""

from __future__ import annotations

import sys

import numpy as np
import torch

from oracle import kvx_oracle as O

TOL = {"f32": 1e-5, "bf16": 3e-3}


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def np32(t):
    """Exact float32 copy on the host (bf16 widens exactly)."""
    return None if t is None else t.detach().float().cpu().numpy()


def run_gpu(kvx, inp, out=None, **kw):
    src = inp["src"]
    cfg = inp["cfg"]
    L_t = inp["idx"].shape[0]
    if out is None:
        out = torch.empty((L_t, 2, cfg.H, inp["T"], cfg.d), dtype=src.dtype, device=src.device)
    kvx.map_cache(src, inp["idx"], inp["W_K"], inp["W_V"], inp["b_K"], inp["b_V"],
                  inp["rope_src"], inp["rope_tgt"], inp["positions"], out, **kw)
    torch.cuda.synchronize()
    return out


class _LazySource:
    """Indexable like src[s, kv]; copies one (layer, K|V) plane to the host on
    first use, so a large cache is never copied whole."""

    def __init__(self, src, tokens):
        self.src = src
        self.ti = None if tokens is None else torch.as_tensor(tokens, device=src.device,
                                                                dtype=torch.long)
        self.cache = {}

    def __getitem__(self, key):
        if key not in self.cache:
            s, kv = key
            plane = self.src[s, kv]
            if self.ti is not None:
                plane = plane.index_select(1, self.ti)
            self.cache[key] = np32(plane)
        return self.cache[key]


def oracle_rows(inp, tokens=None, layers=None):
    """fp64 oracle for the given token rows (all rows if None) and layers."""
    pos = inp["positions"]
    if tokens is not None:
        pos = pos.index_select(0, torch.as_tensor(tokens, device=pos.device, dtype=torch.long))
    src = _LazySource(inp["src"], tokens)
    pos_np = pos.cpu().numpy()
    layers = range(inp["idx"].shape[0]) if layers is None else layers
    out = []
    for l in layers:
        out.append(O.map_layer(
            src, inp["idx"][l], np32(inp["W_K"][l]), np32(inp["W_V"][l]),
            None if inp["b_K"] is None else np32(inp["b_K"][l]),
            None if inp["b_V"] is None else np32(inp["b_V"][l]),
            inp["rope_src"], inp["rope_tgt"], pos_np))
    return np.stack(out)


def rel_errors(got, want):
    """relative Frobenius error per (layer, K|V, head) tensor: array [L, 2, H]."""
    g = got.astype(np.float64)
    diff = np.sqrt(((g - want) ** 2).sum(axis=(-1, -2)))
    ref = np.sqrt((want ** 2).sum(axis=(-1, -2)))
    return np.where(ref > 0, diff / np.where(ref > 0, ref, 1.0), diff)


def assert_parity(got, want, tol, label=""):
    err = rel_errors(got, want)
    worst = np.unravel_index(np.argmax(err), err.shape)
    log(f"[parity] {label}: max relF {err.max():.3e} at (l,kv,h)={tuple(int(x) for x in worst)}, "
        f"median {np.median(err):.3e}, tol {tol:.0e}")
    assert np.isfinite(got).all(), f"{label}: non-finite output"
    assert err.max() <= tol, f"{label}: relF {err.max():.3e} > {tol:.0e}"
    return err


def sample_tokens(T, n, seed, extra=()):
    """First 16, last 16, the given extra rows and a seeded random subset."""
    rng = np.random.default_rng(seed)
    base = set(range(min(16, T))) | set(range(max(0, T - 16), T)) | {int(e) for e in extra if 0 <= e < T}
    pool = np.setdiff1d(np.arange(T), np.fromiter(base, int))
    take = max(0, min(n - len(base), len(pool)))
    pick = rng.choice(pool, size=take, replace=False) if take else np.array([], int)
    return np.sort(np.concatenate([np.fromiter(base, int), pick]).astype(np.int64))
