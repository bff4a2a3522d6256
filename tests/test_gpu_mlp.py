"""Parity of the GPU MLP mapper (Sec. 4.4, through the C ABI) with the fp64
oracle.

The GPU evaluates the networks in bf16 with fp32 accumulation: the stripped
keys, both hidden activations and the output are each rounded once to bf16
(round-to-nearest-even); the oracle evaluates the same bf16 weights and cache
in fp64 without rounding.  With about 1.6e-3 RMS relative error per bf16
rounding, keys carry four roundings (about 3.2e-3 relF) and values three
(about 2.8e-3); tests/test_mlp_tolerance.py replays exactly those roundings
in fp64 on these cases and checks that they stay within the tolerance below
with a margin."""

import numpy as np
import pytest
import torch

from oracle import kvx_oracle as O
from paper_2608_03893_amd import synth
from tests._parity import log

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
Q = synth.CONFIGS["qwen3_14b_32b"]
LL = synth.CONFIGS["llama3.1_8b_70b"]

# relF per (target layer, K|V, head) tensor, against the fp64 oracle
TOL_MLP = 6e-3
# relF against the fp64 replay of the GPU's own bf16 roundings: only fp32
# accumulation order and fp32 RoPE coefficients differ, which flip a rounding
# now and then
TOL_REPLAY = 5e-4

# name -> (config, hidden width F)
MLP_CASES = {
    # ragged token count against the 256- and 512-token tiles, N(0,1) output bias
    "k2_F256_T300": (Q.replace(L_s=4, L_t=3, H=2, k=2, T=300), 256),
    # interleaved pairs with a rebased target theta, no output bias, k = 3
    "k3_interleaved_rebase_F512_T513": (Q.replace(L_s=5, L_t=2, H=2, k=3, T=513, bias="none",
                                                  rope_src=synth.rope_dict(1e4, style=1),
                                                  rope_tgt=synth.rope_dict(1e6, style=1)), 512),
    # one source layer, fewer tokens than one tile
    "k1_F256_T40": (Q.replace(L_s=3, L_t=2, H=1, k=1, T=40, bias="zero"), 256),
    # the largest k built, Llama-3 frequency scaling on both sides
    "k8_llama_F256_T130": (LL.replace(L_s=9, L_t=2, H=1, k=8, T=130), 256),
}


def _np(t):
    return None if t is None else t.detach().float().cpu().numpy().astype(np.float64)


def oracle_nets(net, L_t, H, d):
    """Oracle form of one set of weights: rows = inputs, missing biases as zeros."""
    W1, b1, W2, b2, W3, b3 = (_np(t) for t in net)
    F = W1.shape[2]
    z = lambda b, n: np.zeros((L_t, H, n)) if b is None else b
    return (W1.swapaxes(-1, -2), z(b1, F), W2.swapaxes(-1, -2), z(b2, F), W3.swapaxes(-1, -2),
            z(b3, d))


def oracle_layer(inp, l, tokens=None):
    """fp64 oracle of target layer l [2, H, n, d] on the given token columns."""
    cfg = inp["cfg"]
    src = inp["src"]
    pos = inp["positions"]
    if tokens is not None:
        ti = torch.as_tensor(tokens, device=src.device)
        src = src.index_select(3, ti)
        pos = pos.index_select(0, ti)
    nk = tuple(t[l:l + 1] if t is not None else None for t in inp["mlp_K"])
    nv = tuple(t[l:l + 1] if t is not None else None for t in inp["mlp_V"])
    return O.mlp_map_layer(_np(src), inp["idx"][l], tuple(x[0] for x in oracle_nets(nk, 1, cfg.H, cfg.d)),
                           tuple(x[0] for x in oracle_nets(nv, 1, cfg.H, cfg.d)), inp["rope_src"],
                           inp["rope_tgt"], pos.cpu().numpy())


def _bf16(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(torch.bfloat16).double().numpy()


def bf16_replay_layer(inp, l):
    """Layer l with the GPU's bf16 roundings replayed in fp64: stripped keys,
    both hidden activations and the output rounded once each (RNE)."""
    cfg = inp["cfg"]
    src = _np(inp["src"])
    pos = inp["positions"].cpu().numpy()
    idx = [int(s) for s in inp["idx"][l]]
    xk = np.concatenate([_bf16(O.rope_rotate(src[s, 0], pos, inp["rope_src"], inverse=True))
                         for s in idx], axis=-1)
    xv = np.concatenate([src[s, 1] for s in idx], axis=-1)

    def net(x, p):
        W1, b1, W2, b2, W3, b3 = (t[0] for t in p)
        h1 = _bf16(np.maximum(x @ W1 + b1[:, None, :], 0.0))
        h2 = _bf16(np.maximum(h1 @ W2 + b2[:, None, :], 0.0))
        return h2 @ W3 + b3[:, None, :]
    nk = oracle_nets(tuple(None if t is None else t[l:l + 1] for t in inp["mlp_K"]), 1, cfg.H, cfg.d)
    nv = oracle_nets(tuple(None if t is None else t[l:l + 1] for t in inp["mlp_V"]), 1, cfg.H, cfg.d)
    yk = _bf16(O.rope_rotate(net(xk, nk), pos, inp["rope_tgt"], inverse=False))
    yv = _bf16(net(xv, nv))
    return np.stack([yk, yv], axis=0)


def rel_errors(got, want):
    """relF of every (K|V, head) tensor of one layer: arrays [2, H, n, d]."""
    num = np.sqrt(((got - want) ** 2).sum(axis=(2, 3)))
    den = np.sqrt((want ** 2).sum(axis=(2, 3)))
    return num / np.where(den > 0, den, 1.0)


def _run(gpu_kvx, inp, out=None):
    cfg = inp["cfg"]
    if out is None:
        out = torch.empty((cfg.L_t, 2, cfg.H, inp["T"], cfg.d), dtype=torch.bfloat16, device=DEV)
    gpu_kvx.mlp_map_cache(inp["src"], inp["idx"], inp["mlp_K"], inp["mlp_V"], inp["rope_src"],
                          inp["rope_tgt"], inp["positions"], out)
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("name", list(MLP_CASES))
def test_mlp_parity(gpu_kvx, name):
    cfg, F = MLP_CASES[name]
    log(f"[case] mlp {name}: {cfg.L_s}->{cfg.L_t} H={cfg.H} k={cfg.k} T={cfg.T} F={F}")
    inp = synth.make_mlp_inputs(cfg, F, DEV)
    got = _np(_run(gpu_kvx, inp))
    assert np.isfinite(got).all()
    worst = worst_r = 0.0
    for l in range(cfg.L_t):
        worst = max(worst, float(rel_errors(got[l], oracle_layer(inp, l)).max()))
        worst_r = max(worst_r, float(rel_errors(got[l], bf16_replay_layer(inp, l)).max()))
    log(f"[parity] mlp {name}: max relF {worst:.3e} (tol {TOL_MLP:.0e}); against the bf16 "
        f"replay {worst_r:.3e} (tol {TOL_REPLAY:.0e})")
    assert worst <= TOL_MLP
    assert worst_r <= TOL_REPLAY


def test_mlp_layer_writes_only_its_layer(gpu_kvx):
    cfg, F = MLP_CASES["k2_F256_T300"]
    log("[case] mlp map_layer l=1 into a sentinel-filled target")
    inp = synth.make_mlp_inputs(cfg, F, DEV)
    full = _run(gpu_kvx, inp)
    out = torch.full((cfg.L_t, 2, cfg.H, cfg.T, cfg.d), 7.0, dtype=torch.bfloat16, device=DEV)
    gpu_kvx.mlp_map_layer(1, inp["src"], inp["idx"], inp["mlp_K"], inp["mlp_V"], inp["rope_src"],
                          inp["rope_tgt"], inp["positions"], out)
    torch.cuda.synchronize()
    assert torch.equal(out[1], full[1])
    assert bool((out[0] == 7.0).all()) and bool((out[2] == 7.0).all())


def test_mlp_reuses_stripped_keys_and_tables(gpu_kvx):
    """A second call on the same workspace with the tables and the stripped
    keys flagged as ready gives the same bits."""
    cfg, F = MLP_CASES["k3_interleaved_rebase_F512_T513"]
    log("[case] mlp workspace reuse (tables + stripped keys)")
    inp = synth.make_mlp_inputs(cfg, F, DEV)
    dims = gpu_kvx.Dims(L_s=cfg.L_s, L_t=cfg.L_t, H=cfg.H, T=cfg.T, d=cfg.d, k=cfg.k)
    ws = torch.empty(gpu_kvx.mlp_workspace_bytes(dims, F), dtype=torch.uint8, device=DEV)
    a = torch.empty((cfg.L_t, 2, cfg.H, cfg.T, cfg.d), dtype=torch.bfloat16, device=DEV)
    b = torch.empty_like(a)
    args = (inp["src"], inp["idx"], inp["mlp_K"], inp["mlp_V"], inp["rope_src"], inp["rope_tgt"],
            inp["positions"])
    gpu_kvx.mlp_map_cache(*args, a, workspace=ws)
    gpu_kvx.mlp_map_cache(*args, b, workspace=ws,
                          flags=gpu_kvx.FLAG_TABLES_READY | gpu_kvx.FLAG_KEYS_STRIPPED)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_mlp_empty_call(gpu_kvx):
    cfg, F = MLP_CASES["k1_F256_T40"]
    inp = synth.make_mlp_inputs(cfg.replace(T=0), F, DEV)
    out = torch.empty((cfg.L_t, 2, cfg.H, 0, cfg.d), dtype=torch.bfloat16, device=DEV)
    _run(gpu_kvx, inp, out)


def test_mlp_full_size_sampled(gpu_kvx):
    """The Qwen3-14B -> 32B shape (T = 32768, F = 1024, the launch configuration
    bench.py times): 1024 sampled tokens (both ends, a tile seam and a random
    spread) of four target layers, every head, K and V, against the oracle;
    every output finite."""
    cfg, F = Q, 1024
    log(f"[case] mlp full size {cfg.name} T={cfg.T} F={F}")
    inp = synth.make_mlp_inputs(cfg, F, DEV)
    out = _run(gpu_kvx, inp)
    assert bool(torch.isfinite(out.float()).all())
    rng = np.random.default_rng(11)
    tok = np.unique(np.concatenate([np.arange(0, 64), np.arange(cfg.T - 64, cfg.T),
                                    np.arange(256 * 7 - 32, 256 * 7 + 32),
                                    rng.choice(cfg.T, 1024 - 192, replace=False)]))
    assert tok.size >= 1000
    ti = torch.as_tensor(tok, device=DEV)
    worst = 0.0
    for l in (0, 21, 42, cfg.L_t - 1):
        got = _np(out[l].index_select(2, ti))
        err = rel_errors(got, oracle_layer(inp, l, tok))
        worst = max(worst, float(err.max()))
        log(f"[parity] mlp full size layer {l}: max relF {err.max():.3e}")
    assert worst <= TOL_MLP
