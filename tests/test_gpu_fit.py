"""Parity of the GPU fit, probe and top-k selection (through the C ABI) with
the fp64 oracle.

The GPU strips keys with fp32 coefficients and rounds each stripped key to
bf16 once, accumulates the Gram matrices in fp32 and solves in fp64; the
oracle works in fp64 throughout on the same bf16 caches.  The tolerances are
the effect of that one bf16 rounding of the stripped keys (the values are
not rounded at all), measured by refitting in the oracle on rounded stripped
keys (tests/test_fit_tolerance.py), with a margin."""

import numpy as np
import pytest
import torch

from oracle import kvx_oracle as O
from paper_2608_03893_amd import synth
from tests._parity import log

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
Q = synth.CONFIGS["qwen3_14b_32b"]
L = synth.CONFIGS["llama3.1_8b_70b"]

# relF per (target layer, head) tensor of W and of b
TOL_FIT = {"K": 1e-3, "V": 1e-3}
TOL_R2 = 5e-4            # absolute, per (source layer, target layer, head, K|V)

FIT_CASES = {
    "k3_rebase_N700": (Q.replace(L_s=6, L_t=4, H=2, k=3, rope_src=synth.rope_dict(1e4),
                                 rope_tgt=synth.rope_dict(1e6)), 700),
    "k4_interleaved_N1000": (Q.replace(L_s=7, L_t=3, H=2, rope_src=synth.rope_dict(1e6, style=1),
                                       rope_tgt=synth.rope_dict(1e6, style=1)), 1000),
    "k1_N300": (Q.replace(L_s=4, L_t=3, H=3, k=1), 300),
    "k2_llama_N513": (L.replace(L_s=5, L_t=4, H=2, k=2), 513),
    # two 8192-token prep chunks, the second ragged: the channel sums are
    # added up from per-chunk partials
    "k2_two_chunks_N8269": (Q.replace(L_s=4, L_t=3, H=2, k=2), 8269),
    "k1_one_chunk_N8192": (Q.replace(L_s=3, L_t=2, H=1, k=1), 8192),
    # every target layer lists the same sources in another order: each source
    # pair is computed once and read transposed by some layers.  N stays well
    # above the k * 128 features: at N = 600 for 512 features the design Gram
    # of these lists has condition 7e5, and fp32 accumulation of the Gram
    # alone moves W_K by relF 5e-3 (an fp64 model of the same roundings)
    "k4_permuted_lists_N1500": (Q.replace(L_s=6, L_t=4, H=2), 1500,
                               [[0, 1, 2, 3], [3, 1, 0, 2], [2, 3, 1, 0], [1, 0, 3, 2]]),
    "k3_shared_unsorted_N1200": (Q.replace(L_s=6, L_t=5, H=2, k=3), 1200,
                                [[5, 1, 2], [2, 5, 0], [1, 2, 5], [0, 4, 3], [3, 0, 1]]),
}


def _np(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def _relF(got, want):
    num = np.sqrt(((got - want) ** 2).sum(axis=tuple(range(2, got.ndim))))
    den = np.sqrt((want ** 2).sum(axis=tuple(range(2, want.ndim))))
    return num / np.where(den > 0, den, 1.0)


@pytest.mark.parametrize("name", list(FIT_CASES))
def test_fit_parity(gpu_kvx, name):
    cfg, N, *lists = FIT_CASES[name]
    log(f"[case] fit {name}: {cfg.L_s}->{cfg.L_t} H={cfg.H} k={cfg.k} N={N}")
    c = synth.make_calibration(cfg, N, DEV)
    if lists:
        c["idx"] = np.asarray(lists[0], dtype=np.int32)
    W_K, W_V, b_K, b_V = gpu_kvx.fit_cache(c["src"], c["idx"], c["tgt"], c["rope_src"],
                                           c["rope_tgt"], c["positions"], lam=0.01)
    torch.cuda.synchronize()
    want = O.fit_cache(_np(c["src"]), c["idx"], _np(c["tgt"]), c["rope_src"], c["rope_tgt"],
                       c["positions"].cpu().numpy(), lam=0.01)
    for name_, got, ref, tol in (("W_K", W_K, want[0], TOL_FIT["K"]), ("W_V", W_V, want[1], TOL_FIT["V"]),
                                 ("b_K", b_K, want[2], TOL_FIT["K"]), ("b_V", b_V, want[3], TOL_FIT["V"])):
        g = _np(got)
        assert np.isfinite(g).all(), name_
        err = _relF(g, ref)
        log(f"[parity] fit {name} {name_}: max relF {err.max():.3e} median {np.median(err):.3e} "
            f"tol {tol:.0e}")
        assert err.max() <= tol, f"{name_} relF {err.max():.3e} > {tol:.0e}"


PROBE_CASES = {
    "probe_rebase_N600": (Q.replace(L_s=5, L_t=4, H=2, rope_src=synth.rope_dict(1e4),
                                    rope_tgt=synth.rope_dict(1e6)), 600),
    "probe_interleaved_llama_N900": (L.replace(L_s=6, L_t=3, H=1,
                                               rope_src=synth.rope_dict(5e5, style=1, factor=8.0),
                                               rope_tgt=synth.rope_dict(5e5, style=1, factor=8.0)), 900),
    "probe_three_chunks_N16500": (Q.replace(L_s=4, L_t=2, H=1), 16500),
    # one target layer: the second workgroup of every task has none; 8193
    # tokens: a second prep chunk of one token (64 padded)
    "probe_one_target_N8193": (Q.replace(L_s=4, L_t=1, H=2), 8193),
}


@pytest.mark.parametrize("name", list(PROBE_CASES))
def test_probe_and_topk_parity(gpu_kvx, name):
    cfg, N = PROBE_CASES[name]
    log(f"[case] probe {name}: {cfg.L_s}->{cfg.L_t} H={cfg.H} N={N}")
    c = synth.make_calibration(cfg, N, DEV)
    r2 = gpu_kvx.probe_r2(c["src"], c["tgt"], c["rope_src"], c["rope_tgt"], c["positions"])
    torch.cuda.synchronize()
    want = O.probe_r2(_np(c["src"]), _np(c["tgt"]), c["rope_src"], c["rope_tgt"],
                      c["positions"].cpu().numpy())
    got = _np(r2)
    err = np.abs(got - want)
    log(f"[parity] probe {name}: max |dR2| keys {err[..., 0].max():.2e} values "
        f"{err[..., 1].max():.2e}; R2 range {want.min():.3f} .. {want.max():.3f}")
    assert np.isfinite(got).all()
    assert err.max() <= TOL_R2
    # the planted mix: each target layer draws on its two mixed source layers
    for k in (1, 2, 3):
        idx = gpu_kvx.select_topk(r2, k)
        torch.cuda.synchronize()
        got_idx = idx.cpu().numpy()
        # the selection is an integer decision: the oracle takes it on the same
        # fp32 R2 values the GPU used, and must agree exactly
        np.testing.assert_array_equal(got_idx, O.select_topk(got.astype(np.float32), k))
        # and on the oracle's own R2 wherever the ranking has a clear margin
        ref_idx = O.select_topk(want, k)
        score = want.mean(axis=(2, 3))
        for l in range(cfg.L_t):
            srt = np.sort(score[:, l])[::-1]
            if k < len(srt) and srt[k - 1] - srt[k] > 10 * TOL_R2:
                assert list(got_idx[l]) == list(ref_idx[l])


def test_fit_then_map_reproduces_planted_structure(gpu_kvx):
    """The fitted maps (rounded to bf16) map the calibration source onto the
    target about as well as the oracle's fit does: the residual sums of
    squares of both fits over the value planes agree to 1%."""
    cfg, N = FIT_CASES["k3_rebase_N700"]
    c = synth.make_calibration(cfg, N, DEV)
    W_K, W_V, b_K, b_V = gpu_kvx.fit_cache(c["src"], c["idx"], c["tgt"], c["rope_src"],
                                           c["rope_tgt"], c["positions"], lam=0.01)
    out = torch.empty_like(c["tgt"])
    gpu_kvx.map_cache(c["src"], c["idx"], W_K.bfloat16(), W_V.bfloat16(), b_K.bfloat16(),
                      b_V.bfloat16(), c["rope_src"], c["rope_tgt"], c["positions"], out)
    torch.cuda.synchronize()
    want = O.fit_cache(_np(c["src"]), c["idx"], _np(c["tgt"]), c["rope_src"], c["rope_tgt"],
                       c["positions"].cpu().numpy(), lam=0.01)
    ref = O.map_cache(_np(c["src"]), c["idx"], *want, c["rope_src"], c["rope_tgt"],
                      c["positions"].cpu().numpy())
    tgt = _np(c["tgt"])
    rss_gpu = ((_np(out) - tgt)[:, 1] ** 2).sum()
    rss_ref = ((ref - tgt)[:, 1] ** 2).sum()
    log(f"[parity] fit->map residual (values): GPU {rss_gpu:.4e} oracle {rss_ref:.4e}")
    assert abs(rss_gpu / rss_ref - 1) < 0.01


def _task_planes(c, l, h, kv, idx):
    """The oracle's design and response of one fit task, float64."""
    pos = c["positions"].cpu().numpy()
    X = []
    for s in idx[l]:
        x = _np(c["src"][int(s), kv, h])
        if kv == 0:
            x = O.rope_rotate(x, pos, c["rope_src"], inverse=True)
        X.append(x)
    Y = _np(c["tgt"][l, kv, h])
    if kv == 0:
        Y = O.rope_rotate(Y, pos, c["rope_tgt"], inverse=True)
    return np.concatenate(X, axis=1), Y


def test_fit_full_size_sampled(gpu_kvx):
    """The Qwen3-14B->32B shape (40 -> 64 layers, 8 heads, k = 4) fitted from
    N = 32768 calibration tokens in one call, as the benchmark times it;
    sixteen seeded (layer, head, K|V) tasks against the oracle.  The bar
    scales with the conditioning of each task's design Gram: fp32 accumulation
    over N tokens perturbs the Gram by about sqrt(N / 16) * 2^-24 relative,
    and the solve multiplies that by the condition number kappa."""
    cfg = Q
    N = 32768
    c = synth.make_calibration(cfg, N, DEV)
    idx = np.asarray(c["idx"])
    W_K, W_V, b_K, b_V = gpu_kvx.fit_cache(c["src"], idx, c["tgt"], c["rope_src"],
                                           c["rope_tgt"], c["positions"], lam=0.01)
    torch.cuda.synchronize()
    rng = np.random.default_rng(17)
    for n in range(16):
        l, h, kv = int(rng.integers(cfg.L_t)), int(rng.integers(cfg.H)), n % 2
        X, Y = _task_planes(c, l, h, kv, idx)
        Wr, br = O.ridge_fit(X, Y, 0.01)
        Xc = X - X.mean(0)
        ev = np.linalg.eigvalsh(Xc.T @ Xc + 0.01 * np.eye(X.shape[1]))
        kappa = ev[-1] / ev[0]
        W = _np((W_K if kv == 0 else W_V)[l, h])
        b = _np((b_K if kv == 0 else b_V)[l, h])
        eW = np.linalg.norm(W - Wr) / np.linalg.norm(Wr)
        eb = np.linalg.norm(b - br) / np.linalg.norm(br)
        bar = max(1e-3, 10 * kappa * np.sqrt(N / 16) * 2.0 ** -24)
        log(f"[parity] fit full-size l={l} h={h} {'KV'[kv]}: relF W {eW:.2e} b {eb:.2e} "
            f"kappa {kappa:.1f} bar {bar:.1e}")
        assert eW <= bar and eb <= bar
    del c, W_K, W_V, b_K, b_V
    torch.cuda.empty_cache()


def test_probe_full_size_sampled(gpu_kvx):
    """The probe over the same shape (40 x 64 layer pairs, 8 heads, N = 32768):
    twenty-four seeded (source layer, target layer, head, K|V) entries against
    the oracle's OLS, and the top-4 lists against the oracle's selection on the
    GPU's R2."""
    cfg = Q
    N = 32768
    c = synth.make_calibration(cfg, N, DEV)
    r2 = gpu_kvx.probe_r2(c["src"], c["tgt"], c["rope_src"], c["rope_tgt"], c["positions"])
    idx = gpu_kvx.select_topk(r2, 4)
    torch.cuda.synchronize()
    got = _np(r2)
    assert np.isfinite(got).all()
    pos = c["positions"].cpu().numpy()
    rng = np.random.default_rng(18)
    worst = 0.0
    for n in range(24):
        s, l, h, kv = (int(rng.integers(cfg.L_s)), int(rng.integers(cfg.L_t)),
                       int(rng.integers(cfg.H)), n % 2)
        x, y = _np(c["src"][s, kv, h]), _np(c["tgt"][l, kv, h])
        if kv == 0:
            x = O.rope_rotate(x, pos, c["rope_src"], inverse=True)
            y = O.rope_rotate(y, pos, c["rope_tgt"], inverse=True)
        want = O.ols_r2(x, y)
        worst = max(worst, abs(got[s, l, h, kv] - want))
    log(f"[parity] probe full-size: max |dR2| {worst:.2e} over 24 sampled entries")
    assert worst <= TOL_R2
    np.testing.assert_array_equal(idx.cpu().numpy(), O.select_topk(got.astype(np.float32), 4))
    # the planted mix: each target layer's two mixed source layers are in its top 4
    top = idx.cpu().numpy()
    hits = np.mean([set(c["mix"][l]) <= set(top[l]) for l in range(cfg.L_t)])
    log(f"[parity] probe full-size: planted source pairs found in the top 4 of {hits:.0%} of layers")
    assert hits >= 0.9
    del c, r2
    torch.cuda.empty_cache()


def test_planes_ready_reuses_the_planes(gpu_kvx):
    """KVX_FLAG_PLANES_READY: a fit (or a probe) that starts from the planes
    and channel sums an earlier fit or probe left in the same workspace gives
    bit-identical results to one that builds them.  Without the prep, the
    fit's block plan takes a launch of its own."""
    cfg, N = Q.replace(L_s=5, L_t=4, H=2, k=3), 700
    c = synth.make_calibration(cfg, N, DEV)
    dims = gpu_kvx.Dims(L_s=cfg.L_s, L_t=cfg.L_t, H=cfg.H, T=N, d=cfg.d, k=cfg.k)
    nb = max(gpu_kvx.fit_workspace_bytes(dims), gpu_kvx.probe_workspace_bytes(dims))
    ws = torch.empty(nb, dtype=torch.uint8, device=DEV)

    def fit(flags):
        out = gpu_kvx.fit_cache(c["src"], c["idx"], c["tgt"], c["rope_src"], c["rope_tgt"],
                                c["positions"], lam=0.01, workspace=ws, flags=flags)
        torch.cuda.synchronize()
        return [t.clone() for t in out]

    def probe(flags):
        r2 = gpu_kvx.probe_r2(c["src"], c["tgt"], c["rope_src"], c["rope_tgt"], c["positions"],
                              workspace=ws, flags=flags)
        torch.cuda.synchronize()
        return r2.clone()

    full = fit(0)
    again = fit(gpu_kvx.FLAG_PLANES_READY)
    r2_full = probe(0)
    after_probe = fit(gpu_kvx.FLAG_PLANES_READY)
    fit(0)
    r2_after_fit = probe(gpu_kvx.FLAG_PLANES_READY)
    for a, b, e in zip(full, again, after_probe):
        assert torch.equal(a, b) and torch.equal(a, e)
    assert torch.equal(r2_full, r2_after_fit)
    log(f"[parity] planes-ready fit and probe bit-identical to full calls (N={N})")
