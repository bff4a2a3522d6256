"""Index lists with repeated source layers (allowed by the ABI; each copy
feeds its own row block of W) through every kernel family, against the fp64
oracle."""

import numpy as np
import pytest
import torch

from oracle import kvx_oracle as O
from paper_2608_03893_amd import synth
from tests._parity import TOL, assert_parity, log, np32, oracle_rows, run_gpu

pytestmark = pytest.mark.gpu

DEV = "cuda:0"

# (config, the kernel the default choice launches for it)
CASES = {
    "ks2_k4": (synth.CONFIGS["qwen3_14b_32b"].replace(T=150, L_t=16, L_s=6), "map_ks2_kernel"),
    "ks_k3": (synth.CONFIGS["qwen3_0.6b_4b"].replace(T=97, L_t=16, L_s=5), "map_ks_kernel"),
    "w_k4": (synth.CONFIGS["qwen3_14b_32b"].replace(T=150, L_t=4, L_s=6), "map_w_kernel"),
    "tile_f32": (synth.CONFIGS["tiny"].replace(k=3, T=70), "map_kernel"),
}


def _with_repeats(idx, L_s):
    """Every row repeats its first entry in its last position; one row is a
    single layer k times."""
    idx = np.array(idx, copy=True)
    idx[:, -1] = idx[:, 0]
    idx[0, :] = L_s - 1
    return np.ascontiguousarray(idx.astype(np.int32))


@pytest.mark.parametrize("name", list(CASES))
def test_repeated_source_layers(gpu_kvx, name, monkeypatch):
    cfg, kern = CASES[name]
    monkeypatch.delenv("KVX_KERNEL", raising=False)
    dims = gpu_kvx.Dims(L_s=cfg.L_s, L_t=cfg.L_t, H=cfg.H, T=cfg.T, d=cfg.d, k=cfg.k)
    assert gpu_kvx.map_kernel_name(dims, cfg.dtype) == kern
    inp = synth.make_inputs(cfg, DEV)
    inp["idx"] = _with_repeats(inp["idx"], cfg.L_s)
    log(f"[case] duplicates {name}: idx rows {inp['idx'][:2].tolist()} ...")
    out = run_gpu(gpu_kvx, inp)
    tol = TOL["f32"] if cfg.dtype == "f32" else TOL["bf16"]
    assert_parity(np32(out), oracle_rows(inp), tol, f"duplicates {name}")


def test_repeated_source_layers_cross_head(gpu_kvx):
    cfg = synth.CONFIGS["qwen3_14b_32b"].replace(L_s=4, L_t=3, H=3, k=3, T=200)
    inp = synth.make_xhead_inputs(cfg, H_t=2, device=DEV)
    idx = _with_repeats(inp["idx"], cfg.L_s)
    out = torch.empty((cfg.L_t, 2, 2, cfg.T, cfg.d), dtype=torch.bfloat16, device=DEV)
    gpu_kvx.map_cache_xhead(inp["src"], idx, inp["W_K"], inp["W_V"], inp["b_K"], inp["b_V"],
                            inp["rope_src"], inp["rope_tgt"], inp["positions"], out)
    torch.cuda.synchronize()
    want = O.map_cache_xhead(np32(inp["src"]), idx, np32(inp["W_K"]), np32(inp["W_V"]),
                             np32(inp["b_K"]), np32(inp["b_V"]), inp["rope_src"],
                             inp["rope_tgt"], inp["positions"].cpu().numpy())
    assert_parity(np32(out), want, TOL["bf16"], "duplicates cross-head")
