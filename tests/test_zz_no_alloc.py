"""kvx_map_cache_noalloc, the entry point that allocates nothing, against
kvx_map_cache with a caller workspace: the same kernels on the same inputs,
so the outputs must be bit-identical.  Two calls in a row share the device
scratch; the second maps a smaller input, so stale tables or packed maps of
the first call would show."""

import numpy as np
import pytest
import torch

from paper_2608_03893_amd import synth
from tests._parity import log

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _pair(kvx, cfg):
    inp = synth.make_inputs(cfg, DEV)
    shape = (cfg.L_t, 2, cfg.H, inp["T"], cfg.d)
    ref = torch.full(shape, 5.0, dtype=inp["src"].dtype, device=DEV)
    got = torch.full(shape, -5.0, dtype=inp["src"].dtype, device=DEV)
    args = (inp["src"], inp["idx"], inp["W_K"], inp["W_V"], inp["b_K"], inp["b_V"],
            inp["rope_src"], inp["rope_tgt"], inp["positions"])
    kvx.map_cache(*args, ref)
    kvx.map_cache_noalloc(*args, got)
    torch.cuda.synchronize()
    return ref, got


@pytest.mark.parametrize("first,second", [
    (dict(T=300, L_t=16), dict(T=97, L_t=16)),      # map_ks2_kernel, then a shorter cache
    (dict(T=260, L_t=6), dict(T=33, L_t=3, k=2)),   # map_w_kernel, fewer layers and k
])
def test_noalloc_matches_workspace_entry_point(gpu_kvx, first, second):
    base = synth.CONFIGS["qwen3_14b_32b"]
    for n, kw in enumerate((first, second)):
        cfg = base.replace(**kw)
        log(f"[case] noalloc call {n}: {kw}")
        ref, got = _pair(gpu_kvx, cfg)
        assert torch.equal(got.view(torch.int16), ref.view(torch.int16)), f"call {n} differs"
        assert np.isfinite(got.float().cpu().numpy()).all()


def test_noalloc_fp32_and_rejection(gpu_kvx):
    cfg = synth.CONFIGS["tiny"]
    ref, got = _pair(gpu_kvx, cfg)
    assert torch.equal(got.view(torch.int32), ref.view(torch.int32))
    # a workspace beyond the static scratch is refused before any launch
    big = synth.CONFIGS["qwen3_14b_32b"].replace(T=8, L_t=2)
    inp = synth.make_inputs(big, DEV)
    import ctypes
    dims = gpu_kvx.Dims(L_s=40, L_t=2, H=8, T=200000, d=128, k=4)
    assert gpu_kvx.workspace_bytes(dims) > gpu_kvx.SCRATCH_MAX_BYTES
    L = gpu_kvx.load()
    rs = gpu_kvx.make_rope(inp["rope_src"])
    st = L.kvx_map_cache_noalloc(ctypes.byref(dims), 0, None, None, None, None, None, None,
                                 ctypes.byref(rs), ctypes.byref(rs), None, None, 0, None)
    assert st == 7 and b"static scratch" in L.kvx_last_error()
