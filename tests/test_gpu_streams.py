"""The binding's temporary workspace on a side stream.

A call without a workspace gets a temporary one from the caching allocator.
It must belong to the stream the call is enqueued on, so that the allocator
does not hand its bytes to other work while the tables, the packed maps and
the map kernel still use them.  The test enqueues the map on a side stream
behind a long wait, then immediately allocates and fills memory on the
current stream, and checks the map against the oracle."""

import numpy as np
import pytest
import torch

from paper_2608_03893_amd import synth
from tests._parity import TOL, assert_parity, log, np32, oracle_rows

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


@pytest.mark.parametrize("form", ["per-head", "xhead"])
def test_side_stream_temporary_workspace(gpu_kvx, form):
    cfg = synth.CONFIGS["qwen3_14b_32b"].replace(T=300, L_t=16)
    log(f"[case] side stream, workspace=None, {form}")
    inp = (synth.make_inputs(cfg, DEV) if form == "per-head"
           else synth.make_xhead_inputs(cfg, H_t=cfg.H, device=DEV))
    out = torch.empty((cfg.L_t, 2, cfg.H, cfg.T, cfg.d), dtype=torch.bfloat16, device=DEV)
    side = torch.cuda.Stream(device=DEV)
    # the side stream first runs a long product, so the map's kernels are
    # still queued when the call returns
    big = torch.randn((4096, 4096), device=DEV)
    torch.cuda.synchronize()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for _ in range(8):
            big = big @ big
            big = big / big.norm()
    args = (inp["src"], inp["idx"], inp["W_K"], inp["W_V"], inp["b_K"], inp["b_V"],
            inp["rope_src"], inp["rope_tgt"], inp["positions"], out)
    if form == "per-head":
        gpu_kvx.map_cache(*args, stream=side)
    else:
        gpu_kvx.map_cache_xhead(*args, stream=side)
    # work on the current stream that would overwrite a workspace released
    # to the current stream's pool
    junk = [torch.full((1 << 24,), float("nan"), device=DEV) for _ in range(8)]
    torch.cuda.synchronize()
    del junk, big
    if form == "per-head":
        want = oracle_rows(inp)
    else:
        from tests.test_gpu_xhead import _oracle
        want = _oracle(inp)
    assert_parity(np32(out), want, TOL["bf16"], f"side stream {form}")
    assert np.isfinite(np32(out)).all()
