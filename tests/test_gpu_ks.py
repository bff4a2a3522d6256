"""Parity of the k-split layer-sweep kernel (map_ks_kernel) with the fp64
oracle, and its agreement with the layer-sweep kernel.

The k-split kernel adds the bias as the accumulator's initial value and sums two
partial sums per output, so its fp32 sums round in a different order than the sweep kernel's: the two agree to
a small fraction of the tolerance rather than bit for bit.  Cases cover
several layer groups, idle CU slots, odd layer counts, head counts that leave
XCDs idle, one- and 1000-token parts, a ragged last tile, both RoPE layouts,
re-based RoPE, the slot-addressed target and map_layer.
"""

import numpy as np
import pytest
import torch

from paper_2608_03893_amd import synth
from tests._parity import TOL, assert_parity, log, np32, oracle_rows, rel_errors, run_gpu

pytestmark = pytest.mark.gpu

DEV = "cuda:0"

CASES = {
    "k4_L64_bias": synth.CONFIGS["qwen3_14b_32b"].replace(T=300),
    "k3_interleaved_L40": synth.CONFIGS["qwen3_14b_32b"].replace(
        k=3, T=97, L_t=40, L_s=10, rope_src=synth.rope_dict(1e6, style=1),
        rope_tgt=synth.rope_dict(1e6, style=1)),
    "k2_two_groups_L70": synth.CONFIGS["qwen3_14b_32b"].replace(k=2, T=129, L_t=70, L_s=12),
    "k1_H3_L33": synth.CONFIGS["qwen3_14b_32b"].replace(k=1, H=3, T=64, L_t=33, L_s=5),
    "k4_rebase_L80": synth.CONFIGS["llama3.1_8b_70b"].replace(
        T=200, rope_src=synth.rope_dict(1e4),
        rope_tgt=synth.rope_dict(5e5, factor=8.0, original_max_pos=8192)),
    "k4_T1": synth.CONFIGS["qwen3_14b_32b"].replace(T=1),
    "k4_L3": synth.CONFIGS["qwen3_14b_32b"].replace(T=1000, L_t=3),
    "k3_L36_T4099_nobias": synth.CONFIGS["qwen3_0.6b_4b"].replace(T=4099),
    "k4_interleaved_rebase_T77": synth.CONFIGS["qwen3_14b_32b"].replace(
        T=77, L_t=20, rope_src=synth.rope_dict(1e6, style=1),
        rope_tgt=synth.rope_dict(5e5, style=1, factor=8.0, original_max_pos=8192)),
}


@pytest.mark.parametrize("name", list(CASES))
def test_ks_kernel_parity(gpu_kvx, name, monkeypatch):
    cfg = CASES[name]
    log(f"[case] ks {name}: {cfg}")
    inp = synth.make_inputs(cfg, DEV)
    monkeypatch.setenv("KVX_KERNEL", "sweep")
    ref = run_gpu(gpu_kvx, inp)
    monkeypatch.setenv("KVX_KERNEL", "ks")
    out = torch.full_like(ref, 5.0)
    run_gpu(gpu_kvx, inp, out=out)
    want = oracle_rows(inp)
    assert_parity(np32(out), want, TOL["bf16"], f"ks {name}")
    # agreement with the sweep kernel: the same roundings up to the order of
    # the fp32 bias addition
    d = rel_errors(np32(out), np32(ref).astype(np.float64))
    log(f"[case] ks {name}: max relF vs sweep kernel {d.max():.2e}")
    assert d.max() <= 1e-3, name


def test_ks_kernel_slots_and_map_layer(gpu_kvx, monkeypatch):
    """Slot-addressed target (rows outside slot_mapping untouched) and
    map_layer (one layer: the token axis spread over all CU slots)."""
    monkeypatch.setenv("KVX_KERNEL", "ks")
    cfg = synth.CONFIGS["qwen3_32b_14b_multiturn"].replace(
        sessions=4, new_len=(40, 300), prior_len=(0, 50), L_s=12, L_t=40)
    inp = synth.make_inputs(cfg, DEV)
    lay = inp["paged"]
    S = lay["num_slots"]
    sentinel = -7.0
    pool = torch.full((cfg.L_t, 2, cfg.H, S, cfg.d), sentinel, dtype=inp["src"].dtype, device=DEV)
    gpu_kvx.map_cache_slots(inp["src"], inp["idx"], inp["W_K"], inp["W_V"], inp["b_K"],
                            inp["b_V"], inp["rope_src"], inp["rope_tgt"], inp["positions"],
                            inp["slot_mapping"], pool)
    torch.cuda.synchronize()
    slots = lay["slot_mapping"].astype(np.int64)
    got = np32(pool.index_select(3, torch.as_tensor(slots, device=DEV)))
    assert_parity(got, oracle_rows(inp), TOL["bf16"], "ks slots")
    untouched = np.setdiff1d(np.arange(S), slots)
    if len(untouched):
        rest = pool.index_select(3, torch.as_tensor(untouched, device=DEV))
        assert bool((rest == sentinel).all()), "a slot outside slot_mapping was written"

    dense = synth.make_inputs(synth.CONFIGS["qwen3_14b_32b"].replace(T=700, L_t=6), DEV)
    out = torch.full((6, 2, 8, 700, 128), 3.0, dtype=torch.bfloat16, device=DEV)
    for l in (0, 5, 2):
        gpu_kvx.map_layer(l, dense["src"], dense["idx"], dense["W_K"], dense["W_V"], dense["b_K"],
                          dense["b_V"], dense["rope_src"], dense["rope_tgt"], dense["positions"], out)
    torch.cuda.synchronize()
    want = oracle_rows(dense, layers=[0, 5, 2])
    assert_parity(np32(out[[0, 5, 2]]), want, TOL["bf16"], "ks map_layer")
    for l in (1, 3, 4):
        assert bool((out[l] == 3.0).all()), l


SLOT_CASES = {
    "k4_rebased_tgt": dict(k=4, rope_src=synth.rope_dict(1e6),
                           rope_tgt=synth.rope_dict(5e5, factor=8.0, original_max_pos=8192)),
    "k3_interleaved_rebased": dict(k=3, rope_src=synth.rope_dict(1e6, style=1),
                                   rope_tgt=synth.rope_dict(5e5, style=1, factor=8.0,
                                                            original_max_pos=8192)),
    "k1_same_rope": dict(k=1),
}


@pytest.mark.parametrize("name", list(SLOT_CASES))
def test_ks_kernel_slots_rope_variants(gpu_kvx, name, monkeypatch):
    """Slot-addressed target with each RoPE combination (a target RoPE that
    differs from the source one is a kernel variant of its own)."""
    monkeypatch.setenv("KVX_KERNEL", "ks")
    cfg = synth.CONFIGS["qwen3_32b_14b_multiturn"].replace(
        sessions=3, new_len=(30, 200), prior_len=(0, 40), L_s=10, L_t=20, **SLOT_CASES[name])
    inp = synth.make_inputs(cfg, DEV)
    S = inp["paged"]["num_slots"]
    pool = torch.full((cfg.L_t, 2, cfg.H, S, cfg.d), -7.0, dtype=inp["src"].dtype, device=DEV)
    gpu_kvx.map_cache_slots(inp["src"], inp["idx"], inp["W_K"], inp["W_V"], inp["b_K"],
                            inp["b_V"], inp["rope_src"], inp["rope_tgt"], inp["positions"],
                            inp["slot_mapping"], pool)
    torch.cuda.synchronize()
    slots = inp["paged"]["slot_mapping"].astype(np.int64)
    got = np32(pool.index_select(3, torch.as_tensor(slots, device=DEV)))
    assert_parity(got, oracle_rows(inp), TOL["bf16"], f"ks slots {name}")
    untouched = np.setdiff1d(np.arange(S), slots)
    if len(untouched):
        rest = pool.index_select(3, torch.as_tensor(untouched, device=DEV))
        assert bool((rest == -7.0).all()), "a slot outside slot_mapping was written"


def test_ks_kernel_full_size_sampled(gpu_kvx, monkeypatch):
    """The benchmark workload through the k-split kernel, sampled rows and
    two whole layers against the oracle."""
    from tests._parity import sample_tokens
    monkeypatch.setenv("KVX_KERNEL", "ks")
    cfg = synth.CONFIGS["qwen3_14b_32b"]
    inp = synth.make_inputs(cfg, DEV)
    out = run_gpu(gpu_kvx, inp)
    T = inp["T"]
    tok = sample_tokens(T, 1024, seed=cfg.seed)
    want = oracle_rows(inp, tokens=tok)
    got = np32(out.index_select(3, torch.as_tensor(tok, device=DEV)))
    assert_parity(got, want, TOL["bf16"], "ks qwen3_14b_32b sampled")
    for l in (0, 63):
        assert_parity(np32(out[l:l + 1]), oracle_rows(inp, layers=[l]), TOL["bf16"],
                      f"ks qwen3_14b_32b layer {l} all T")
    del out, inp
    torch.cuda.empty_cache()
