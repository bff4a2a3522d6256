"""Parity of the k-split kernel with the mid-tile barrier (map_ks2_kernel,
k = 2 and 4) with the fp64 oracle, and its agreement with the layer-sweep
kernel.

Like the k-split kernel it adds the bias as the accumulator's initial value
and sums two partial sums per output, so its fp32 sums round in a different
order than the sweep kernel's: the two agree to a small fraction of the
tolerance rather than bit for bit.  Cases cover several layer groups, idle CU
slots, odd layer counts, head counts that leave XCDs idle, one- and 1000-token
parts, a ragged last tile, both RoPE layouts, re-based RoPE, the
slot-addressed target and map_layer.
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
    "k2_interleaved_L40": synth.CONFIGS["qwen3_14b_32b"].replace(
        k=2, T=97, L_t=40, L_s=10, rope_src=synth.rope_dict(1e6, style=1),
        rope_tgt=synth.rope_dict(1e6, style=1)),
    "k2_two_groups_L70": synth.CONFIGS["qwen3_14b_32b"].replace(k=2, T=129, L_t=70, L_s=12),
    "k4_H16_L33": synth.CONFIGS["qwen3_14b_32b"].replace(H=16, T=64, L_t=33, L_s=5),
    "k4_rebase_L80": synth.CONFIGS["llama3.1_8b_70b"].replace(
        T=200, rope_src=synth.rope_dict(1e4),
        rope_tgt=synth.rope_dict(5e5, factor=8.0, original_max_pos=8192)),
    "k4_T1": synth.CONFIGS["qwen3_14b_32b"].replace(T=1),
    "k4_L17_T1000": synth.CONFIGS["qwen3_14b_32b"].replace(T=1000, L_t=17),
    "k2_L36_T4099_nobias": synth.CONFIGS["qwen3_0.6b_4b"].replace(k=2, T=4099),
    "k4_interleaved_rebase_T77": synth.CONFIGS["qwen3_14b_32b"].replace(
        T=77, L_t=20, rope_src=synth.rope_dict(1e6, style=1),
        rope_tgt=synth.rope_dict(5e5, style=1, factor=8.0, original_max_pos=8192)),
}


@pytest.mark.parametrize("name", list(CASES))
def test_ks2_kernel_parity(gpu_kvx, name, monkeypatch):
    cfg = CASES[name]
    log(f"[case] ks2 {name}: {cfg}")
    inp = synth.make_inputs(cfg, DEV)
    monkeypatch.setenv("KVX_KERNEL", "sweep")
    ref = run_gpu(gpu_kvx, inp)
    monkeypatch.setenv("KVX_KERNEL", "ks2")
    dims = gpu_kvx.Dims(L_s=cfg.L_s, L_t=cfg.L_t, H=cfg.H, T=inp["T"], d=cfg.d, k=cfg.k)
    assert gpu_kvx.map_kernel_name(dims, "bf16") == "map_ks2_kernel", name
    out = torch.full_like(ref, 5.0)
    run_gpu(gpu_kvx, inp, out=out)
    want = oracle_rows(inp)
    assert_parity(np32(out), want, TOL["bf16"], f"ks2 {name}")
    # agreement with the sweep kernel: the same roundings up to the order of
    # the fp32 bias addition
    d = rel_errors(np32(out), np32(ref).astype(np.float64))
    log(f"[case] ks2 {name}: max relF vs sweep kernel {d.max():.2e}")
    assert d.max() <= 1e-3, name


def test_ks2_kernel_slots_and_map_layer(gpu_kvx, monkeypatch):
    """Slot-addressed target (rows outside slot_mapping untouched) and
    map_layer (one layer: the token axis spread over all CU slots)."""
    monkeypatch.setenv("KVX_KERNEL", "ks2")
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
    assert_parity(got, oracle_rows(inp), TOL["bf16"], "ks2 slots")
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
    assert_parity(np32(out[[0, 5, 2]]), want, TOL["bf16"], "ks2 map_layer")
    for l in (1, 3, 4):
        assert bool((out[l] == 3.0).all()), l


SLOT_CASES = {
    "k4_rebased_tgt": dict(k=4, rope_src=synth.rope_dict(1e6),
                           rope_tgt=synth.rope_dict(5e5, factor=8.0, original_max_pos=8192)),
    "k2_interleaved_rebased": dict(k=2, rope_src=synth.rope_dict(1e6, style=1),
                                   rope_tgt=synth.rope_dict(5e5, style=1, factor=8.0,
                                                            original_max_pos=8192)),
    "k4_same_rope": dict(k=4),
}


@pytest.mark.parametrize("name", list(SLOT_CASES))
def test_ks2_kernel_slots_rope_variants(gpu_kvx, name, monkeypatch):
    """Slot-addressed target with each RoPE combination (a target RoPE that
    differs from the source one is a kernel variant of its own)."""
    monkeypatch.setenv("KVX_KERNEL", "ks2")
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
    assert_parity(got, oracle_rows(inp), TOL["bf16"], f"ks2 slots {name}")
    untouched = np.setdiff1d(np.arange(S), slots)
    if len(untouched):
        rest = pool.index_select(3, torch.as_tensor(untouched, device=DEV))
        assert bool((rest == -7.0).all()), "a slot outside slot_mapping was written"


def _banded(L_s, L_t, k):
    """Each target layer lists the k source layers nearest its relative depth
    (neighbouring target layers share most of them)."""
    rows = []
    for l in range(L_t):
        c = int(round(l * (L_s - 1) / max(L_t - 1, 1)))
        lo = min(max(c - k // 2, 0), L_s - k)
        rows.append(list(range(lo + k - 1, lo - 1, -1)) if l % 2 else list(range(lo, lo + k)))
    return rows


# Lists whose target layers share sources: the kernel pairs target layers by
# shared sources, and the second layer of a pair reads a shared source from
# the first layer's slot instead of loading it again.
SHARED_CASES = {
    "k4_banded_L40": (synth.CONFIGS["qwen3_14b_32b"].replace(T=300, L_t=40, L_s=12),
                      _banded(12, 40, 4)),
    "k4_same_permuted_L9": (synth.CONFIGS["qwen3_14b_32b"].replace(T=150, L_t=9, L_s=6),
                            [[3, 1, 4, 0], [0, 3, 1, 4], [4, 0, 3, 1], [1, 4, 0, 3], [3, 4, 1, 0],
                             [0, 1, 4, 3], [1, 3, 0, 4], [4, 3, 0, 1], [3, 1, 4, 0]]),
    "k4_repeats_interleaved_L12": (synth.CONFIGS["qwen3_14b_32b"].replace(
        T=93, L_t=12, L_s=5, rope_src=synth.rope_dict(1e6, style=1),
        rope_tgt=synth.rope_dict(1e6, style=1)),
        [[2, 2, 0, 1], [1, 2, 2, 4], [0, 0, 0, 0], [0, 3, 0, 3], [4, 4, 4, 1], [1, 4, 2, 2],
         [3, 3, 2, 2], [2, 3, 3, 2], [0, 1, 2, 3], [3, 2, 1, 0], [4, 0, 4, 0], [1, 1, 1, 1]]),
    "k2_banded_L70": (synth.CONFIGS["qwen3_14b_32b"].replace(k=2, T=129, L_t=70, L_s=12),
                      _banded(12, 70, 2)),
}


@pytest.mark.parametrize("name", list(SHARED_CASES))
def test_ks2_kernel_shared_sources(gpu_kvx, name, monkeypatch):
    cfg, lists = SHARED_CASES[name]
    log(f"[case] ks2 shared {name}: {cfg}")
    inp = synth.make_inputs(cfg, DEV)
    inp["idx"] = np.asarray(lists, dtype=np.int32)
    assert inp["idx"].shape == (cfg.L_t, cfg.k)
    monkeypatch.setenv("KVX_KERNEL", "ks2")
    dims = gpu_kvx.Dims(L_s=cfg.L_s, L_t=cfg.L_t, H=cfg.H, T=inp["T"], d=cfg.d, k=cfg.k)
    assert gpu_kvx.map_kernel_name(dims, "bf16") == "map_ks2_kernel", name
    out = torch.empty((cfg.L_t, 2, cfg.H, inp["T"], cfg.d), dtype=torch.bfloat16, device=DEV)
    out.fill_(5.0)
    run_gpu(gpu_kvx, inp, out=out)
    assert_parity(np32(out), oracle_rows(inp), TOL["bf16"], f"ks2 shared {name}")


def test_ks2_kernel_full_size_sampled(gpu_kvx, monkeypatch):
    """The benchmark workload through the mid-tile-barrier kernel, sampled rows and
    two whole layers against the oracle."""
    from tests._parity import sample_tokens
    monkeypatch.setenv("KVX_KERNEL", "ks2")
    cfg = synth.CONFIGS["qwen3_14b_32b"]
    inp = synth.make_inputs(cfg, DEV)
    out = run_gpu(gpu_kvx, inp)
    T = inp["T"]
    tok = sample_tokens(T, 1024, seed=cfg.seed)
    want = oracle_rows(inp, tokens=tok)
    got = np32(out.index_select(3, torch.as_tensor(tok, device=DEV)))
    assert_parity(got, want, TOL["bf16"], "ks2 qwen3_14b_32b sampled")
    for l in (0, 63):
        assert_parity(np32(out[l:l + 1]), oracle_rows(inp, layers=[l]), TOL["bf16"],
                      f"ks2 qwen3_14b_32b layer {l} all T")
    del out, inp
    torch.cuda.empty_cache()
