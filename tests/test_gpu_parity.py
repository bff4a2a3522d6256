"""Parity of the HIP path (through the C ABI) with the fp64 oracle.

Small cases are compared on every element; the full-size workloads are run
in the same launch configuration the benchmark uses and compared on a seeded
token sample that includes the first and last rows, plus every row of a few
whole tensors.  Bar: relative Frobenius error per (layer, head, K|V) tensor
<= 3e-3 for bf16 I/O with fp32 accumulation, <= 1e-5 for fp32 I/O.
"""

import numpy as np
import pytest
import torch

from paper_2608_03893_amd import synth
from tests._parity import (TOL, assert_parity, log, np32, oracle_rows, run_gpu,
                           sample_tokens)

pytestmark = pytest.mark.gpu

DEV = "cuda:0"

SMALL = {
    "tiny_f32": synth.CONFIGS["tiny"],
    "tiny_bf16": synth.CONFIGS["tiny"].replace(dtype="bf16"),
    "tiny_f32_interleaved": synth.CONFIGS["tiny"].replace(
        rope_src=synth.rope_dict(1e4, style=1), rope_tgt=synth.rope_dict(1e4, style=1)),
    "tiny_bf16_interleaved_bias": synth.CONFIGS["tiny"].replace(
        dtype="bf16", bias="normal", rope_src=synth.rope_dict(1e4, style=1),
        rope_tgt=synth.rope_dict(1e4, style=1)),
    "tiny_f32_rebase_llama": synth.CONFIGS["tiny"].replace(
        rope_src=synth.rope_dict(1e4),
        rope_tgt=synth.rope_dict(5e5, factor=8.0, low_freq_factor=1.0, high_freq_factor=4.0,
                                 original_max_pos=8192)),
    "tiny_f32_d128_ragged": synth.CONFIGS["tiny"].replace(d=128, T=203, k=3, bias="normal"),
    "qwen3_0.6b_4b_T333": synth.CONFIGS["qwen3_0.6b_4b"].replace(T=333),
    "qwen3_14b_32b_T200_bias": synth.CONFIGS["qwen3_14b_32b"].replace(T=200),
    "llama_T130_positions_far": synth.CONFIGS["llama3.1_8b_70b"].replace(T=130, L_t=12),
    "bf16_T1": synth.CONFIGS["qwen3_0.6b_4b"].replace(T=1, L_t=4),
    "f32_d128_k1": synth.CONFIGS["tiny"].replace(d=128, k=1, T=65),
    # bf16, d = 128, k <= 4: the W-stationary kernel
    "w_k1_T300": synth.CONFIGS["qwen3_0.6b_4b"].replace(k=1, T=300, L_t=6),
    "w_k2_T513_bias": synth.CONFIGS["qwen3_14b_32b"].replace(k=2, T=513, L_t=6, L_s=9),
    "w_interleaved_k3_bias": synth.CONFIGS["qwen3_14b_32b"].replace(
        k=3, T=290, L_t=6, L_s=10, rope_src=synth.rope_dict(1e6, style=1),
        rope_tgt=synth.rope_dict(1e6, style=1)),
    "w_rebase_k4": synth.CONFIGS["qwen3_14b_32b"].replace(
        T=260, L_t=6, rope_src=synth.rope_dict(1e4),
        rope_tgt=synth.rope_dict(5e5, factor=8.0, original_max_pos=8192)),
    "w_H3_generic_order": synth.CONFIGS["qwen3_14b_32b"].replace(H=3, T=270, L_t=5),
}


@pytest.mark.parametrize("name", list(SMALL))
def test_small_full_parity(gpu_kvx, name):
    cfg = SMALL[name]
    log(f"[case] {name}: {cfg}")
    inp = synth.make_inputs(cfg, DEV)
    if name == "llama_T130_positions_far":
        # large positions: the angle reduction must hold far from 0
        inp["positions"] = inp["positions"] + 60000
    out = run_gpu(gpu_kvx, inp)
    want = oracle_rows(inp)
    assert_parity(np32(out), want, TOL[cfg.dtype], name)


@pytest.mark.parametrize("tokens_per_wg", ["256", "512", "1024"])
def test_w_kernel_token_ranges(gpu_kvx, tokens_per_wg, monkeypatch):
    """Several workgroups per task (ragged last range): parity, and bit-identical
    results for every split of the token axis."""
    cfg = synth.CONFIGS["qwen3_14b_32b"].replace(T=777, L_t=5)
    inp = synth.make_inputs(cfg, DEV)
    ref = run_gpu(gpu_kvx, inp)                    # default split (one range)
    monkeypatch.setenv("KVX_TOKENS_PER_WG", tokens_per_wg)
    out = run_gpu(gpu_kvx, inp)
    assert torch.equal(out.view(torch.int16), ref.view(torch.int16))
    assert_parity(np32(out), oracle_rows(inp), TOL["bf16"], f"ranges of {tokens_per_wg}")


def test_tile_and_w_kernels_agree_with_oracle(gpu_kvx, monkeypatch):
    cfg = synth.CONFIGS["qwen3_14b_32b"].replace(T=400, L_t=4)
    inp = synth.make_inputs(cfg, DEV)
    want = oracle_rows(inp)
    w = run_gpu(gpu_kvx, inp)
    monkeypatch.setenv("KVX_KERNEL", "tile")
    tile = run_gpu(gpu_kvx, inp)
    assert_parity(np32(w), want, TOL["bf16"], "W-stationary kernel")
    assert_parity(np32(tile), want, TOL["bf16"], "tile kernel")


SWEEP = {
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
}


@pytest.mark.parametrize("name", list(SWEEP))
def test_sweep_kernel_matches_w_kernel(gpu_kvx, name, monkeypatch):
    """The layer-sweep kernel is bit-identical to the W-stationary kernel (same
    roundings, same accumulation order) and matches the oracle: several layer
    groups, idle CU slots, odd layer counts, head counts that leave XCDs idle,
    ragged and single-token tiles."""
    cfg = SWEEP[name]
    log(f"[case] sweep {name}: {cfg}")
    inp = synth.make_inputs(cfg, DEV)
    monkeypatch.setenv("KVX_KERNEL", "w")
    ref = run_gpu(gpu_kvx, inp)
    monkeypatch.setenv("KVX_KERNEL", "sweep")
    out = torch.full_like(ref, 5.0)
    run_gpu(gpu_kvx, inp, out=out)
    assert torch.equal(out.view(torch.int16), ref.view(torch.int16)), name
    assert_parity(np32(out), oracle_rows(inp), TOL["bf16"], f"sweep {name}")


def test_sweep_kernel_map_layer_and_slots(gpu_kvx, monkeypatch):
    """map_layer (one target layer: the token axis is split over the CU slots)
    and the slot-addressed target through the sweep kernel."""
    cfg = synth.CONFIGS["qwen3_32b_14b_multiturn"].replace(
        sessions=4, new_len=(40, 300), prior_len=(0, 50), L_s=12, L_t=40)
    inp = synth.make_inputs(cfg, DEV)
    lay = inp["paged"]
    S = lay["num_slots"]
    pools = {}
    for kern in ("w", "sweep"):
        monkeypatch.setenv("KVX_KERNEL", kern)
        pool = torch.full((cfg.L_t, 2, cfg.H, S, cfg.d), -7.0, dtype=inp["src"].dtype, device=DEV)
        gpu_kvx.map_cache_slots(inp["src"], inp["idx"], inp["W_K"], inp["W_V"], inp["b_K"],
                                inp["b_V"], inp["rope_src"], inp["rope_tgt"], inp["positions"],
                                inp["slot_mapping"], pool)
        torch.cuda.synchronize()
        pools[kern] = pool
    assert torch.equal(pools["w"].view(torch.int16), pools["sweep"].view(torch.int16))
    dense = synth.make_inputs(synth.CONFIGS["qwen3_14b_32b"].replace(T=700, L_t=6), DEV)
    monkeypatch.setenv("KVX_KERNEL", "w")
    ref = run_gpu(gpu_kvx, dense)
    monkeypatch.setenv("KVX_KERNEL", "sweep")
    out = torch.full_like(ref, 3.0)
    for l in (0, 5, 2):
        gpu_kvx.map_layer(l, dense["src"], dense["idx"], dense["W_K"], dense["W_V"], dense["b_K"],
                          dense["b_V"], dense["rope_src"], dense["rope_tgt"], dense["positions"], out)
    torch.cuda.synchronize()
    for l in range(6):
        if l in (0, 5, 2):
            assert torch.equal(out[l].view(torch.int16), ref[l].view(torch.int16)), l
        else:
            assert bool((out[l] == 3.0).all()), l


FULL = ["qwen3_0.6b_4b", "qwen3_14b_32b", "llama3.1_8b_70b"]


@pytest.mark.parametrize("name", FULL)
def test_full_size_sampled_parity(gpu_kvx, name):
    cfg = synth.CONFIGS[name]
    log(f"[case] full {name}: generating inputs T={cfg.T}")
    inp = synth.make_inputs(cfg, DEV)
    out = run_gpu(gpu_kvx, inp)
    T = inp["T"]
    tok = sample_tokens(T, 1024, seed=cfg.seed)
    log(f"[case] full {name}: oracle on {len(tok)} sampled rows")
    want = oracle_rows(inp, tokens=tok)
    got = np32(out.index_select(3, torch.as_tensor(tok, device=DEV)))
    assert_parity(got, want, TOL[cfg.dtype], f"{name} sampled")
    # whole-T check of a few tensors
    rng = np.random.default_rng(cfg.seed + 7)
    for l in rng.choice(cfg.L_t, size=2, replace=False):
        want_l = oracle_rows(inp, layers=[int(l)])
        assert_parity(np32(out[int(l):int(l) + 1]), want_l, TOL[cfg.dtype], f"{name} layer {l} all T")
    del out, inp
    torch.cuda.empty_cache()


def test_paged_multiturn_parity(gpu_kvx):
    """Ragged sessions mapped into a paged pool through the slot entry point."""
    cfg = synth.CONFIGS["qwen3_32b_14b_multiturn"].replace(
        sessions=5, new_len=(20, 90), prior_len=(0, 40), L_s=12, L_t=7)
    _paged_case(gpu_kvx, cfg, full=True)


def test_paged_multiturn_full_size_sampled(gpu_kvx):
    _paged_case(gpu_kvx, synth.CONFIGS["qwen3_32b_14b_multiturn"], full=False)


def _paged_case(kvx, cfg, full):
    log(f"[case] paged {cfg.name} sessions={cfg.sessions} full={full}")
    inp = synth.make_inputs(cfg, DEV)
    lay = inp["paged"]
    T = inp["T"]
    S = lay["num_slots"]
    sentinel = -12345.0
    pool = torch.full((cfg.L_t, 2, cfg.H, S, cfg.d), sentinel, dtype=inp["src"].dtype, device=DEV)
    kvx.map_cache_slots(inp["src"], inp["idx"], inp["W_K"], inp["W_V"], inp["b_K"], inp["b_V"],
                        inp["rope_src"], inp["rope_tgt"], inp["positions"],
                        inp["slot_mapping"], pool)
    torch.cuda.synchronize()
    slots = lay["slot_mapping"].astype(np.int64)
    if full:
        tok = np.arange(T)
    else:
        tok = sample_tokens(T, 1024, seed=cfg.seed, extra=lay["cu_seqlens"][:-1])
    want = oracle_rows(inp, tokens=tok)
    got = np32(pool.index_select(3, torch.as_tensor(slots[tok], device=DEV)))
    assert_parity(got, want, TOL[cfg.dtype], f"{cfg.name} paged")
    # slots that no row names keep the sentinel
    untouched = np.setdiff1d(np.arange(S), slots)
    rng = np.random.default_rng(0)
    if len(untouched) > 4096:
        untouched = rng.choice(untouched, 4096, replace=False)
    if len(untouched):
        rest = pool.index_select(3, torch.as_tensor(untouched, device=DEV))
        assert bool((rest == sentinel).all()), "a slot outside slot_mapping was written"
    del pool, inp
    torch.cuda.empty_cache()
