"""Bit-exact layout, gather and write-set checks of the HIP path.

One-hot maps reveal which source row and channel lands where; sentinel-filled
targets show that nothing outside the intended rows is written; repeated
calls must be bit-identical (no atomics, no split reductions).
"""

import numpy as np
import pytest
import torch

from oracle import kvx_oracle as O
from paper_2608_03893_amd import synth
from tests._parity import TOL, assert_parity, log, np32, oracle_rows, run_gpu

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


def _base(dtype="bf16", d=128, T=100, k=3, L_s=6, L_t=5, H=3, style=0):
    r = synth.rope_dict(1e6, style=style)
    cfg = synth.CONFIGS["qwen3_0.6b_4b"].replace(dtype=dtype, d=d, T=T, k=k, L_s=L_s,
                                                 L_t=L_t, H=H, rope_src=r, rope_tgt=r)
    return synth.make_inputs(cfg, DEV)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("style", [0, 1])
def test_one_hot_probes_select_exact_rows(gpu_kvx, dtype, style):
    """W_V with a single 1 at (block i, channel c) -> column n copies V of source
    layer idx[l][i], channel c, bit for bit.  Keys: the same probe after strip
    and re-apply at equal RoPE returns the source key up to two roundings."""
    inp = _base(dtype=dtype, style=style)
    cfg = inp["cfg"]
    d, k = cfg.d, cfg.k
    rng = np.random.default_rng(3)
    WV = torch.zeros_like(inp["W_V"])
    WK = torch.zeros_like(inp["W_K"])
    probes = {}
    for l in range(cfg.L_t):
        for h in range(cfg.H):
            i = int(rng.integers(k))
            for n in range(d):
                c = int(rng.integers(d))
                WV[l, h, i * d + c, n] = 1.0
                probes[(l, h, n)] = (i, c)
            for n in range(d):
                WK[l, h, i * d + n, n] = 1.0   # identity on block i
            probes[(l, h, "K")] = i
    inp["W_V"], inp["W_K"] = WV, WK
    inp["b_K"] = inp["b_V"] = None
    out = run_gpu(gpu_kvx, inp)
    src = inp["src"]
    for l in range(cfg.L_t):
        for h in range(cfg.H):
            cols = [probes[(l, h, n)] for n in range(d)]
            want = torch.stack([src[inp["idx"][l][i], 1, h, :, c] for i, c in cols], dim=-1)
            assert torch.equal(_bits(out[l, 1, h]), _bits(want)), (l, h)
            i = probes[(l, h, "K")]
            kw = np32(src[inp["idx"][l][i], 0, h])
            err = np.linalg.norm(np32(out[l, 0, h]) - kw) / np.linalg.norm(kw)
            assert err <= TOL[dtype], (l, h, err)


def test_identity_map_values_bit_exact(gpu_kvx):
    inp = _base(k=1)
    cfg = inp["cfg"]
    eye = torch.eye(cfg.d, dtype=inp["W_K"].dtype, device=DEV)
    inp["W_K"] = eye.expand(cfg.L_t, cfg.H, cfg.d, cfg.d).contiguous()
    inp["W_V"] = inp["W_K"].clone()
    inp["b_K"] = inp["b_V"] = None
    out = run_gpu(gpu_kvx, inp)
    for l in range(cfg.L_t):
        s = int(inp["idx"][l][0])
        assert torch.equal(_bits(out[l, 1]), _bits(inp["src"][s, 1]))
        want = np32(inp["src"][s, 0])
        got = np32(out[l, 0])
        assert np.linalg.norm(got - want) / np.linalg.norm(want) <= 3e-3


def test_map_layer_writes_only_its_layer(gpu_kvx):
    inp = _base()
    cfg = inp["cfg"]
    full = run_gpu(gpu_kvx, inp)
    out = torch.full_like(full, 7.0)
    for l in (0, 3):
        gpu_kvx.map_layer(l, inp["src"], inp["idx"], inp["W_K"], inp["W_V"], inp["b_K"],
                          inp["b_V"], inp["rope_src"], inp["rope_tgt"], inp["positions"], out)
    torch.cuda.synchronize()
    for l in range(cfg.L_t):
        if l in (0, 3):
            assert torch.equal(_bits(out[l]), _bits(full[l]))
        else:
            assert bool((out[l] == 7.0).all())


def test_tables_ready_flag_reuses_workspace(gpu_kvx):
    inp = _base()
    cfg = inp["cfg"]
    ref = run_gpu(gpu_kvx, inp)
    from paper_2608_03893_amd import kvx
    dims = kvx.Dims(L_s=cfg.L_s, L_t=cfg.L_t, H=cfg.H, T=inp["T"], d=cfg.d, k=cfg.k)
    ws = torch.empty(kvx.workspace_bytes(dims), dtype=torch.uint8, device=DEV)
    kvx.rope_prepare(inp["positions"], inp["rope_src"], inp["rope_tgt"], cfg.d, ws)
    out = torch.empty_like(ref)
    for l in range(cfg.L_t):
        kvx.map_layer(l, inp["src"], inp["idx"], inp["W_K"], inp["W_V"], inp["b_K"], inp["b_V"],
                      inp["rope_src"], inp["rope_tgt"], inp["positions"], out, workspace=ws,
                      flags=kvx.FLAG_TABLES_READY)
    torch.cuda.synchronize()
    assert torch.equal(_bits(out), _bits(ref))


def test_repeat_calls_are_bit_identical(gpu_kvx):
    inp = _base(T=777)
    a = run_gpu(gpu_kvx, inp)
    b = run_gpu(gpu_kvx, inp)
    assert torch.equal(_bits(a), _bits(b))


def test_empty_token_range_is_a_no_op(gpu_kvx):
    inp = _base(T=0)
    out = torch.empty((inp["cfg"].L_t, 2, inp["cfg"].H, 0, inp["cfg"].d),
                      dtype=inp["src"].dtype, device=DEV)
    run_gpu(gpu_kvx, inp, out=out)


def test_block_order_permutation_matches(gpu_kvx):
    """Permuting the index list with W's row blocks gives the same output."""
    inp = _base(dtype="f32", k=3)
    cfg = inp["cfg"]
    ref = run_gpu(gpu_kvx, inp)
    perm = [2, 0, 1]
    q = dict(inp)
    q["idx"] = inp["idx"][:, perm].copy()
    blk = lambda W: W.reshape(cfg.L_t, cfg.H, 3, cfg.d, cfg.d)[:, :, perm].reshape(W.shape).contiguous()
    q["W_K"], q["W_V"] = blk(inp["W_K"]), blk(inp["W_V"])
    out = run_gpu(gpu_kvx, q)
    # same products, same order of summation within a block: tiny fp32 differences only
    assert_parity(np32(out), np32(ref).astype(np.float64), 1e-6, "block order")


def test_slots_skip_padding_and_out_of_range(gpu_kvx):
    inp = _base(T=40)
    cfg = inp["cfg"]
    S = 64
    slot_np = np.random.default_rng(1).permutation(S)[:40].astype(np.int32)
    slot_np[5] = -1          # padding row
    slot_np[17] = S + 3      # beyond the pool: skipped
    slots = torch.from_numpy(slot_np).to(DEV)
    pool = torch.full((cfg.L_t, 2, cfg.H, S, cfg.d), -3.0, dtype=inp["src"].dtype, device=DEV)
    from paper_2608_03893_amd import kvx
    kvx.map_cache_slots(inp["src"], inp["idx"], inp["W_K"], inp["W_V"], inp["b_K"], inp["b_V"],
                        inp["rope_src"], inp["rope_tgt"], inp["positions"], slots, pool)
    dense = run_gpu(gpu_kvx, inp)
    torch.cuda.synchronize()
    written = set()
    for t in range(40):
        s = int(slot_np[t])
        if 0 <= s < S:
            assert torch.equal(_bits(pool[:, :, :, s]), _bits(dense[:, :, :, t]))
            written.add(s)
    for s in range(S):
        if s not in written:
            assert bool((pool[:, :, :, s] == -3.0).all()), s


def test_weights_packed_flag_reuses_packed_maps(gpu_kvx):
    """A call with KVX_FLAG_WEIGHTS_PACKED (and tables ready) reuses what an
    earlier call left in the workspace, bit for bit; map_layer too."""
    inp = _base(T=300, k=4)
    cfg = inp["cfg"]
    from paper_2608_03893_amd import kvx
    dims = kvx.Dims(L_s=cfg.L_s, L_t=cfg.L_t, H=cfg.H, T=inp["T"], d=cfg.d, k=cfg.k)
    ws = torch.empty(kvx.workspace_bytes(dims), dtype=torch.uint8, device=DEV)
    ref = run_gpu(gpu_kvx, inp, workspace=ws)
    both = kvx.FLAG_TABLES_READY | kvx.FLAG_WEIGHTS_PACKED
    again = run_gpu(gpu_kvx, inp, workspace=ws, flags=both)
    assert torch.equal(_bits(again), _bits(ref))
    out = torch.zeros_like(ref)
    for l in range(cfg.L_t):
        kvx.map_layer(l, inp["src"], inp["idx"], inp["W_K"], inp["W_V"], inp["b_K"], inp["b_V"],
                      inp["rope_src"], inp["rope_tgt"], inp["positions"], out, workspace=ws,
                      flags=both)
    torch.cuda.synchronize()
    assert torch.equal(_bits(out), _bits(ref))
