"""Seeded synthetic inputs for the KV-cache mapper.

This module only draws random tensors and index lists.  It holds none of the
mapping arithmetic (no RoPE, no gather, no contraction), so both the HIP path
and the fp64 checker can consume what it produces.

The shapes follow the paper's matched-KV family pairs (8 KV heads, head
dimension 128; layer counts of Qwen3 and Llama 3.1 models).  No model caches
or weights are available, so the caches are synthetic stand-ins with a
low-rank-plus-noise structure and a few large key channels, and the mapper
weights are random with the 1/fan-in variance a fitted map of that width
would have.
"""

from __future__ import annotations

import dataclasses
import math
from dataclasses import dataclass, field

import numpy as np
import torch

__all__ = ["MapConfig", "CONFIGS", "make_inputs", "paged_layout", "rope_dict",
           "make_calibration", "make_mlp_inputs"]


def rope_dict(theta, style=0, factor=1.0, low_freq_factor=1.0,
              high_freq_factor=4.0, original_max_pos=8192) -> dict:
    return dict(theta=float(theta), style=int(style), factor=float(factor),
                low_freq_factor=float(low_freq_factor),
                high_freq_factor=float(high_freq_factor),
                original_max_pos=int(original_max_pos))


@dataclass(frozen=True)
class MapConfig:
    """One synthetic mapping workload.

    kv_kind "lognormal": K, V ~ N(0,1) times a per-(layer, K|V, head, channel)
    scale drawn from LogNormal(0, 0.5).
    kv_kind "latent": per (layer, K|V, head) a rank-32 latent Z[T,32] ~ N(0,1)
    times a projection P[32,d] ~ N(0,1/32), plus N(0, 0.1^2) noise; keys get
    4 seeded channels scaled by 10.
    bias: "none" (no bias), "zero" (explicit zeros) or "normal" (N(0,1)).
    Paged workloads (sessions > 0) draw per-session new-turn lengths and
    prior-turn lengths and address the target through a block table.
    """

    name: str
    L_s: int
    L_t: int
    H: int
    d: int
    k: int
    T: int
    dtype: str                      # "f32" | "bf16"
    rope_src: dict
    rope_tgt: dict
    seed: int
    bias: str = "none"
    kv_kind: str = "latent"
    idx_sorted: bool = True
    sessions: int = 0
    new_len: tuple = (0, 0)         # inclusive range of new-turn lengths
    prior_len: tuple = (0, 0)       # inclusive range of prior-turn lengths
    block: int = 16
    note: str = field(default="", compare=False)

    def replace(self, **kw) -> "MapConfig":
        return dataclasses.replace(self, **kw)

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16


_Q_ROPE = rope_dict(1e6)
_LLAMA_ROPE = rope_dict(5e5, factor=8.0, low_freq_factor=1.0,
                        high_freq_factor=4.0, original_max_pos=8192)

CONFIGS = {
    "tiny": MapConfig(
        "tiny", L_s=4, L_t=6, H=2, d=64, k=2, T=256, dtype="f32",
        rope_src=rope_dict(1e4), rope_tgt=rope_dict(1e4), seed=1,
        bias="zero", kv_kind="lognormal", idx_sorted=False,
        note="tiny CPU-checkable map, fp32"),
    "qwen3_0.6b_4b": MapConfig(
        "qwen3_0.6b_4b", L_s=28, L_t=36, H=8, d=128, k=3, T=4096,
        dtype="bf16", rope_src=_Q_ROPE, rope_tgt=_Q_ROPE, seed=2,
        note="Qwen3-0.6B->4B-shaped map"),
    "qwen3_14b_32b": MapConfig(
        "qwen3_14b_32b", L_s=40, L_t=64, H=8, d=128, k=4, T=32768,
        dtype="bf16", rope_src=_Q_ROPE, rope_tgt=_Q_ROPE, seed=3,
        bias="normal", note="Qwen3-14B->32B-shaped map, T=32768"),
    "llama3.1_8b_70b": MapConfig(
        "llama3.1_8b_70b", L_s=32, L_t=80, H=8, d=128, k=4, T=65536,
        dtype="bf16", rope_src=_LLAMA_ROPE, rope_tgt=_LLAMA_ROPE, seed=4,
        note="Llama-3.1-8B->70B-shaped map with Llama-3 frequency scaling"),
    "qwen3_32b_14b_multiturn": MapConfig(
        "qwen3_32b_14b_multiturn", L_s=64, L_t=40, H=8, d=128, k=4, T=0,
        dtype="bf16", rope_src=_Q_ROPE, rope_tgt=_Q_ROPE, seed=5,
        sessions=16, new_len=(2048, 16384), prior_len=(0, 8192), block=16,
        note="Qwen3-32B->14B multi-turn handoff into a paged cache"),
}


def _draw_idx(cfg: MapConfig, rng: np.random.Generator) -> np.ndarray:
    rows = []
    for _ in range(cfg.L_t):
        r = rng.choice(cfg.L_s, size=cfg.k, replace=False)
        rows.append(np.sort(r) if cfg.idx_sorted else r)
    return np.ascontiguousarray(np.stack(rows).astype(np.int32))


def paged_layout(cfg: MapConfig):
    """Sessions, positions and slot addresses of a paged workload (host, int).

    Returns dict(new_lens, prior_lens, cu_seqlens, positions[T], slot_mapping[T],
    block_table (list of int arrays), num_blocks, num_slots).  Physical blocks
    are a seeded permutation shared out across sessions; the slot of position
    p in session s is block_table[s][p // block] * block + p % block.
    """
    rng = np.random.default_rng(cfg.seed + 1000)
    S = cfg.sessions
    new = rng.integers(cfg.new_len[0], cfg.new_len[1] + 1, size=S)
    prior = rng.integers(cfg.prior_len[0], cfg.prior_len[1] + 1, size=S)
    nblk = [int(math.ceil((p + n) / cfg.block)) for p, n in zip(prior, new)]
    total = int(sum(nblk))
    perm = rng.permutation(total).astype(np.int64)
    tables, off = [], 0
    for nb in nblk:
        tables.append(perm[off:off + nb])
        off += nb
    pos, slots = [], []
    for s in range(S):
        p = np.arange(prior[s], prior[s] + new[s], dtype=np.int64)
        pos.append(p)
        slots.append(tables[s][p // cfg.block] * cfg.block + p % cfg.block)
    cu = np.concatenate([[0], np.cumsum(new)]).astype(np.int64)
    return dict(new_lens=new, prior_lens=prior, cu_seqlens=cu,
                positions=np.concatenate(pos).astype(np.int32),
                slot_mapping=np.concatenate(slots).astype(np.int32),
                block_table=tables, num_blocks=total,
                num_slots=total * cfg.block)


def _gen(device, seed):
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def _kv_lognormal(cfg, T, g, device):
    shape = (cfg.L_s, 2, cfg.H, T, cfg.d)
    x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    scale = torch.exp(0.5 * torch.randn((cfg.L_s, 2, cfg.H, 1, cfg.d),
                                        generator=g, device=device))
    return (x * scale).to(cfg.torch_dtype)


def _kv_latent(cfg, T, g, device):
    out = torch.empty((cfg.L_s, 2, cfg.H, T, cfg.d), dtype=cfg.torch_dtype,
                      device=device)
    r = 32
    for s in range(cfg.L_s):
        z = torch.randn((2, cfg.H, T, r), generator=g, device=device)
        p = torch.randn((2, cfg.H, r, cfg.d), generator=g, device=device) / math.sqrt(r)
        layer = torch.matmul(z, p)
        layer += 0.1 * torch.randn(layer.shape, generator=g, device=device)
        # four large key channels per (layer, head)
        ch = torch.stack([torch.randperm(cfg.d, generator=g, device=device)[:4]
                          for _ in range(cfg.H)])              # [H, 4]
        boost = torch.ones((cfg.H, cfg.d), device=device)
        boost.scatter_(1, ch, 10.0)
        layer[0] *= boost[:, None, :]
        out[s].copy_(layer.to(cfg.torch_dtype))
        del z, p, layer
    return out


def make_inputs(cfg: MapConfig, device="cpu") -> dict:
    """Draw every input of one mapping call.

    Returns a dict with torch tensors on ``device``: src [L_s,2,H,T,d],
    W_K, W_V [L_t,H,k*d,d], b_K, b_V [L_t,H,d] or None, positions [T] int32;
    a host int32 array idx [L_t,k]; rope_src / rope_tgt dicts; and for paged
    workloads slot_mapping [T] int32 plus the paged-layout description.
    """
    device = torch.device(device)
    rng = np.random.default_rng(cfg.seed)
    idx = _draw_idx(cfg, rng)
    out = dict(cfg=cfg, idx=idx, rope_src=dict(cfg.rope_src),
               rope_tgt=dict(cfg.rope_tgt))
    if cfg.sessions:
        lay = paged_layout(cfg)
        T = int(lay["positions"].shape[0])
        out["paged"] = lay
        out["positions"] = torch.from_numpy(lay["positions"]).to(device)
        out["slot_mapping"] = torch.from_numpy(lay["slot_mapping"]).to(device)
        out["num_slots"] = lay["num_slots"]
    else:
        T = cfg.T
        out["positions"] = torch.arange(T, dtype=torch.int32, device=device)
    out["T"] = T
    g = _gen(device, cfg.seed)
    if cfg.kv_kind == "lognormal":
        out["src"] = _kv_lognormal(cfg, T, g, device)
    else:
        out["src"] = _kv_latent(cfg, T, g, device)
    kd = cfg.k * cfg.d
    wstd = 1.0 / math.sqrt(kd)
    wshape = (cfg.L_t, cfg.H, kd, cfg.d)
    out["W_K"] = (torch.randn(wshape, generator=g, device=device) * wstd).to(cfg.torch_dtype)
    out["W_V"] = (torch.randn(wshape, generator=g, device=device) * wstd).to(cfg.torch_dtype)
    bshape = (cfg.L_t, cfg.H, cfg.d)
    if cfg.bias == "none":
        out["b_K"] = out["b_V"] = None
    elif cfg.bias == "zero":
        out["b_K"] = torch.zeros(bshape, dtype=cfg.torch_dtype, device=device)
        out["b_V"] = torch.zeros(bshape, dtype=cfg.torch_dtype, device=device)
    else:
        out["b_K"] = torch.randn(bshape, generator=g, device=device).to(cfg.torch_dtype)
        out["b_V"] = torch.randn(bshape, generator=g, device=device).to(cfg.torch_dtype)
    return out


def make_xhead_inputs(cfg: MapConfig, H_t: int | None = None, device="cpu") -> dict:
    """Inputs of one cross-head mapping call: the source cache, index lists,
    positions and RoPEs of ``cfg`` (H_s = cfg.H source heads), with maps
    W_K, W_V [L_t, H_t, k*H_s*d, d] ~ N(0, 1/(k*H_s*d)) and, unless
    cfg.bias is "none", biases [L_t, H_t, d]."""
    if cfg.sessions:
        raise ValueError("the cross-head inputs cover dense workloads only")
    device = torch.device(device)
    H_t = cfg.H if H_t is None else int(H_t)
    rng = np.random.default_rng(cfg.seed)
    out = dict(cfg=cfg, idx=_draw_idx(cfg, rng), rope_src=dict(cfg.rope_src),
               rope_tgt=dict(cfg.rope_tgt), T=cfg.T, H_t=H_t)
    out["positions"] = torch.arange(cfg.T, dtype=torch.int32, device=device)
    g = _gen(device, cfg.seed)
    out["src"] = (_kv_lognormal(cfg, cfg.T, g, device) if cfg.kv_kind == "lognormal"
                  else _kv_latent(cfg, cfg.T, g, device))
    F = cfg.k * cfg.H * cfg.d
    wshape = (cfg.L_t, H_t, F, cfg.d)
    for name in ("W_K", "W_V"):
        w = torch.empty(wshape, dtype=cfg.torch_dtype, device=device)
        for l in range(cfg.L_t):   # one layer at a time keeps the fp32 draw small
            w[l].copy_((torch.randn(wshape[1:], generator=g, device=device)
                        / math.sqrt(F)).to(cfg.torch_dtype))
        out[name] = w
    bshape = (cfg.L_t, H_t, cfg.d)
    if cfg.bias == "none":
        out["b_K"] = out["b_V"] = None
    elif cfg.bias == "zero":
        out["b_K"] = torch.zeros(bshape, dtype=cfg.torch_dtype, device=device)
        out["b_V"] = torch.zeros(bshape, dtype=cfg.torch_dtype, device=device)
    else:
        out["b_K"] = torch.randn(bshape, generator=g, device=device).to(cfg.torch_dtype)
        out["b_V"] = torch.randn(bshape, generator=g, device=device).to(cfg.torch_dtype)
    return out


def make_calibration(cfg: MapConfig, N: int, device="cpu", seed: int | None = None) -> dict:
    """Two models' caches of the same N calibration tokens, for fitting.

    The source cache is drawn as the map's source cache (cfg.kv_kind).  Each
    target (layer, K|V, head) plane is a fresh latent plane of the same kind
    plus a mix of the same head's planes of two seeded source layers, each
    multiplied by a random d x d matrix (in the stored, rotated space), so
    values carry strong linear structure and keys a weaker one, as real
    cross-model caches do.  Positions are 0 .. N-1.  Returns dict(src, tgt,
    positions, idx (the map's index lists of cfg), rope_src, rope_tgt,
    mix [L_t, 2] the two source layers behind each target layer).
    """
    device = torch.device(device)
    seed = cfg.seed + 2000 if seed is None else seed
    rng = np.random.default_rng(seed)
    src_cfg = cfg.replace(T=N)
    g = _gen(device, seed)
    src = (_kv_lognormal(src_cfg, N, g, device) if cfg.kv_kind == "lognormal"
           else _kv_latent(src_cfg, N, g, device))
    tcfg = cfg.replace(L_s=cfg.L_t, T=N)
    tgt = (_kv_lognormal(tcfg, N, g, device) if cfg.kv_kind == "lognormal"
           else _kv_latent(tcfg, N, g, device))
    mix = np.stack([rng.choice(cfg.L_s, size=2, replace=False) for _ in range(cfg.L_t)])
    d = cfg.d
    for l in range(cfg.L_t):
        acc = 0.5 * tgt[l].float()
        for s in mix[l]:
            m = torch.randn((2, cfg.H, d, d), generator=g, device=device) / math.sqrt(d)
            acc = acc + torch.matmul(src[int(s)].float(), m)
        tgt[l].copy_(acc.to(cfg.torch_dtype))
    return dict(cfg=cfg, src=src, tgt=tgt, N=N,
                positions=torch.arange(N, dtype=torch.int32, device=device),
                idx=_draw_idx(cfg, np.random.default_rng(cfg.seed)),
                rope_src=dict(cfg.rope_src), rope_tgt=dict(cfg.rope_tgt), mix=mix)


def make_mlp_inputs(cfg: MapConfig, F: int = 1024, device="cpu") -> dict:
    """Inputs of one MLP-mapper call: the source cache, index lists, positions
    and RoPEs of ``cfg`` (as make_inputs draws them), and for keys and values
    a network per (target layer, head) in nn.Linear's [out, in] layout:
    W1 [L_t, H, F, k*d] ~ N(0, 2/(k*d)), W2 [L_t, H, F, F] ~ N(0, 2/F) (the
    fan-in variance that keeps ReLU activations at the input's scale),
    W3 [L_t, H, d, F] ~ N(0, 1/F), hidden biases ~ N(0, 0.1^2), output bias
    per cfg.bias.  Returns the make_inputs dict without W_K/W_V/b_K/b_V plus
    mlp_K, mlp_V = (W1, b1, W2, b2, W3, b3) and F."""
    if cfg.sessions:
        raise ValueError("the MLP inputs cover dense workloads only")
    if cfg.dtype != "bf16":
        raise ValueError("the MLP mapper runs in bf16")
    device = torch.device(device)
    rng = np.random.default_rng(cfg.seed)
    out = dict(cfg=cfg, idx=_draw_idx(cfg, rng), rope_src=dict(cfg.rope_src),
               rope_tgt=dict(cfg.rope_tgt), T=cfg.T, F=F)
    out["positions"] = torch.arange(cfg.T, dtype=torch.int32, device=device)
    g = _gen(device, cfg.seed)
    out["src"] = (_kv_lognormal(cfg, cfg.T, g, device) if cfg.kv_kind == "lognormal"
                  else _kv_latent(cfg, cfg.T, g, device))
    kd, d, L_t, H = cfg.k * cfg.d, cfg.d, cfg.L_t, cfg.H
    bt = cfg.torch_dtype

    def draw(shape, std):
        w = torch.empty(shape, dtype=bt, device=device)
        for l in range(shape[0]):   # one layer at a time keeps the fp32 draw small
            w[l].copy_((torch.randn(shape[1:], generator=g, device=device) * std).to(bt))
        return w

    for name in ("mlp_K", "mlp_V"):
        W1 = draw((L_t, H, F, kd), math.sqrt(2.0 / kd))
        b1 = draw((L_t, H, F), 0.1)
        W2 = draw((L_t, H, F, F), math.sqrt(2.0 / F))
        b2 = draw((L_t, H, F), 0.1)
        W3 = draw((L_t, H, d, F), math.sqrt(1.0 / F))
        if cfg.bias == "none":
            b3 = None
        elif cfg.bias == "zero":
            b3 = torch.zeros((L_t, H, d), dtype=bt, device=device)
        else:
            b3 = draw((L_t, H, d), 1.0)
        out[name] = (W1, b1, W2, b2, W3, b3)
    return out
