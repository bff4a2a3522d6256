#!/usr/bin/env python3
"""Benchmark of the KV-cache mapper on one MI355X.

One step = one kvx_map_cache call over the whole synthetic cache (RoPE
tables, gather + strip, contraction, bias, re-RoPE, store for every target
layer, head, K and V), inputs resident in HBM.  Prints one JSON line with
mapped tokens/s, the roofline position of the map kernel (timed alone with
HIP events on the launch stream) and the fp64 oracle timed on host cores on
a bounded token sample.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline] [--cpu-full]
    python bench.py --form xhead ...   (the cross-head form on the same workload)
    python bench.py --op fit|probe [--calib-tokens N]   (fitting the mapper, probing layer pairs)
    python bench.py --op mlp [--hidden F]   (the MLP mapper of Sec. 4.4 on the same workload)

The paged multi-turn workload (--workload qwen3_32b_14b_multiturn) times
kvx_map_cache_slots into the paged target pool.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM = 8.0e12         # B/s, MI355X HBM3E
PEAK_BF16 = 2.5e15        # flop/s, dense bf16 matrix cores
PEAK_F32_MFMA = 157.3e12  # flop/s, fp32 matrix/vector peak
METRIC = "mapped KV tokens/sec (all layers x heads) + % of HBM/MFMA roofline"
# sources whose text determines each map kernel's code (traffic figures are
# tied to their hash)
KERNEL_SOURCES = {
    "map_ks2_kernel": ["paper_2608_03893_amd/csrc/kvx_map_ks2.hip",
                       "paper_2608_03893_amd/csrc/kvx_asm.h",
                       "paper_2608_03893_amd/csrc/kvx_bf16.h",
                       "paper_2608_03893_amd/csrc/kvx_internal.h"],
    "map_ks_kernel": ["paper_2608_03893_amd/csrc/kvx_map_ks.hip",
                      "paper_2608_03893_amd/csrc/kvx_asm.h",
                      "paper_2608_03893_amd/csrc/kvx_bf16.h",
                      "paper_2608_03893_amd/csrc/kvx_internal.h"],
    "map_sweep_kernel": ["paper_2608_03893_amd/csrc/kvx_map_sweep.hip",
                         "paper_2608_03893_amd/csrc/kvx_bf16.h",
                         "paper_2608_03893_amd/csrc/kvx_internal.h"],
    "map_w_kernel": ["paper_2608_03893_amd/csrc/kvx_map_bf16.hip",
                     "paper_2608_03893_amd/csrc/kvx_internal.h"],
    "map_kernel": ["paper_2608_03893_amd/csrc/kvx_kernels.hip",
                   "paper_2608_03893_amd/csrc/kvx_internal.h"],
    "gram_kernel": ["paper_2608_03893_amd/csrc/kvx_fit.hip",
                    "paper_2608_03893_amd/csrc/kvx_bf16.h",
                    "paper_2608_03893_amd/csrc/kvx_internal.h",
                    "paper_2608_03893_amd/csrc/kvx_fitplan.h"],
    "mlp_gemm_kernel": ["paper_2608_03893_amd/csrc/kvx_mlp.hip",
                        "paper_2608_03893_amd/csrc/kvx_asm.h",
                        "paper_2608_03893_amd/csrc/kvx_bf16.h",
                        "paper_2608_03893_amd/csrc/kvx_internal.h"],
    "xhead_gemm_kernel": ["paper_2608_03893_amd/csrc/kvx_xhead.hip",
                          "paper_2608_03893_amd/csrc/kvx_asm.h",
                          "paper_2608_03893_amd/csrc/kvx_bf16.h",
                          "paper_2608_03893_amd/csrc/kvx_internal.h"],
}
METRIC_XHEAD = ("cross-head mapped KV tokens/sec (all layers x heads) + % of MFMA roofline")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def kernel_hash(kernel: str) -> str:
    h = hashlib.sha256()
    for p in KERNEL_SOURCES[kernel]:
        h.update(open(os.path.join(ROOT, p), "rb").read())
    return h.hexdigest()[:16]


def algorithmic(cfg, idx, T, has_bias, paged=False):
    """Algorithmic bytes and flops of one full-cache map launch.

    bytes = source layers in the union of the index lists (K and V) + target
    rows written + W_K + W_V + biases + positions (+ the slot of each row for a
    paged target); flops = 2*T*(k*d)*d per (target layer, head, K|V)."""
    import numpy as np
    e = 2 if cfg.dtype == "bf16" else 4
    union = len(np.unique(idx))
    src = union * 2 * cfg.H * T * cfg.d * e
    tgt = cfg.L_t * 2 * cfg.H * T * cfg.d * e
    w = 2 * cfg.L_t * cfg.H * cfg.k * cfg.d * cfg.d * e
    b = 2 * cfg.L_t * cfg.H * cfg.d * e if has_bias else 0
    pos = T * 4 * (2 if paged else 1)
    flops = 2.0 * T * cfg.k * cfg.d * cfg.d * cfg.L_t * cfg.H * 2
    return dict(bytes=src + tgt + w + b + pos, flops=flops, union_layers=union,
                src_bytes=src, tgt_bytes=tgt, w_bytes=w)


def traffic_for(workload, kernel, key="hbm_bytes_per_launch"):
    """Measured HBM bytes per launch (or, with key, per call) from the
    committed counter summary, if it was taken on the current source of this
    kernel; else None."""
    try:
        rec = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    ent = rec.get(workload, {}).get(kernel)
    if not ent or ent.get("kernel_hash") != kernel_hash(kernel):
        return None
    return ent.get(key)


def cpu_info():
    """Host CPU model and the cores this process may use."""
    model = ""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except AttributeError:
        usable = os.cpu_count()
    return dict(cpu_model=model, host_cpus=os.cpu_count(), usable_cpus=usable)


def _blas_threads():
    try:
        from threadpoolctl import threadpool_info
        blas = [p for p in threadpool_info() if p.get("user_api") == "blas"]
        return max([p.get("num_threads", 1) for p in blas] or [1])
    except Exception:
        return 1


def _oracle_rate(inp, budget_s, full):
    """Tokens/s of the fp64 oracle over successive 64-token chunks of the
    workload (all target layers, heads, K and V): the whole workload when
    full, else until budget_s seconds of oracle time are spent."""
    from oracle import kvx_oracle as O
    WK = inp["W_K"].float().cpu().numpy()
    WV = inp["W_V"].float().cpu().numpy()
    bK = None if inp["b_K"] is None else inp["b_K"].float().cpu().numpy()
    bV = None if inp["b_V"] is None else inp["b_V"].float().cpu().numpy()
    chunk, done, spent = 64, 0, 0.0
    while (full or spent < budget_s) and done < inp["T"]:
        n = min(chunk, inp["T"] - done)
        src = inp["src"][:, :, :, done:done + n].float().cpu().numpy()
        pos = inp["positions"][done:done + n].cpu().numpy()
        t0 = time.perf_counter()
        for l in range(inp["idx"].shape[0]):
            O.map_layer(src, inp["idx"][l], WK[l], WV[l], None if bK is None else bK[l],
                        None if bV is None else bV[l], inp["rope_src"], inp["rope_tgt"], pos)
        spent += time.perf_counter() - t0
        done += n
    return done, spent


def cpu_baseline(inp, budget_s, full=False):
    """The fp64 oracle on the host cores: with every BLAS thread, then with
    one thread (a third of the budget).  The oracle's cost is linear in the
    token count, so a sampled run's tokens/s stands for the whole workload."""
    threads = _blas_threads()
    done, spent = _oracle_rate(inp, budget_s, full)
    try:
        from threadpoolctl import threadpool_limits
        with threadpool_limits(limits=1, user_api="blas"):
            done1, spent1 = _oracle_rate(inp, budget_s / 3, full=False)
        rate1 = done1 / spent1
    except Exception:
        done1, rate1 = 0, None
    T = inp["T"]
    whole = done >= T
    return dict(value=done / spent, unit="tokens/s", cores=int(threads), kind="oracle",
                sample=(f"{'all' if whole else 'first'} {done} of {T} tokens in 64-token "
                        f"chunks, all {inp['idx'].shape[0]} target layers x {inp['cfg'].H} heads "
                        f"x K,V; fp64 NumPy; {spent:.1f} s of oracle time"
                        + ("" if whole else "; tokens/s extrapolates to the whole workload, "
                           "the oracle's cost being linear in tokens")),
                seconds=spent, full=bool(whole), extrapolated=not whole,
                threads_all=dict(threads=int(threads), tokens_per_s=done / spent, tokens=done),
                threads_1=dict(threads=1, tokens_per_s=rate1, tokens=done1),
                **cpu_info())


def cpu_baseline_xhead(inp, budget_s):
    """The fp64 oracle of the cross-head form on successive 16-token chunks
    (all target layers, heads, K and V) until budget_s seconds are spent."""
    from oracle import kvx_oracle as O
    try:
        from threadpoolctl import threadpool_info
        blas = [p for p in threadpool_info() if p.get("user_api") == "blas"]
        threads = max([p.get("num_threads", 1) for p in blas] or [1])
    except Exception:
        threads = 1
    L_t = inp["idx"].shape[0]
    chunk, done, spent = 16, 0, 0.0
    while spent < budget_s and done < inp["T"]:
        n = min(chunk, inp["T"] - done)
        src = inp["src"][:, :, :, done:done + n].float().cpu().numpy()
        pos = inp["positions"][done:done + n].cpu().numpy()
        for l in range(L_t):
            WK, WV = inp["W_K"][l].float().cpu().numpy(), inp["W_V"][l].float().cpu().numpy()
            bK = None if inp["b_K"] is None else inp["b_K"][l].float().cpu().numpy()
            bV = None if inp["b_V"] is None else inp["b_V"][l].float().cpu().numpy()
            t0 = time.perf_counter()
            O.map_layer_xhead(src, inp["idx"][l], WK, WV, bK, bV, inp["rope_src"],
                              inp["rope_tgt"], pos)
            spent += time.perf_counter() - t0
        done += n
    return dict(value=done / spent, unit="tokens/s", cores=int(threads), kind="oracle",
                sample=f"first {done} of {inp['T']} tokens in {chunk}-token chunks, all "
                       f"{L_t} target layers x {inp['H_t']} heads x K,V (cross-head form); "
                       f"fp64 NumPy; {spent:.1f} s of oracle time",
                seconds=spent, full=done >= inp["T"], extrapolated=done < inp["T"],
                **cpu_info())


def main_xhead(args, torch, kvx, synth, dev):
    """The cross-head form (every source KV head feeds every target head) on
    the same workload: one kvx_map_cache_xhead call per step."""
    cfg = synth.CONFIGS[args.workload]
    log(f"[bench] generating {cfg.name} (cross-head maps) on {dev}")
    inp = synth.make_xhead_inputs(cfg, H_t=cfg.H, device=dev)
    T, H_t = inp["T"], inp["H_t"]
    out = torch.empty((cfg.L_t, 2, H_t, T, cfg.d), dtype=inp["src"].dtype, device=dev)
    dims = kvx.XDims(L_s=cfg.L_s, L_t=cfg.L_t, H_s=cfg.H, H_t=H_t, T=T, d=cfg.d, k=cfg.k)
    ws = torch.empty(kvx.xhead_workspace_bytes(dims), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev)

    def step(flags=0):
        kvx.map_cache_xhead(inp["src"], inp["idx"], inp["W_K"], inp["W_V"], inp["b_K"],
                            inp["b_V"], inp["rope_src"], inp["rope_tgt"], inp["positions"], out,
                            workspace=ws, flags=flags, stream=stream)

    def timed(flags, n):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        w0 = time.perf_counter()
        e0.record(stream)
        for _ in range(n):
            step(flags)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n, (time.perf_counter() - w0) * 1e3 / n

    log(f"[bench] warmup {args.warmup}")
    for _ in range(args.warmup):
        step()
    log(f"[bench] timing {args.steps} steps")
    ev, wall = timed(0, args.steps)
    ms_step = max(ev, wall)
    # the product kernel alone: tables, packed maps and stripped keys reused
    ms_kernel, _ = timed(kvx.FLAG_TABLES_READY | kvx.FLAG_WEIGHTS_PACKED
                         | kvx.FLAG_KEYS_STRIPPED, args.steps)
    F, N = cfg.k * cfg.H * cfg.d, H_t * cfg.d
    flops = 2.0 * T * F * N * cfg.L_t * 2
    t_k = ms_kernel * 1e-3
    roof = dict(bound="mfma", achieved=flops / t_k / 1e12, peak=PEAK_BF16 / 1e12,
                unit="TFLOP/s")
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["traffic"] = traffic_for(cfg.name + "_xhead", "xhead_gemm_kernel")
    roof["kernel"] = "xhead_gemm_kernel"
    roof["kernel_ms"] = ms_kernel
    roof["alg_flops"] = flops
    roof["roofline_ms"] = flops / PEAK_BF16 * 1e3
    result = {
        "metric": METRIC_XHEAD,
        "value": T / (ms_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {"workload": cfg.name + "_xhead", "L_s": cfg.L_s, "L_t": cfg.L_t,
                   "H_s": cfg.H, "H_t": H_t, "d": cfg.d, "k": cfg.k, "T": T,
                   "bias": inp["b_K"] is not None, "rope_src": cfg.rope_src,
                   "rope_tgt": cfg.rope_tgt},
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        log(f"[bench] oracle on host cores for about {args.cpu_seconds:.0f} s")
        result["cpu_baseline"] = cpu_baseline_xhead(inp, args.cpu_seconds)
    else:
        result["cpu_baseline"] = None
    print(json.dumps(result), flush=True)


METRIC_FIT = "fitted calibration tokens/sec (all layers x heads) + % of MFMA roofline"
METRIC_PROBE = "probed calibration tokens/sec (all layer pairs x heads) + % of MFMA roofline"


def cpu_baseline_fit(c, op, budget_s):
    """The fp64 oracle on a bounded sample of the fit's (target layer, head,
    K|V) tasks, or of the probe's (source layer, target layer, head, K|V)
    entries, on the whole calibration set; the rate is scaled to the whole
    job (the oracle's cost is the same for every task or entry)."""
    import numpy as np
    from oracle import kvx_oracle as O
    cfg, N = c["cfg"], c["N"]
    pos = c["positions"].cpu().numpy()
    idx = np.asarray(c["idx"])
    f = lambda t: t.double().cpu().numpy()
    rng = np.random.default_rng(5)
    done, spent = 0, 0.0
    while spent < budget_s and done < 64:
        kv = done % 2
        h = int(rng.integers(cfg.H))
        if op == "fit":
            l = int(rng.integers(cfg.L_t))
            xs = [f(c["src"][int(sidx), kv, h]) for sidx in idx[l]]
            y = f(c["tgt"][l, kv, h])
            t0 = time.perf_counter()
            if kv == 0:
                xs = [O.rope_rotate(x, pos, c["rope_src"], inverse=True) for x in xs]
                y = O.rope_rotate(y, pos, c["rope_tgt"], inverse=True)
            O.ridge_fit(np.concatenate(xs, axis=1), y, 0.01)
        else:
            sl, l = int(rng.integers(cfg.L_s)), int(rng.integers(cfg.L_t))
            x, y = f(c["src"][sl, kv, h]), f(c["tgt"][l, kv, h])
            t0 = time.perf_counter()
            if kv == 0:
                x = O.rope_rotate(x, pos, c["rope_src"], inverse=True)
                y = O.rope_rotate(y, pos, c["rope_tgt"], inverse=True)
            O.ols_r2(x, y)
        spent += time.perf_counter() - t0
        done += 1
    total = (cfg.L_t * cfg.H * 2) if op == "fit" else (cfg.L_s * cfg.L_t * cfg.H * 2)
    per = spent / done
    what = "(target layer, head, K|V) ridge fits" if op == "fit" else \
        "(source layer, target layer, head, K|V) OLS probes"
    return dict(value=N / (per * total), unit="tokens/s", cores=_blas_threads(), kind="oracle",
                sample=f"{done} of {total} seeded {what} on all {N} calibration tokens, fp64 NumPy, "
                       f"{spent:.1f} s; tokens/s = N / (seconds per task x {total} tasks)",
                seconds=spent, full=False, extrapolated=True, **cpu_info())


def main_fitprobe(args, torch, kvx, synth, dev):
    """The step before the map: fitting the mapper (--op fit) or probing every
    source-target layer pair (--op probe) from calibration caches of N tokens."""
    import numpy as np
    cfg = synth.CONFIGS[args.workload]
    N = args.calib_tokens
    op = args.op
    log(f"[bench] generating calibration caches of {cfg.name}, N={N}, on {dev}")
    c = synth.make_calibration(cfg, N, dev)
    dims = kvx.Dims(L_s=cfg.L_s, L_t=cfg.L_t, H=cfg.H, T=N, d=cfg.d, k=cfg.k)
    stream = torch.cuda.current_stream(dev)
    if op == "fit":
        ws = torch.empty(kvx.fit_workspace_bytes(dims), dtype=torch.uint8, device=dev)
        kd = cfg.k * cfg.d
        outs = (torch.empty((cfg.L_t, cfg.H, kd, cfg.d), dtype=torch.float32, device=dev),
                torch.empty((cfg.L_t, cfg.H, kd, cfg.d), dtype=torch.float32, device=dev),
                torch.empty((cfg.L_t, cfg.H, cfg.d), dtype=torch.float32, device=dev),
                torch.empty((cfg.L_t, cfg.H, cfg.d), dtype=torch.float32, device=dev))

        def step(flags=0):
            kvx.fit_cache(c["src"], c["idx"], c["tgt"], c["rope_src"], c["rope_tgt"],
                          c["positions"], lam=0.01, out=outs, workspace=ws, flags=flags,
                          stream=stream)
        # distinct Gram blocks: a block of two source layers is shared by every
        # target layer whose list holds the pair; cross blocks are per target
        rows = [[int(v) for v in row] for row in np.asarray(c["idx"])]
        pairs = {frozenset((a, b)) for row in rows for a in row for b in row}
        blocks = cfg.H * 2 * (len(pairs) + sum(len(set(row)) for row in rows))
        per_target = cfg.L_t * cfg.H * 2 * (cfg.k * (cfg.k + 1) // 2 + cfg.k)
    else:
        ws = torch.empty(kvx.probe_workspace_bytes(dims), dtype=torch.uint8, device=dev)
        r2 = torch.empty((cfg.L_s, cfg.L_t, cfg.H, 2), dtype=torch.float32, device=dev)
        top = torch.empty((cfg.L_t, cfg.k), dtype=torch.int32, device=dev)

        def step(flags=0):
            kvx.probe_r2(c["src"], c["tgt"], c["rope_src"], c["rope_tgt"], c["positions"],
                         out=r2, workspace=ws, flags=flags, stream=stream)
            kvx.select_topk(r2, cfg.k, out=top, stream=stream)
        blocks = cfg.L_s * cfg.H * 2 * (cfg.L_t + 1)
        per_target = blocks

    def timed(flags, n):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        w0 = time.perf_counter()
        e0.record(stream)
        for _ in range(n):
            step(flags)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n, (time.perf_counter() - w0) * 1e3 / n

    log(f"[bench] warmup {args.warmup}")
    for _ in range(args.warmup):
        step()
    log(f"[bench] timing {args.steps} steps")
    ev, wall = timed(0, args.steps)
    ms_step = max(ev, wall)
    # without the prep pass: the Gram kernel and the solve (fit) or probe kernel
    ms_kernel, _ = timed(kvx.FLAG_PLANES_READY, args.steps)
    flops = 2.0 * N * 128 * 128 * blocks
    alg_bytes = (cfg.L_s + cfg.L_t) * 2 * cfg.H * N * cfg.d * 2
    roof = dict(bound="mfma", achieved=flops / (ms_kernel * 1e-3) / 1e12, peak=PEAK_BF16 / 1e12,
                unit="TFLOP/s")
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["traffic"] = traffic_for(f"{cfg.name}_{op}_N{N}", "gram_kernel")
    roof["kernel"] = "gram_kernel + " + ("fit_solve_kernel" if op == "fit" else "probe_kernel")
    roof["kernel_ms"] = ms_kernel
    roof["prep_ms"] = ms_step - ms_kernel
    roof["alg_flops"] = flops
    roof["alg_bytes"] = alg_bytes
    roof["gram_blocks"] = blocks
    roof["gram_blocks_per_target_layer"] = per_target
    roof["roofline_ms"] = max(flops / PEAK_BF16, alg_bytes / PEAK_HBM) * 1e3
    result = {
        "metric": METRIC_FIT if op == "fit" else METRIC_PROBE,
        "value": N / (ms_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}_{op}", "L_s": cfg.L_s, "L_t": cfg.L_t, "H": cfg.H,
                   "d": cfg.d, "k": cfg.k, "N": N, "lambda": 0.01 if op == "fit" else 0.0,
                   "rope_src": cfg.rope_src, "rope_tgt": cfg.rope_tgt},
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        log(f"[bench] oracle on host cores for about {args.cpu_seconds:.0f} s")
        result["cpu_baseline"] = cpu_baseline_fit(c, op, args.cpu_seconds)
    else:
        result["cpu_baseline"] = None
    print(json.dumps(result), flush=True)


METRIC_MLP = "MLP-mapped KV tokens/sec (all layers x heads) + % of MFMA roofline"


def cpu_baseline_mlp(inp, budget_s):
    """The oracle's MLP mapper on host cores: whole target layers (every head,
    K and V) on consecutive 64-token chunks, about budget_s seconds; tokens/s
    of the whole cache = chunk tokens / (seconds per layer-chunk x L_t)."""
    import numpy as np
    from oracle import kvx_oracle as O
    cfg = inp["cfg"]
    f = lambda t: None if t is None else t.double().cpu().numpy()

    def nets(net, l):
        W1, b1, W2, b2, W3, b3 = (f(t[l]) if t is not None else None for t in net)
        b3 = np.zeros((cfg.H, cfg.d)) if b3 is None else b3
        return (W1.swapaxes(-1, -2), b1, W2.swapaxes(-1, -2), b2, W3.swapaxes(-1, -2), b3)
    chunk = 64
    done, spent, l = 0, 0.0, 0
    while spent < budget_s and done < 100000:
        l = done % cfg.L_t
        t0 = (done * chunk) % (cfg.T - chunk)
        src = f(inp["src"][:, :, :, t0:t0 + chunk])
        pos = inp["positions"][t0:t0 + chunk].cpu().numpy()
        nk, nv = nets(inp["mlp_K"], l), nets(inp["mlp_V"], l)
        w0 = time.perf_counter()
        O.mlp_map_layer(src, inp["idx"][l], nk, nv, inp["rope_src"], inp["rope_tgt"], pos)
        spent += time.perf_counter() - w0
        done += 1
    per_tok_layer = spent / (done * chunk)
    return dict(value=1.0 / (per_tok_layer * cfg.L_t), unit="tokens/s", cores=_blas_threads(),
                kind="oracle",
                sample=f"{done} chunks of {chunk} consecutive tokens, one target layer each (all "
                       f"{cfg.H} heads, K and V), fp64 NumPy, {spent:.1f} s; tokens/s = 1 / "
                       f"(seconds per token per layer x {cfg.L_t} layers)",
                seconds=spent, full=False, extrapolated=True, **cpu_info())


def vendor_gemm_reference(torch, dev, cfg, T, F, reps=20):
    """The MLP layers' plain products through torch.bmm (hipBLASLt), bf16 in
    and out, over the 2H networks of one target layer: a reference point for
    mlp_gemm_kernel, which also gathers, strips, adds biases and applies ReLU
    and the target RoPE.  ms per launch-sized batch, mean of `reps`."""
    nets, kd = 2 * cfg.H, cfg.k * cfg.d
    out = {}
    for name, (K, N) in (("layer1", (kd, F)), ("layer2", (F, F)), ("layer3", (F, cfg.d))):
        g = torch.Generator(device=dev).manual_seed(7)
        x = torch.randn((nets, T, K), device=dev, generator=g).to(torch.bfloat16)
        w = torch.randn((nets, K, N), device=dev, generator=g).to(torch.bfloat16).contiguous()
        y = torch.empty((nets, T, N), device=dev, dtype=torch.bfloat16)
        for _ in range(3):
            torch.bmm(x, w, out=y)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            torch.bmm(x, w, out=y)
        e1.record()
        torch.cuda.synchronize()
        out[name + "_ms"] = e0.elapsed_time(e1) / reps
        del x, w, y
    return out


def main_mlp(args, torch, kvx, synth, dev):
    """The MLP mapper (Sec. 4.4): one kvx_mlp_map_cache call over the whole
    cache per step, synthetic bf16 networks of hidden width F."""
    cfg = synth.CONFIGS[args.workload]
    F = args.hidden
    log(f"[bench] generating {cfg.name} inputs with MLP networks of width {F} on {dev}")
    inp = synth.make_mlp_inputs(cfg, F, dev)
    T = inp["T"]
    dims = kvx.Dims(L_s=cfg.L_s, L_t=cfg.L_t, H=cfg.H, T=T, d=cfg.d, k=cfg.k)
    ws = torch.empty(kvx.mlp_workspace_bytes(dims, F), dtype=torch.uint8, device=dev)
    out = torch.empty((cfg.L_t, 2, cfg.H, T, cfg.d), dtype=torch.bfloat16, device=dev)
    stream = torch.cuda.current_stream(dev)

    def step(flags=0):
        kvx.mlp_map_cache(inp["src"], inp["idx"], inp["mlp_K"], inp["mlp_V"], inp["rope_src"],
                          inp["rope_tgt"], inp["positions"], out, workspace=ws, flags=flags,
                          stream=stream)

    def timed(flags, n):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        w0 = time.perf_counter()
        e0.record(stream)
        for _ in range(n):
            step(flags)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n, (time.perf_counter() - w0) * 1e3 / n

    log(f"[bench] warmup {args.warmup}")
    for _ in range(args.warmup):
        step()
    log(f"[bench] timing {args.steps} steps")
    ev, wall = timed(0, args.steps)
    ms_step = max(ev, wall)
    # the three network layers alone (tables and stripped keys reused)
    ms_kernel, _ = timed(kvx.FLAG_TABLES_READY | kvx.FLAG_KEYS_STRIPPED, args.steps)
    kd = cfg.k * cfg.d
    macs_tok = kd * F + F * F + F * cfg.d
    flops = 2.0 * T * macs_tok * cfg.L_t * cfg.H * 2
    roof = dict(bound="mfma", achieved=flops / (ms_kernel * 1e-3) / 1e12, peak=PEAK_BF16 / 1e12,
                unit="TFLOP/s")
    roof["frac"] = roof["achieved"] / roof["peak"]
    # bytes of the 192 launches of one call, the unit kernel_ms times
    roof["traffic"] = traffic_for(f"{cfg.name}_mlp_F{F}", "mlp_gemm_kernel", "hbm_bytes_per_call")
    roof["kernel"] = "mlp_gemm_kernel (layers 1, 2, 3)"
    roof["kernel_ms"] = ms_kernel
    roof["alg_flops"] = flops
    roof["roofline_ms"] = flops / PEAK_BF16 * 1e3
    result = {
        "metric": METRIC_MLP,
        "value": T / (ms_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}_mlp", "L_s": cfg.L_s, "L_t": cfg.L_t, "H": cfg.H,
                   "d": cfg.d, "k": cfg.k, "T": T, "F": F, "rope_src": cfg.rope_src,
                   "rope_tgt": cfg.rope_tgt},
        "roofline": roof,
    }
    if args.vendor_gemm:
        log("[bench] vendor GEMM (torch.bmm) on the three layer shapes")
        roof["vendor_gemm"] = vendor_gemm_reference(torch, dev, cfg, T, F)
    if not args.no_cpu_baseline:
        log(f"[bench] oracle on host cores for about {args.cpu_seconds:.0f} s")
        result["cpu_baseline"] = cpu_baseline_mlp(inp, args.cpu_seconds)
    else:
        result["cpu_baseline"] = None
    print(json.dumps(result), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", default="qwen3_14b_32b")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-full", action="store_true",
                    help="time the oracle over the whole workload instead of a sample")
    ap.add_argument("--form", choices=("per-head", "xhead"), default="per-head",
                    help="per-head map (default, the headline line) or the cross-head form")
    ap.add_argument("--op", choices=("map", "fit", "probe", "mlp"), default="map",
                    help="map (default, the headline line), the fit / probe that precede it, "
                         "or the MLP mapper")
    ap.add_argument("--hidden", type=int, default=1024, help="hidden width F for --op mlp")
    ap.add_argument("--vendor-gemm", action="store_true",
                    help="--op mlp: also time torch.bmm on the three layer shapes")
    ap.add_argument("--calib-tokens", type=int, default=32768,
                    help="calibration tokens N for --op fit / probe")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the mapper shards by KV head with no exchange, "
              "and this build runs on a single MI355X; use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2608_03893_amd import kvx, synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    kvx.load()
    dev = torch.device("cuda:0")
    if args.op in ("fit", "probe"):
        return main_fitprobe(args, torch, kvx, synth, dev)
    if args.op == "mlp":
        return main_mlp(args, torch, kvx, synth, dev)
    if args.form == "xhead":
        return main_xhead(args, torch, kvx, synth, dev)
    cfg = synth.CONFIGS[args.workload]
    paged = bool(cfg.sessions)
    log(f"[bench] generating {cfg.name} on {dev}")
    inp = synth.make_inputs(cfg, dev)
    T = inp["T"]
    dims = kvx.Dims(L_s=cfg.L_s, L_t=cfg.L_t, H=cfg.H, T=T, d=cfg.d, k=cfg.k)
    ws = torch.empty(max(kvx.workspace_bytes(dims, cfg.dtype), 1), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev)
    if paged:
        # the paged target pool of the multi-turn handoff: new-turn rows go to
        # their sessions' slots, the rest of the pool is left as it was
        out = torch.empty((cfg.L_t, 2, cfg.H, inp["num_slots"], cfg.d), dtype=inp["src"].dtype,
                          device=dev)

        def step(flags=0):
            kvx.map_cache_slots(inp["src"], inp["idx"], inp["W_K"], inp["W_V"], inp["b_K"],
                                inp["b_V"], inp["rope_src"], inp["rope_tgt"], inp["positions"],
                                inp["slot_mapping"], out, workspace=ws, flags=flags, stream=stream)
    else:
        out = torch.empty((cfg.L_t, 2, cfg.H, T, cfg.d), dtype=inp["src"].dtype, device=dev)

        def step(flags=0):
            kvx.map_cache(inp["src"], inp["idx"], inp["W_K"], inp["W_V"], inp["b_K"], inp["b_V"],
                          inp["rope_src"], inp["rope_tgt"], inp["positions"], out, workspace=ws,
                          flags=flags, stream=stream)

    log(f"[bench] warmup {args.warmup}")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"[bench] timing {args.steps} steps")
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms_step = max(e0.elapsed_time(e1), wall * 1e3) / args.steps

    # map kernel alone: tables and packed maps built once, then only the map launches
    step()
    log("[bench] timing the map kernel alone")
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(args.steps):
        step(flags=kvx.FLAG_TABLES_READY | kvx.FLAG_WEIGHTS_PACKED)
    e1.record(stream)
    torch.cuda.synchronize()
    ms_kernel = e0.elapsed_time(e1) / args.steps

    alg = algorithmic(cfg, inp["idx"], T, inp["b_K"] is not None, paged)
    t_k = ms_kernel * 1e-3
    mfma_peak = PEAK_BF16 if cfg.dtype == "bf16" else PEAK_F32_MFMA
    t_hbm, t_mfma = alg["bytes"] / PEAK_HBM, alg["flops"] / mfma_peak
    if t_hbm >= t_mfma:
        roof = dict(bound="hbm", achieved=alg["bytes"] / t_k / 1e9, peak=PEAK_HBM / 1e9,
                    unit="GB/s")
    else:
        roof = dict(bound="mfma", achieved=alg["flops"] / t_k / 1e12, peak=mfma_peak / 1e12,
                    unit="TFLOP/s")
    roof["frac"] = roof["achieved"] / roof["peak"]
    kname = kvx.map_kernel_name(dims, cfg.dtype)
    roof["traffic"] = traffic_for(cfg.name, kname)
    roof["kernel"] = kname
    roof["kernel_ms"] = ms_kernel
    roof["alg_bytes"] = alg["bytes"]
    roof["alg_flops"] = alg["flops"]
    roof["hbm_frac"] = alg["bytes"] / t_k / PEAK_HBM
    roof["mfma_frac"] = alg["flops"] / t_k / mfma_peak
    roof["roofline_ms"] = max(t_hbm, t_mfma) * 1e3

    result = {
        "metric": METRIC,
        "value": T / (ms_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {"workload": cfg.name, "L_s": cfg.L_s, "L_t": cfg.L_t, "H": cfg.H,
                   "d": cfg.d, "k": cfg.k, "T": T, "bias": inp["b_K"] is not None,
                   "rope_src": cfg.rope_src, "rope_tgt": cfg.rope_tgt,
                   "rows_per_s": T * cfg.L_t * cfg.H * 2 / (ms_step * 1e-3)},
        "roofline": roof,
    }
    if paged:
        lay = inp["paged"]
        result["config"].update(sessions=cfg.sessions, block=cfg.block,
                                num_slots=int(inp["num_slots"]),
                                new_lens=[int(x) for x in lay["new_lens"]],
                                prior_lens=[int(x) for x in lay["prior_lens"]])
    if not args.no_cpu_baseline:
        log(f"[bench] oracle on host cores ({'whole workload' if args.cpu_full else f'about {args.cpu_seconds:.0f} s'})")
        result["cpu_baseline"] = cpu_baseline(inp, args.cpu_seconds, full=args.cpu_full)
    else:
        result["cpu_baseline"] = None
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
