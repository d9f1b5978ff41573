#!/usr/bin/env python3
"""Throughput of Archer cached-prompt diffusion-LM decoding on one MI355X.

One bench step = one archer_decode call: Algorithm 1 end to end over one
batch of synthetic input -- the initial full forward, T denoising decisions,
and before each later forward a refresh (FullForward, new prompt K/V cache)
or a cached forward (CachedForward over the response rows only), chosen by
the refresh rule.  Inputs are resident in HBM before the timed region.

Reported (one JSON line on stdout):
  value                  denoising steps/s = steps * T / wall
  response_tok_per_s     completed response tokens/s = steps * B * G / wall
  speedup_vs_full_refresh  wall(refresh every step) / wall(Archer), same inputs and T
  roofline               the kernel class with the most time in the timed region,
                         algorithmic bytes (or flops) / its HIP-event time
  cpu_baseline           the oracle on this host's cores on a bounded sample

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--policy age|hamming|always]
"""

from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
PEAK_BF16_TFLOPS = 2500.0
PEAK_FP32_TFLOPS = 157.3

# kernel symbol of each timed class as rocprofv3 names it (tile shapes of csrc/gemm.hip)
KERNEL_OF_CLASS = {
    "gemm_qkv": "gemm_bf16_kernel<128, 64, 3>", "gemm_o": "gemm_bf16_kernel<128, 64, 1>",
    "gemm_gateup": "gemm_bf16_kernel<128, 64, 2>", "gemm_down": "gemm_bf16_kernel<128, 64, 1>",
    "gemm_head": "gemm_bf16_kernel<128, 64, 0>", "attn": "attn_bf16_kernel<128>",
    "attn_merge": "attn_merge_kernel<bf16>", "norm": "rmsnorm_kernel<bf16>", "embed": "embed_kernel<bf16>",
    "decide": "rowstats_kernel + select_kernel",
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def cpu_baseline(w, lens, T, K_refresh, policy):
    """Time the oracle (as it is) on one layer at the workload's shapes and extrapolate."""
    import dataclasses

    import numpy as np

    from oracle import decoder as od
    from oracle import model as om
    from oracle import numerics as on
    from synth.gen import model_weights, prompts

    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        cores = os.cpu_count() or 1
    m1 = dataclasses.replace(w.model, n_layers=1)
    log("cpu baseline: generating one layer of host weights")
    W = model_weights(m1, seed=w.weight_seed)
    p = prompts(w, lens)[0]
    G = w.decode.resp_len
    g = np.full(G, m1.mask_id)
    g[: G // 8] = np.arange(G // 8)
    t0 = time.perf_counter()
    z, cache, (hid, c) = om.full_forward(W, m1, p, g, keep_hidden=True)
    t_full1 = time.perf_counter() - t0
    t0 = time.perf_counter()
    zc, _ = om.cached_forward(W, m1, g, cache, len(p))
    t_cached1 = time.perf_counter() - t0
    t0 = time.perf_counter()
    on.linear(c, W["lm_head"])
    t_head = time.perf_counter() - t0
    t0 = time.perf_counter()
    od.decide(zc.astype(np.float32), g, m1.mask_id, w.decode.unmask_per_step, w.decode.remask_threshold)
    t_dec = time.perf_counter() - t0
    L = w.model.n_layers
    t_full = L * max(t_full1 - t_head, 0.0) + t_head
    t_cached = L * max(t_cached1 - t_head, 0.0) + t_head
    R = T if policy == "always" else math.ceil(T / max(K_refresh, 1))
    total = R * t_full + (T - R) * t_cached + T * t_dec
    log(f"cpu baseline: full layer+head {t_full1:.2f}s cached {t_cached1:.2f}s head {t_head:.2f}s "
        f"decide {t_dec:.2f}s -> decode {total:.1f}s extrapolated")
    return {"value": T / total, "unit": "steps/s", "cores": int(cores), "kind": "oracle",
            "sample": (f"one layer of the workload model at full width (FullForward over {len(p) + G} rows, "
                       f"CachedForward over {G} rows, LM head over {G} rows, one decision over {G}x"
                       f"{w.model.vocab} logits), float64 NumPy; extrapolated to {L} layers and the "
                       f"{T}-step schedule with {R} refreshes"),
            "measured_s": round(t_full1 + t_cached1 + t_head + t_dec, 2)}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="llada_p512")
    ap.add_argument("--policy", default="age", choices=["age", "hamming", "always"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-full-refresh", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              f"(asked for --gpus {args.gpus}); run it with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2608_08086_amd import archer
    from synth.device import model_weights_cuda
    from synth.gen import prompt_lengths, prompts
    from synth.workloads import get_workload

    w = get_workload(args.workload)
    m, dec = w.model, w.decode
    B, G, T, k = dec.batch, dec.resp_len, dec.steps, dec.unmask_per_step
    Kr = dec.refresh_every
    lens = prompt_lengths(w)
    pol = {"age": archer.AGE, "hamming": archer.HAMMING, "always": archer.ALWAYS}[args.policy]
    log(f"bench: workload {w.name} B={B} P={lens if len(lens) <= 4 else (min(lens), max(lens))} G={G} T={T} "
        f"k={k} policy={args.policy} K={Kr}")
    t0 = time.perf_counter()
    Wd = model_weights_cuda(m, seed=w.weight_seed)
    torch.cuda.synchronize()
    log(f"bench: device weights ready in {time.perf_counter() - t0:.1f}s")
    ctx = archer.Context(m, Wd, B, max(lens), sum(lens), G)
    prompt = torch.from_numpy(np.concatenate(prompts(w, lens)).astype(np.int32)).cuda()
    resp = torch.full((B, G), m.mask_id, dtype=torch.int32, device="cuda")

    def decode(policy, K):
        resp.fill_(m.mask_id)
        return ctx.decode(prompt, lens, resp, policy=policy, K=K, steps=T, k=k, tau=dec.remask_threshold,
                          trace=True)

    # warm-up, with every kernel class timed once to find the dominant one
    for i in range(args.warmup):
        if i == 0:
            ctx.timing_begin(range(archer.K_COUNT))
        decode(pol, Kr)
        if i == 0:
            warm = ctx.timing_end()
    if args.warmup == 0:
        ctx.timing_begin(range(archer.K_COUNT))
        decode(pol, Kr)
        warm = ctx.timing_end()
    dom = max(warm, key=lambda n: warm[n]["ms"])
    log("bench: warm-up ms per class " + ", ".join(f"{n}={v['ms']:.1f}" for n, v in warm.items() if v["launches"]))

    torch.cuda.synchronize()
    ctx.timing_begin([archer.K_NAMES.index(dom)])
    t0 = time.perf_counter()
    for _ in range(args.steps):
        _, tr = decode(pol, Kr)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    tim = ctx.timing_end()[dom]
    refreshed = int(tr["refreshed"].sum().item())
    log(f"bench: {args.steps} decodes in {wall:.3f}s -> {args.steps * T / wall:.1f} steps/s; "
        f"refreshes per decode {refreshed}/{T * B}")

    full_sps = None
    if not args.no_full_refresh and args.policy != "always":
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        decode(archer.ALWAYS, 0)
        torch.cuda.synchronize()
        full_wall = time.perf_counter() - t0
        full_sps = T / full_wall
        log(f"bench: full refresh every step: {full_sps:.1f} steps/s")

    sps = args.steps * T / wall
    tok = args.steps * B * G / wall
    ai = tim["flops"] / max(tim["bytes"], 1.0)
    peak_f = PEAK_BF16_TFLOPS if m.dtype == "bf16" else PEAK_FP32_TFLOPS
    ridge = peak_f * 1e12 / (PEAK_HBM_GBS * 1e9)
    sec = tim["ms"] / 1e3
    if tim["flops"] > 0 and ai >= ridge:
        roof = {"bound": "mfma", "achieved": round(tim["flops"] / sec / 1e12, 2), "peak": peak_f,
                "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": round(tim["bytes"] / sec / 1e9, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
    roof["traffic"] = None
    roof.update({"kernel": KERNEL_OF_CLASS.get(dom, dom), "class": dom, "launches": tim["launches"],
                 "avg_us": round(tim["ms"] * 1e3 / max(tim["launches"], 1), 2),
                 "algorithmic_bytes_per_launch": round(tim["bytes"] / max(tim["launches"], 1)),
                 "flops_per_launch": round(tim["flops"] / max(tim["launches"], 1)),
                 "mfma_frac": round(tim["flops"] / sec / 1e12 / peak_f, 4)})

    out = {
        "metric": "denoising steps/s + response tok/s at 1 GPU; speedup vs full refresh; % roofline",
        "value": round(sps, 3), "unit": "steps/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(wall / args.steps * 1e3, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": m.dtype,
        "data": "synthetic: seeded random-init weights N(0, 0.02) drawn on the GPU, uniform-random prompt tokens",
        "config": {"workload": f"{w.name}: {w.note}", "batch": B, "prompt_len": lens[0] if len(set(lens)) == 1
                   else [min(lens), max(lens)], "resp_len": G, "denoising_steps_per_decode": T,
                   "unmask_per_step": k, "policy": args.policy, "K": Kr},
        "response_tok_per_s": round(tok, 2),
        "recomputed_positions_per_s": round(tok * T, 1),
        "refresh_fraction": round(refreshed / (T * B), 4),
        "full_refresh_steps_per_s": None if full_sps is None else round(full_sps, 3),
        "speedup_vs_full_refresh": None if full_sps is None else round(sps / full_sps, 3),
        "roofline": roof,
        "warmup_ms_by_class": {n: round(v["ms"], 2) for n, v in warm.items() if v["launches"]},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, lens, T, Kr, args.policy)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
