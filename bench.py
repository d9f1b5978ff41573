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

# kernel symbol of each timed class for the LLaDA-8B shape as rocprofv3 names it
# (gemm_lds_kernel template arguments: BM, BN, wave grid, stages, epilogue,
# two-term A, split mode; see csrc/gemm_lds.hip)
KERNEL_OF_CLASS = {
    "gemm_qkv": "gemm_lds_kernel<128, 192, 2, 2, 4, 3, true, 2> + gemm_reduce_kernel<3, bf16>",
    "gemm_o": "gemm_lds_kernel<128, 128, 2, 2, 4, 1, true, 2> + gemm_reduce_kernel<1, bf16>",
    "gemm_gateup": "gemm_lds_kernel<128, 192, 2, 2, 4, 2, true, 0>",
    "gemm_down": "gemm_lds_kernel<128, 128, 2, 2, 4, 1, true, 2> + gemm_reduce_kernel<1, bf16>",
    "gemm_head": "gemm_lds_kernel<128, 128, 2, 2, 4, 0, true, 0>",
    "attn": "attn_bf16_kernel<128, QB, NW> + attn_merge_kernel<128> (CachedForward passes)",
    "attn_full": "attn_bf16_kernel<128, QB, NW> + attn_merge_kernel<128> (FullForward passes)",
    "norm": "rmsnorm_kernel<bf16>", "embed": "embed_kernel<bf16>", "decide": "rowstats_kernel + select_kernel",
}
# classes whose bf16 launches multiply two-term activations (two MFMAs per fragment)
TWO_TERM = {"gemm_qkv", "gemm_o", "gemm_gateup", "gemm_down", "gemm_head"}
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_gemm_gateup_llada_p512.json")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def src_hash(paths):
    """First 16 hex digits of the SHA-256 of the concatenated files."""
    import hashlib
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def committed_traffic(cls):
    """HBM bytes per launch from the committed rocprofv3 PMC record, if it
    was taken on the current kernel sources; else None."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
        if rec.get("class") != cls or rec.get("kernel_sources_sha256_16") != src_hash(rec["kernel_sources"]):
            return None
    except (OSError, ValueError, KeyError):
        return None
    return rec.get("hbm_bytes_per_launch")


def cpu_baseline(w, lens, T, K_refresh, policy, sample_layers=9):
    """Time the oracle (as it is) on the first layers of the workload model at
    full width and extrapolate to the whole decode."""
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
    S = min(sample_layers, w.model.n_layers)
    mS = dataclasses.replace(w.model, n_layers=S)
    log(f"cpu baseline: generating {S} layers of host weights")
    W = model_weights(mS, seed=w.weight_seed)
    p = prompts(w, lens)[0]
    G = w.decode.resp_len
    g = np.full(G, mS.mask_id)
    g[: G // 8] = np.arange(G // 8)
    t0 = time.perf_counter()
    z, cache, (hid, c) = om.full_forward(W, mS, p, g, keep_hidden=True)
    t_fullS = time.perf_counter() - t0
    t0 = time.perf_counter()
    zc, _ = om.cached_forward(W, mS, g, cache, len(p))
    t_cachedS = time.perf_counter() - t0
    t0 = time.perf_counter()
    on.linear(c, W["lm_head"])
    t_head = time.perf_counter() - t0
    t0 = time.perf_counter()
    od.decide(zc.astype(np.float32), g, mS.mask_id, w.decode.unmask_per_step, w.decode.remask_threshold)
    t_dec = time.perf_counter() - t0
    L = w.model.n_layers
    t_full = L / S * max(t_fullS - t_head, 0.0) + t_head
    t_cached = L / S * max(t_cachedS - t_head, 0.0) + t_head
    R = T if policy == "always" else math.ceil(T / max(K_refresh, 1))
    total = R * t_full + (T - R) * t_cached + T * t_dec
    measured = t_fullS + t_cachedS + t_head + t_dec
    log(f"cpu baseline: {S}-layer full {t_fullS:.2f}s cached {t_cachedS:.2f}s head {t_head:.2f}s "
        f"decide {t_dec:.2f}s -> decode {total:.1f}s extrapolated")
    return {"value": T / total, "unit": "steps/s", "cores": int(cores), "kind": "oracle",
            "sample": (f"the first {S} layers of the workload model at full width: one FullForward over "
                       f"{len(p) + G} rows, one CachedForward over {G} rows, the LM head over {G} rows and "
                       f"one decision over {G}x{w.model.vocab} logits, float64 NumPy ({measured:.1f} s); "
                       f"per-layer cost extrapolated to {L} layers and the {T}-step schedule with {R} refreshes"),
            "measured_s": round(measured, 2)}


def sweep(kind, reps=10):
    """Per-update and radius sweeps on the LLaDA-8B-shaped random-init model
    (the paper's prompt-length and radius studies, App. F and App. B):
      update:   FullForward vs CachedForward per-update time at G = 256 for
                P in {128, 256, 512, 1024, 2048} (mean of `reps` synchronised calls)
      response: the same at P = 512 for G in {64, 128, 256, 512}
      radius:   whole decodes (P 512, G 256, T 256) under the age and Hamming
                rules for K in {1, 2, 4, 8, 16, 32, never}: steps/s, realised refresh fraction
    Prints one JSON object."""
    import numpy as np
    import torch

    from paper_2608_08086_amd import archer
    from synth.device import model_weights_cuda
    from synth.gen import prompts
    from synth.workloads import get_workload

    w = get_workload("llada_p512")
    m = w.model
    Wd = archer.pack_weights(model_weights_cuda(m, seed=w.weight_seed), drop_source=True)
    torch.cuda.synchronize()

    def timed(fn, n):
        fn()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(n):
            fn()
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) / n * 1e3

    def per_update(P, G):
        ctx = archer.Context(m, Wd, 1, P, P, G)
        wl = w.with_decode(prompt_len=P, resp_len=G)
        prompt = torch.from_numpy(prompts(wl, [P])[0].astype(np.int32)).cuda()
        resp = torch.full((1, G), m.mask_id, dtype=torch.int32, device="cuda")
        resp[0, : G // 4] = torch.arange(G // 4, dtype=torch.int32, device="cuda")
        logits = ctx.new_logits(1)
        full = timed(lambda: ctx.refresh_prompt(prompt, [P], resp, logits=logits), reps)
        cached = timed(lambda: ctx.step(resp, logits=logits), 2 * reps)
        ctx.close()
        return {"P": P, "G": G, "full_ms": round(full, 3), "cached_ms": round(cached, 3),
                "speedup": round(full / cached, 3), "ideal_speedup": round((P + G) / G, 3),
                "measured_over_ideal": round(full / cached / ((P + G) / G), 3)}

    out = {"sweep": kind, "model": "LLaDA-8B shape (32 layers, d 4096, 32 heads x 128, F 12288, V 126464), "
           "bf16, random init", "data": "synthetic"}
    if kind == "update":
        out["rows"] = [per_update(P, 256) for P in (128, 256, 512, 1024, 2048)]
        log(json.dumps(out["rows"]))
    elif kind == "response":
        out["rows"] = [per_update(512, G) for G in (64, 128, 256, 512)]
    elif kind == "radius":
        P, G, T = 512, 256, 256
        ctx = archer.Context(m, Wd, 1, P, P, G)
        prompt = torch.from_numpy(prompts(w, [P])[0].astype(np.int32)).cuda()
        resp = torch.full((1, G), m.mask_id, dtype=torch.int32, device="cuda")
        rows = []
        for pol_name, pol in (("age", archer.AGE), ("hamming", archer.HAMMING)):
            for K in (1, 2, 4, 8, 16, 32, archer.NEVER):
                def run():
                    resp.fill_(m.mask_id)
                    return ctx.decode(prompt, [P], resp, policy=pol, K=K, steps=T, k=1, tau=0.1, trace=True)
                run()
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                _, tr = run()
                torch.cuda.synchronize()
                wall = time.perf_counter() - t0
                q = int(tr["refreshed"].sum().item()) / T
                rows.append({"policy": pol_name, "K": "never" if K == archer.NEVER else K,
                             "steps_per_s": round(T / wall, 2), "decode_s": round(wall, 4),
                             "refresh_fraction": round(q, 4)})
                log(json.dumps(rows[-1]))
        out["rows"] = rows
        out["config"] = {"P": P, "G": G, "T": T, "k": 1, "tau": 0.1}
    else:
        raise SystemExit(f"unknown sweep {kind}")
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="llada_p512")
    ap.add_argument("--policy", default="age", choices=["age", "hamming", "always"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-full-refresh", action="store_true")
    ap.add_argument("--timing-every", type=int, default=7,
                    help="time every n-th launch of the measured kernel classes (1 = all)")
    ap.add_argument("--decode-steps", type=int, default=0,
                    help="profiling only: override the workload's denoising steps per decode")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="profiling only: end with a 1 GiB device copy (known HBM traffic) for PMC scaling")
    ap.add_argument("--sweep", choices=["update", "response", "radius"],
                    help="run a sweep instead of the throughput bench (prints its own JSON object)")
    ap.add_argument("--probe", action="store_true",
                    help="run the cache-validity probe (shadow full forwards at cached steps) on the "
                         "workload instead of the throughput bench (prints its own JSON object)")
    ap.add_argument("--probe-every", type=int, default=4, help="probe every n-th cached forward")
    args = ap.parse_args()
    if args.sweep:
        sweep(args.sweep)
        return
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
    if args.decode_steps:
        T = args.decode_steps
    Kr = dec.refresh_every
    lens = prompt_lengths(w)
    pol = {"age": archer.AGE, "hamming": archer.HAMMING, "always": archer.ALWAYS}[args.policy]
    log(f"bench: workload {w.name} B={B} P={lens if len(lens) <= 4 else (min(lens), max(lens))} G={G} T={T} "
        f"k={k} policy={args.policy} K={Kr}")
    t0 = time.perf_counter()
    Wd = model_weights_cuda(m, seed=w.weight_seed)
    if m.dtype == "bf16":
        # projection matrices in the k-block layout (packed once, outside the timed region)
        Wd = archer.pack_weights(Wd, drop_source=True)
    torch.cuda.synchronize()
    log(f"bench: device weights ready in {time.perf_counter() - t0:.1f}s")
    ctx = archer.Context(m, Wd, B, max(lens), sum(lens), G)
    prompt = torch.from_numpy(np.concatenate(prompts(w, lens)).astype(np.int32)).cuda()
    resp = torch.full((B, G), m.mask_id, dtype=torch.int32, device="cuda")
    if args.probe:
        from paper_2608_08086_amd import probe

        # the shadow context's prompt cache is the scratch cache of the fresh forwards
        shadow = archer.Context(m, Wd, B, max(lens), sum(lens), G)
        t0 = time.perf_counter()
        _, tr, recs = probe.shadow_probe(ctx, shadow, prompt, lens, resp, policy=pol, K=Kr, steps=T, k=k,
                                         tau=dec.remask_threshold, every=args.probe_every)
        torch.cuda.synchronize()
        out = {"probe": "decision-level cache validity (non-intervening shadow full forwards)",
               "workload": f"{w.name}: {w.note}", "policy": args.policy, "K": Kr, "steps": T,
               "probe_every_cached_forward": args.probe_every, "wall_s": round(time.perf_counter() - t0, 3),
               "refresh_fraction": round(float(tr["refreshed"].mean()), 4),
               "data": "synthetic: random-init weights and prompts; values are not comparable to the paper's",
               **probe.summarize(recs)}
        print(json.dumps(out))
        return

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
    # a sample of the launches (every 7th of each class: 7 is coprime with the
    # layer count and the refresh period, so every layer and both pass kinds
    # are sampled) -- each event pair idles the GPU for a few microseconds
    ctx.timing_begin(sorted({archer.K_NAMES.index(dom), archer.K_ATTN}), every=args.timing_every)
    t0 = time.perf_counter()
    for _ in range(args.steps):
        _, tr = decode(pol, Kr)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    tims = ctx.timing_end()
    tim = tims[dom]
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
    peak_f = PEAK_BF16_TFLOPS if m.dtype == "bf16" else PEAK_FP32_TFLOPS
    ridge = peak_f * 1e12 / (PEAK_HBM_GBS * 1e9)
    sec = tim["ms"] / 1e3
    nl = max(tim["launches"], 1)
    exec_flops = tim["flops"] * (2 if (m.dtype == "bf16" and dom in TWO_TERM) else 1)
    # the binding unit follows the executed work: two-term GEMMs issue 2x the
    # algorithmic MFMA work, which moves them past the ridge
    if exec_flops > 0 and exec_flops / max(tim["bytes"], 1.0) >= ridge:
        roof = {"bound": "mfma", "achieved": round(tim["flops"] / sec / 1e12, 2), "peak": peak_f,
                "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": round(tim["bytes"] / sec / 1e9, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
    roof["traffic"] = committed_traffic(dom)
    roof.update({"kernel": KERNEL_OF_CLASS.get(dom, dom), "class": dom, "launches": tim["launches"],
                 "avg_us": round(tim["ms"] * 1e3 / nl, 2),
                 "algorithmic_bytes_per_launch": round(tim["bytes"] / nl),
                 "algorithmic_flops_per_launch": round(tim["flops"] / nl),
                 "algorithmic_hbm_GBps": round(tim["bytes"] / sec / 1e9, 1),
                 "algorithmic_tflops": round(tim["flops"] / sec / 1e12, 2),
                 "executed_mfma_frac": round(exec_flops / sec / 1e12 / peak_f, 4),
                 "timing": f"HIP events around every {args.timing_every}th launch of the class in the timed "
                           f"region, on the library's stream"})

    # the cache-reading attention of the cached passes, against the HBM roofline
    at = tims["attn"]
    att_roof = None
    if at["launches"] and m.dtype == "bf16":
        asec = at["ms"] / 1e3
        att_roof = {"bound": "hbm", "achieved": round(at["bytes"] / asec / 1e9, 1), "peak": PEAK_HBM_GBS,
                    "unit": "GB/s", "frac": round(at["bytes"] / asec / 1e9 / PEAK_HBM_GBS, 4),
                    "kernel": KERNEL_OF_CLASS["attn"], "class": "attn", "launches": at["launches"],
                    "avg_us": round(at["ms"] * 1e3 / at["launches"], 2),
                    "algorithmic_bytes_per_launch": round(at["bytes"] / at["launches"]),
                    "algorithmic_flops_per_launch": round(at["flops"] / at["launches"]),
                    "algorithmic_tflops": round(at["flops"] / asec / 1e12, 2),
                    "mfma_frac": round(at["flops"] / asec / 1e12 / PEAK_BF16_TFLOPS, 4),
                    "timing": f"HIP events around every {args.timing_every}th launch (attention + split-KV "
                              f"merge) in the timed region, on the library's stream"}

    out = {
        "metric": "denoising steps/s + response tok/s at 1 GPU; speedup vs full refresh; % roofline",
        "value": round(sps, 3), "unit": "steps/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(wall / args.steps * 1e3, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": m.dtype,
        "data": "synthetic: seeded random-init weights N(0, 0.02) drawn on the GPU, uniform-random prompt tokens",
        "config": {"workload": f"{w.name}: {w.note}", "batch": B, "prompt_len": lens[0] if len(set(lens)) == 1
                   else [min(lens), max(lens)], "resp_len": G, "denoising_steps_per_decode": T,
                   "unmask_per_step": k, "policy": args.policy, "K": Kr,
                   "weight_layout": "kblock" if m.dtype == "bf16" else "rowmajor"},
        "response_tok_per_s": round(tok, 2),
        "recomputed_positions_per_s": round(tok * T, 1),
        "refresh_fraction": round(refreshed / (T * B), 4),
        "full_refresh_steps_per_s": None if full_sps is None else round(full_sps, 3),
        "speedup_vs_full_refresh": None if full_sps is None else round(sps / full_sps, 3),
        "roofline": roof,
        "attention_roofline": att_roof,
        "warmup_ms_by_class": {n: round(v["ms"], 2) for n, v in warm.items() if v["launches"]},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, lens, T, Kr, args.policy)
    if args.copy_calibration:
        # an elementwise kernel of known HBM traffic: reads 1 GiB, writes 1 GiB
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        torch.mul(src, 2.0, out=dst)
        torch.cuda.synchronize()
        log("bench: calibration kernel (1 GiB read + 1 GiB write) done")
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
