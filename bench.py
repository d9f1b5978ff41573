#!/usr/bin/env python3
"""Throughput of Archer cached-prompt diffusion-LM decoding on one MI355X.

The workload (default: the batched ragged one -- LLaDA-8B shape, 16
sequences with seeded prompt lengths in [256, 2048], G 256, T 256, refresh
every 8 decisions) is decoded by Algorithm 1 as one decode session of the
library (archer_session_begin / archer_session_advance).  One bench step is
one refresh period of that decode: K decisions, each followed by its forward
-- K - 1 cached forwards (CachedForward over the response rows only) and one
refresh (FullForward, new prompt K/V cache) under the age rule.  Every step
does the same work, and 32 steps are one whole 256-decision decode; when the
schedule ends, the next decode's first forward (a refresh of every sequence)
closes the step.  Inputs are resident in HBM before the timed region.

Reported (one JSON line on stdout):
  value                  denoising steps/s = steps * K / wall
  response_tok_per_s     completed response tokens/s = value * B * G / T
  speedup_vs_full_refresh  wall(refresh at every forward) / wall(Archer), same work per step
  roofline               the kernel class with the most time in the timed region:
                         algorithmic flops (or bytes) / its HIP-event time, the
                         attainable min(peak, AI * HBM) and the calibrated HBM traffic
  gemm_rooflines         every projection class, cached and refresh passes apart
  attention_roofline     the cache-reading attention of the cached passes against HBM
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

# classes whose bf16 launches multiply two-term activations (two MFMAs per fragment),
# except gate/up in models with fp16 gate/up operands
GEMM_CLASSES = ("gemm_qkv", "gemm_o", "gemm_gateup", "gemm_down", "gemm_head",
                "gemm_qkv_full", "gemm_o_full", "gemm_gateup_full", "gemm_down_full")
SINGLE_TERM_OF = {c: c.replace("gemm_", "").replace("_full", "") for c in GEMM_CLASSES}
TRAFFIC_DIR = os.path.join(ROOT, "profiles")


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


def committed_traffic(workload, cls):
    """HBM bytes per launch from the committed rocprofv3 PMC record of this
    workload and kernel class, if it was taken on the current kernel sources;
    else None."""
    path = os.path.join(TRAFFIC_DIR, f"traffic_{cls}_{workload}.json")
    try:
        with open(path) as f:
            rec = json.load(f)
        if rec.get("class") != cls or rec.get("kernel_sources_sha256_16") != src_hash(rec["kernel_sources"]):
            return None
    except (OSError, ValueError, KeyError):
        return None
    return rec.get("hbm_bytes_per_launch")


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, lens, T, K_refresh, policy):
    """Time the oracle (as it is) on a bounded sample of the workload and
    extrapolate to the whole decode.

    Sample: the first S layers of the workload model at full width for the
    shortest and the longest prompt of the batch (one sequence when all are
    equal): one FullForward, one CachedForward, the LM head and one decision
    each.  Per sequence b the per-layer times are interpolated linearly in its
    row count between the two samples and scaled to all layers; the decode is
    R refreshes, T - R cached forwards and T decisions per sequence."""
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
    sample = sorted({int(np.argmin(lens)), int(np.argmax(lens))})
    S = min(9 if len(sample) == 1 else 4, w.model.n_layers)
    mS = dataclasses.replace(w.model, n_layers=S)
    log(f"cpu baseline: generating {S} layers of host weights")
    W = model_weights(mS, seed=w.weight_seed)
    ps = prompts(w, lens)
    G = w.decode.resp_len
    L = w.model.n_layers
    g = np.full(G, mS.mask_id)
    g[: G // 8] = np.arange(G // 8)
    per = {}
    measured = 0.0
    for b in sample:
        p = ps[b]
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
        measured += t_fullS + t_cachedS + t_head + t_dec
        # per-layer times (the head is measured once and counted once per forward)
        per[len(p)] = (max(t_fullS - t_head, 0.0) / S, max(t_cachedS - t_head, 0.0) / S, t_head, t_dec)
        log(f"cpu baseline: P {len(p)}: {S}-layer full {t_fullS:.2f}s cached {t_cachedS:.2f}s "
            f"head {t_head:.2f}s decide {t_dec:.2f}s")
    Ps = sorted(per)

    def at(P, i):
        if len(Ps) == 1:
            return per[Ps[0]][i]
        lo, hi = Ps[0], Ps[-1]
        return per[lo][i] + (P - lo) * (per[hi][i] - per[lo][i]) / (hi - lo)

    R = T if policy == "always" else math.ceil(T / max(K_refresh, 1))
    total = 0.0
    for P in lens:
        t_full = L * at(P, 0) + at(P, 2)
        t_cached = L * at(P, 1) + at(P, 2)
        total += R * t_full + (T - R) * t_cached + T * at(P, 3)
    log(f"cpu baseline: decode {total:.1f}s extrapolated")
    plist = " and ".join(str(len(ps[b])) for b in sample)
    return {"value": T / total, "unit": "steps/s", "cores": int(cores), "kind": "oracle",
            "cpu_model": cpu_model(),
            "sample": (f"the first {S} of {L} layers of the workload model at full width, for the prompt(s) of "
                       f"length {plist} of the batch: one FullForward, one CachedForward over {G} rows, the "
                       f"LM head over {G} rows and one decision over {G}x{w.model.vocab} logits each, float64 "
                       f"NumPy ({measured:.1f} s); per-layer times interpolated linearly in the prompt length "
                       f"for the {len(lens)} sequence(s), scaled to {L} layers and the {T}-decision schedule "
                       f"with {R} refreshes per sequence"),
            "measured_s": round(measured, 2)}


def sweep(kind, reps=10):
    """Per-update and radius sweeps on the LLaDA-8B-shaped random-init model
    (the paper's prompt-length and radius studies, App. E and App. B):
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


def roofline_of(t, peak_f, two_term, timing_every, traffic=None):
    """Roofline object of one timed kernel class: algorithmic flops / bytes of the timed launches
    over their HIP-event time; the binding unit follows the executed work (two-term GEMMs issue
    2x the algorithmic MFMA work); attainable = min(peak, AI * HBM) at the algorithmic AI."""
    sec = t["ms"] / 1e3
    n = max(t["launches"], 1)
    ridge = peak_f * 1e12 / (PEAK_HBM_GBS * 1e9)
    exec_flops = t["flops"] * (2 if two_term else 1)
    tflops = t["flops"] / sec / 1e12
    gbs = t["bytes"] / sec / 1e9
    ai = t["flops"] / max(t["bytes"], 1.0)
    attainable_tflops = min(peak_f, ai * PEAK_HBM_GBS / 1e3)
    if exec_flops > 0 and exec_flops / max(t["bytes"], 1.0) >= ridge:
        r = {"bound": "mfma", "achieved": round(tflops, 2), "peak": peak_f, "unit": "TFLOP/s"}
    else:
        r = {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s"}
    r["frac"] = round(r["achieved"] / r["peak"], 4)
    r["traffic"] = traffic
    r.update({"launches": t["launches"], "avg_us": round(t["ms"] * 1e3 / n, 2),
              "algorithmic_bytes_per_launch": round(t["bytes"] / n),
              "algorithmic_flops_per_launch": round(t["flops"] / n),
              "algorithmic_hbm_GBps": round(gbs, 1), "algorithmic_tflops": round(tflops, 2),
              "arithmetic_intensity": round(ai, 1),
              "attainable_tflops": round(attainable_tflops, 1),
              "attainable_frac": round(tflops / attainable_tflops, 4) if attainable_tflops > 0 else None,
              "two_term_activation": bool(two_term),
              "executed_mfma_frac": round(exec_flops / sec / 1e12 / peak_f, 4),
              "timing": f"HIP events around every {timing_every}th launch of the class in the timed "
                        f"region, on the library's stream"})
    return r


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10, help="timed refresh periods")
    ap.add_argument("--warmup", type=int, default=2, help="untimed refresh periods before the timed ones")
    ap.add_argument("--workload", default="llada_ragged16")
    ap.add_argument("--policy", default="age", choices=["age", "hamming", "always"])
    ap.add_argument("--single-term", default="",
                    help="comma-separated projections (qkv,o,gateup,down,head) with single-bf16 activations")
    ap.add_argument("--two-term-gateup", action="store_true",
                    help="gate/up with two-term bf16 operands instead of the model's fp16 ones")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-full-refresh", action="store_true")
    ap.add_argument("--timing-every", type=int, default=7,
                    help="time every n-th launch of the measured kernel classes (1 = all)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="profiling only: end with a 1 GiB device copy (known HBM traffic) for PMC scaling")
    ap.add_argument("--sweep", choices=["update", "response", "radius"],
                    help="run a sweep instead of the throughput bench (prints its own JSON object)")
    ap.add_argument("--probe", action="store_true",
                    help="run the cache-validity probe (shadow full forwards at cached steps) on the "
                         "workload instead of the throughput bench (prints its own JSON object)")
    ap.add_argument("--probe-every", type=int, default=4, help="probe every n-th cached forward")
    ap.add_argument("--probe-steps", type=int, default=0, help="probe: decisions to run (0 = the workload's T)")
    args = ap.parse_args()
    if args.sweep:
        sweep(args.sweep)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              f"(asked for --gpus {args.gpus}); run it with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import dataclasses

    import numpy as np
    import torch

    from paper_2608_08086_amd import archer
    from synth.device import model_weights_cuda
    from synth.gen import prompt_lengths, prompts
    from synth.workloads import get_workload

    w = get_workload(args.workload)
    if args.single_term:
        w = w.with_model(single_term=tuple(x for x in args.single_term.split(",") if x))
    if args.two_term_gateup:
        w = w.with_model(gateup_fp16=False)
    m, dec = w.model, w.decode
    B, G, T, k = dec.batch, dec.resp_len, dec.steps, dec.unmask_per_step
    Kr = dec.refresh_every
    lens = prompt_lengths(w)
    pol = {"age": archer.AGE, "hamming": archer.HAMMING, "always": archer.ALWAYS}[args.policy]
    log(f"bench: workload {w.name} B={B} P={lens if len(lens) <= 4 else (min(lens), max(lens))} G={G} T={T} "
        f"k={k} policy={args.policy} K={Kr} single_term={list(m.single_term)} gateup_fp16={m.gateup_fp16}")
    t0 = time.perf_counter()
    Wd = model_weights_cuda(m, seed=w.weight_seed)
    if m.dtype == "bf16":
        # projection matrices in the k-block layout (packed once, outside the timed region)
        Wd = archer.pack_weights(Wd, drop_source=True)
    torch.cuda.synchronize()
    log(f"bench: device weights ready in {time.perf_counter() - t0:.1f}s")
    ctx = archer.Context(m, Wd, B, max(lens), sum(lens), G)
    prompt = torch.from_numpy(np.concatenate(prompts(w, lens)).astype(np.int32)).cuda()
    resp0 = torch.full((B, G), m.mask_id, dtype=torch.int32, device="cuda")
    if args.probe:
        from paper_2608_08086_amd import probe

        # the shadow context's prompt cache is the scratch cache of the fresh forwards
        shadow = archer.Context(m, Wd, B, max(lens), sum(lens), G)
        Tp = args.probe_steps or T
        t0 = time.perf_counter()
        _, tr, recs = probe.shadow_probe(ctx, shadow, prompt, lens, resp0, policy=pol, K=Kr, steps=Tp, k=k,
                                         tau=dec.remask_threshold, every=args.probe_every)
        torch.cuda.synchronize()
        out = {"probe": "decision-level cache validity (non-intervening shadow full forwards)",
               "workload": f"{w.name}: {w.note}", "policy": args.policy, "K": Kr, "steps": Tp,
               "probe_every_cached_forward": args.probe_every, "wall_s": round(time.perf_counter() - t0, 3),
               "refresh_fraction": round(float(tr["refreshed"].mean()), 4),
               "data": "synthetic: random-init weights and prompts; values are not comparable to the paper's",
               **probe.summarize(recs)}
        print(json.dumps(out))
        return

    period = max(1, min(Kr, T))

    def runner(policy, K):
        """One bench step = `period` decisions of a decode session (with their forwards)."""
        st = {"t": 0}
        tr = ctx.session_begin(prompt, lens, resp0, policy=policy, K=K, steps=T, k=k,
                               tau=dec.remask_threshold, trace=True)

        def step():
            st["t"] = ctx.session_advance(period)
            if st["t"] >= T:
                # the schedule is complete: the next decode's forward 0 closes this period
                ctx.session_begin(prompt, lens, resp0, policy=policy, K=K, steps=T, k=k,
                                  tau=dec.remask_threshold, trace=False)
                st["t"] = 0
        return step, tr

    step, tr = runner(pol, Kr)
    # warm-up, with every kernel class timed in the first period to find the dominant one
    args.warmup = max(args.warmup, 1)
    for i in range(args.warmup):
        if i == 0:
            ctx.timing_begin(range(archer.K_COUNT))
        step()
        if i == 0:
            warm = ctx.timing_end()
    dom = max(warm, key=lambda n: warm[n]["ms"])
    log("bench: warm-up ms per class " + ", ".join(f"{n}={v['ms']:.1f}" for n, v in warm.items() if v["launches"]))

    torch.cuda.synchronize()
    # a sample of the launches (every 7th of each class: 7 is coprime with the
    # layer count and the refresh period, so every layer and both pass kinds
    # are sampled) -- each event pair idles the GPU for a few microseconds
    measured = sorted({archer.K_NAMES.index(c) for c in GEMM_CLASSES} | {archer.K_ATTN, archer.K_NAMES.index(dom)})
    ctx.timing_begin(measured, every=args.timing_every)
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    tims = ctx.timing_end()
    sps = args.steps * period / wall
    log(f"bench: {args.steps} refresh periods of {period} decisions in {wall:.3f}s -> {sps:.2f} steps/s")

    # refresh fraction of the timed forwards: those of the first decode's trace,
    # plus, if the timed steps reached the end of its schedule, the next
    # decode's forward 0 that closed that period (later decodes repeat it)
    ref = tr["refreshed"].cpu().numpy()
    lo = args.warmup * period + 1
    wrapped = (args.warmup + args.steps) * period >= T
    hi = T if wrapped else (args.warmup + args.steps) * period + 1
    n_ref = float(ref[lo:hi].sum()) + (B if wrapped else 0)
    n_fwd = (hi - lo) * B + (B if wrapped else 0)
    refresh_fraction = n_ref / n_fwd if n_fwd > 0 else None

    full_sps = None
    if not args.no_full_refresh and args.policy != "always":
        fstep, _ = runner(archer.ALWAYS, 0)
        fstep()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        fstep()
        torch.cuda.synchronize()
        full_sps = period / (time.perf_counter() - t0)
        log(f"bench: refresh at every forward: {full_sps:.2f} steps/s")

    tok = sps * B * G / T
    peak_f = PEAK_BF16_TFLOPS if m.dtype == "bf16" else PEAK_FP32_TFLOPS
    single = set(m.single_term)

    def two_term(cls):
        if m.gateup_fp16 and SINGLE_TERM_OF.get(cls) == "gateup":
            return False   # one fp16 MFMA per fragment
        return m.dtype == "bf16" and cls in GEMM_CLASSES and SINGLE_TERM_OF[cls] not in single

    gemm_roofs = {}
    for cls in GEMM_CLASSES:
        if tims[cls]["launches"]:
            gemm_roofs[cls] = roofline_of(tims[cls], peak_f, two_term(cls), args.timing_every,
                                          committed_traffic(w.name, cls))
    # the dominant class: the most time in the timed region (event time x sampling stride)
    dom_t = max((c for c in tims if tims[c]["launches"]), key=lambda c: tims[c]["ms"])
    roof = roofline_of(tims[dom_t], peak_f, two_term(dom_t), args.timing_every, committed_traffic(w.name, dom_t))
    roof = {"class": dom_t, **roof}

    # the cache-reading attention of the cached passes, against the HBM roofline
    at = tims["attn"]
    att_roof = None
    if at["launches"] and m.dtype == "bf16":
        asec = at["ms"] / 1e3
        att_roof = {"bound": "hbm", "achieved": round(at["bytes"] / asec / 1e9, 1), "peak": PEAK_HBM_GBS,
                    "unit": "GB/s", "frac": round(at["bytes"] / asec / 1e9 / PEAK_HBM_GBS, 4),
                    "traffic": committed_traffic(w.name, "attn"),
                    "class": "attn", "launches": at["launches"],
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
        "config": {"workload": f"{w.name}: {w.note}", "batch": B,
                   "prompt_len": lens[0] if len(set(lens)) == 1 else [min(lens), max(lens)],
                   "prompt_total": sum(lens), "resp_len": G, "denoising_steps_per_decode": T,
                   "unmask_per_step": k, "policy": args.policy, "K": Kr,
                   "bench_step": f"one refresh period: {period} decisions with their forwards",
                   "single_term_activations": sorted(single),
                   "gateup_fp16": bool(m.dtype == "bf16" and m.gateup_fp16),
                   "weight_layout": "kblock" if m.dtype == "bf16" else "rowmajor"},
        "response_tok_per_s": round(tok, 3),
        "recomputed_positions_per_s": round(sps * B * G, 1),
        "refresh_fraction": None if refresh_fraction is None else round(refresh_fraction, 4),
        "full_refresh_steps_per_s": None if full_sps is None else round(full_sps, 3),
        "speedup_vs_full_refresh": None if full_sps is None else round(sps / full_sps, 3),
        "roofline": roof,
        "gemm_rooflines": gemm_roofs,
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
