#!/usr/bin/env python3
"""Throughput of the routed prefill KV-eviction pass on one MI355X.

Workload: a LLaMA-3.1-8B-shaped prompt (32 layers, 32 query / 8 KV heads, head_dim 128, bf16)
of L = 8192 tokens, batch 1, evicted under the 32-layer mixed route (StreamingLLM on layers
0-1, SnapKV 2-15, H2O 16-27, SnapKV 28-31) with PyramidKV-style budgets: a linear ramp from
1024 (layer 0) to 128 (layer 31) rescaled to the aggregate capacity 32 x 512 (Eq. 3 of the
paper, b_min 48).  Window 32, max-pool 7.  Synthetic seeded N(0,1) Q/K/V with planted sink,
heavy-hitter and recency structure.

One step = one full eviction pass over all 32 layers (window scoring, softmax, window sum,
pooling, group mean, per-head top-k, K/V gather), inputs resident in HBM.  Beside the headline
line's roofline (the scoring kernel) the record carries the other measured configurations: the
single-layer latency (L = 1024), the batch-8 budget sweep, the 32K long-context routes, the
H2O / TOVA composition, decode steps, the entropy profile, full-span H2O, a measured copy ceiling
and the CPU oracle.  Prints one JSON line.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
L_CTX, N_LAYERS, HQ, HKV, D, W, POOL, AVG_BUDGET, B_MIN = 8192, 32, 32, 8, 128, 32, 7, 512, 48
WORKLOAD_ID = 2
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "score_pipe_kernel_route8k_traffic.json")
SCORE_KERNEL = "score_pipe_kernel<1, false>"
COPY_CAL_BYTES = 1 << 30     # plain device copy used to scale the PMC byte counters


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def algorithmic_bytes(rules, budgets, B=1):
    """Bytes the pass must move: every scored layer's K and window Q once, every retained K/V
    row read and written once, and the int32 index of every retained row written once."""
    from synth.workloads import SNAPKV, H2O
    score = sum(B * (HKV * L_CTX * D * 2 + HQ * W * D * 2) for r in rules if r in (SNAPKV, H2O))
    keep = sum(min(b, L_CTX) for b in budgets)
    gather = B * HKV * keep * D * 2 * 4
    index = B * HKV * keep * 4
    return score, score + gather + index


def cpu_baseline(xs, rules, budgets, max_seconds=20.0):
    """Time the CPU oracle (float64 NumPy, all host cores) on whole passes over the same 32-layer
    input, repeated until about max_seconds of work; report layer-tokens/s."""
    import threadpoolctl
    from oracle import prefill as OP
    # one untimed warm-up layer (BLAS thread start-up, first-touch page faults)
    l0 = next(l for l in range(N_LAYERS) if rules[l] in (OP.SNAPKV, OP.H2O))
    OP.evict_layer(rules[l0], budgets[l0], xs[l0]["q"], xs[l0]["k"], xs[l0]["v"], window=W, pool_kernel=POOL)
    passes, t_total = 0, 0.0
    while passes == 0 or t_total < max_seconds:
        t0 = time.perf_counter()
        for l in range(N_LAYERS):
            OP.evict_layer(rules[l], budgets[l], xs[l]["q"], xs[l]["k"], xs[l]["v"], window=W, pool_kernel=POOL)
        t_total += time.perf_counter() - t0
        passes += 1
    info = threadpoolctl.threadpool_info()
    blas_threads = max([i.get("num_threads", 1) for i in info] or [1])
    return {
        "value": passes * N_LAYERS * L_CTX / t_total,
        "unit": "layer-tokens/s",
        "cores": blas_threads,
        "host_cores_available": len(os.sched_getaffinity(0)),
        "kind": "oracle",
        "sample": f"{passes} whole passes (all 32 layers) over the same 8K route input, {t_total:.1f} s",
    }


def decode_measure(dev, steps=10, warmup=2, B=64, C=1024, n_layers=32):
    """Decode-step throughput at the 64-sequence shape: 32 layers, 32 query / 8 KV heads,
    capacity 1024 per layer, cache resident in HBM (random bf16 contents: the kernel's work does
    not depend on the values).  Two plans: H2O on every layer (recent half protected) and the
    H2O 0-15 / TOVA 16-31 composition.  Algorithmic bytes per step: every cached key row read
    once (C x 256 B per sequence, layer and KV head), the slot positions read, H2O's accumulated
    scores read and written, the new query / key read and the new key / value row written."""
    import torch
    import paper_2606_15157_amd as rkv
    g = torch.Generator(device=dev).manual_seed(20260615)
    kc = [torch.randn((B, HKV, C, D), generator=g, device=dev, dtype=torch.bfloat16) for _ in range(n_layers)]
    vc = [torch.randn((B, HKV, C, D), generator=g, device=dev, dtype=torch.bfloat16) for _ in range(n_layers)]
    pos0 = (torch.arange(C, device=dev, dtype=torch.int32) * 8).expand(B, HKV, C).contiguous()
    acc = [torch.rand((B, HKV, C), generator=g, device=dev) for _ in range(n_layers)]
    n_in = warmup + steps
    qs = [[torch.randn((B, HQ, D), generator=g, device=dev, dtype=torch.bfloat16) for _ in range(n_layers)]
          for _ in range(n_in)]
    ks = [[torch.randn((B, HKV, D), generator=g, device=dev, dtype=torch.bfloat16) for _ in range(n_layers)]
          for _ in range(n_in)]
    out = {}
    for name, rules in (("h2o", [rkv.H2O] * n_layers),
                        ("h2o_tova", [rkv.H2O] * (n_layers // 2) + [rkv.TOVA] * (n_layers - n_layers // 2))):
        plan = rkv.Plan([rkv.H2O] * n_layers, [C] * n_layers, rules, [C] * n_layers, window=W)
        state = {"k_cache": kc, "v_cache": vc, "pos": [pos0.clone() for _ in range(n_layers)],
                 "acc": [a if r == rkv.H2O else None for a, r in zip(acc, rules)]}
        stream = torch.cuda.current_stream(dev)
        p0 = 8 * C
        for i in range(warmup):
            rkv.decode_step(plan, state, qs[i], ks[i], ks[i], p0 + i, stream=stream)
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for i in range(warmup, n_in):
            rkv.decode_step(plan, state, qs[i], ks[i], ks[i], p0 + i, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / steps
        n_h2o = sum(1 for r in rules if r == rkv.H2O)
        units = B * HKV * n_layers
        alg = units * C * (D * 2 + 4) + B * HKV * n_h2o * C * 8 + B * n_layers * (HQ + HKV) * D * 2 + units * 2 * D * 2
        out[name] = {"us_per_step": us, "algorithmic_bytes_per_step": alg, "achieved_GBps": alg / (us * 1e-6) / 1e9,
                     "hbm_frac": alg / (us * 1e-6) / 1e9 / HBM_PEAK_GBPS,
                     "sequence_tokens_per_s": B / (us * 1e-6)}
        log(f"decode {name}: {us:.1f} us/step ({out[name]['achieved_GBps']:.0f} GB/s)")
    del kc, vc, acc, qs, ks
    torch.cuda.empty_cache()
    return {"workload": f"{B} sequences x {n_layers} layers, 32 q / 8 kv heads, d=128, capacity {C} per layer, "
                        f"{steps} timed steps", **out}


def entropy_measure(dev, reps=3, n_layers=32, L=4096):
    """Entropy profile of a calibration-shaped input: 32 layers, 32 query / 8 KV heads, every
    query of a 4096-token sequence (random bf16 contents: the work does not depend on them).
    Algorithmic work: the causal logits, sum over query positions t of (t + 1) keys x 2 d flop
    per query head, on bf16 MFMA; one exponential per logit."""
    import torch
    import paper_2606_15157_amd as rkv
    g = torch.Generator(device=dev).manual_seed(20260616)
    q = [torch.randn((1, HQ, L, D), generator=g, device=dev, dtype=torch.bfloat16) for _ in range(n_layers)]
    k = [torch.randn((1, HKV, L, D), generator=g, device=dev, dtype=torch.bfloat16) for _ in range(n_layers)]
    stream = torch.cuda.current_stream(dev)
    rkv.entropy_profile(q, k, stream=stream)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        out = rkv.entropy_profile(q, k, stream=stream)
    e1.record(stream)
    torch.cuda.synchronize()
    if int(out["status"].item()) != 0:
        raise RuntimeError("entropy profile reported a non-finite row")
    ms = e0.elapsed_time(e1) / reps
    flop = n_layers * HQ * (L * (L + 1) // 2) * D * 2
    tflops = flop / (ms * 1e-3) / 1e12
    log(f"entropy profile: {ms:.3f} ms ({tflops:.0f} TFLOP/s causal)")
    del q, k
    torch.cuda.empty_cache()
    return {"workload": f"{n_layers} layers, 32 q / 8 kv heads, d=128, every query of a {L}-token sequence",
            "ms": ms, "algorithmic_flop": flop, "achieved_TFLOPs": tflops, "peak_TFLOPs": 2500.0,
            "mfma_frac": tflops / 2500.0, "exps_per_s": n_layers * HQ * (L * (L + 1) // 2) / (ms * 1e-3)}


def fullspan_measure(dev, reps=3):
    """The 8K route with its H2O layers (16-27) accumulating over every prompt query instead of
    the window (their queries: all 8192 positions).  Same budgets; random bf16 inputs.  The
    full-span layers dominate: their causal logits, sum_t (t + 1) x 2 d flop per query head
    (counted once)."""
    import torch
    import paper_2606_15157_amd as rkv
    from synth.workloads import mixed_route, pyramid_weights
    rules = [rkv.H2O_FULL if r == rkv.H2O else r for r in mixed_route(N_LAYERS)]
    budgets = rkv.allocate_budgets(pyramid_weights(N_LAYERS), N_LAYERS * AVG_BUDGET, B_MIN)
    g = torch.Generator(device=dev).manual_seed(20260617)
    q = [torch.randn((1, HQ, L_CTX if r == rkv.H2O_FULL else W, D), generator=g, device=dev, dtype=torch.bfloat16)
         for r in rules]
    k = [torch.randn((1, HKV, L_CTX, D), generator=g, device=dev, dtype=torch.bfloat16) for _ in rules]
    v = [torch.randn((1, HKV, L_CTX, D), generator=g, device=dev, dtype=torch.bfloat16) for _ in rules]
    plan = rkv.Plan(rules, budgets, window=W, pool_kernel=POOL)
    out = rkv.alloc_outputs(plan, 1, HKV, L_CTX, D, dev)
    ws = rkv.alloc_workspace(plan, 1, L_CTX, HQ, HKV, dev)
    call = rkv.PreparedPrefill(plan, q, k, v, out, ws)
    stream = torch.cuda.current_stream(dev)
    call(stream)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        call(stream)
    e1.record(stream)
    torch.cuda.synchronize()
    if rkv.prefill_check(ws) != 0:
        raise RuntimeError("full-span pass reported a failure")
    ms = e0.elapsed_time(e1) / reps
    n_full = sum(1 for r in rules if r == rkv.H2O_FULL)
    # the method's work: every causal logit once (the kernels compute them twice, in the row-normaliser
    # and the column-sum pass; that second pass is an implementation choice and is not counted)
    flop = n_full * HQ * (L_CTX * (L_CTX + 1) // 2) * D * 2
    log(f"full-span route: {ms:.3f} ms per pass ({flop / (ms * 1e-3) / 1e12:.0f} TFLOP/s on the full-span logits)")
    del q, k, v, out, ws, call
    torch.cuda.empty_cache()
    return {"workload": "32-layer mixed route at L=8192 with H2O layers 16-27 accumulating over all 8192 queries",
            "ms_per_pass": ms, "full_span_flop": flop, "achieved_TFLOPs": flop / (ms * 1e-3) / 1e12,
            "peak_TFLOPs": 2500.0, "mfma_frac": flop / (ms * 1e-3) / 1e12 / 2500.0,
            "layer_tokens_per_s": N_LAYERS * L_CTX / (ms * 1e-3)}


def percentiles(samples_ms):
    """median / p10 / p90 / mean of per-step durations in microseconds."""
    import numpy as np
    a = np.asarray(samples_ms, dtype=np.float64) * 1e3
    return {"median_us": float(np.median(a)), "p10_us": float(np.percentile(a, 10)),
            "p90_us": float(np.percentile(a, 90)), "mean_us": float(a.mean()), "n": int(a.size)}


def time_steps(fn, stream, steps, warmup):
    """Run fn(stream) warmup times, then `steps` times with a HIP event pair around each call on
    `stream`; returns the per-step durations (ms)."""
    import torch
    for _ in range(warmup):
        fn(stream)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for a, b in ev:
        a.record(stream)
        fn(stream)
        b.record(stream)
    torch.cuda.synchronize()
    return [a.elapsed_time(b) for a, b in ev]


def route_bytes(rules, budgets, B, L, Hq=HQ, Hkv=HKV, d=D, w=W):
    """Algorithmic bytes of one pass: every window-scored layer's K and window queries read once, every
    retained K / V row read and written once, every retained index written once."""
    from synth.workloads import SNAPKV, H2O
    score = sum(B * (Hkv * L * d * 2 + Hq * w * d * 2) for r in rules if r in (SNAPKV, H2O))
    keep = sum(min(b, L) for b in budgets)
    return score, score + B * Hkv * keep * (d * 2 * 4 + 4)


def route_flop(rules, B, L, Hq=HQ, d=D, w=W):
    """Window logits of the window-scored layers: B Hq w L 2 d per layer (masked keys included)."""
    from synth.workloads import SNAPKV, H2O
    return sum(B * Hq * w * L * d * 2 for r in rules if r in (SNAPKV, H2O))


def run_route(dev, rules, budgets, B, L, w, workload, steps, warmup, n_hh):
    """Time the eviction pass of one route over seeded device inputs (same recipe as the parity
    tests' large shapes); returns per-step stats, the score-stage time and the byte accounting."""
    import torch
    import paper_2606_15157_amd as rkv
    from synth import prefill_layer_torch
    xs = [prefill_layer_torch(workload, l, batch=B, seq_len=L, window=w, n_hh=n_hh) for l in range(len(rules))]
    q, k, v = [x["q"] for x in xs], [x["k"] for x in xs], [x["v"] for x in xs]
    del xs
    plan = rkv.Plan(rules, budgets, window=w, pool_kernel=POOL)
    out = rkv.alloc_outputs(plan, B, HKV, L, D, dev)
    ws = rkv.alloc_workspace(plan, B, L, HQ, HKV, dev)
    call = rkv.PreparedPrefill(plan, q, k, v, out, ws)
    stream = torch.cuda.current_stream(dev)
    per = time_steps(call, stream, steps, warmup)
    if rkv.prefill_check(ws) != 0:
        raise RuntimeError("eviction pass reported a failure")
    stage = {}
    for name, sid in (("score", rkv.STAGE_SCORE), ("select", rkv.STAGE_SELECT), ("gather", rkv.STAGE_GATHER),
                      ("zero", rkv.STAGE_ZERO)):
        rkv.profile_enable(sid)
        for _ in range(max(3, steps // 2)):
            call(stream)
        torch.cuda.synchronize()
        n, tot = rkv.profile_read()
        rkv.profile_enable(-1)
        stage[name] = tot / max(n, 1)
    sb, pb = route_bytes(rules, budgets, B, L, w=w)
    flop = route_flop(rules, B, L, w=w)
    st = percentiles(per)
    ms = st["median_us"] * 1e-3
    # scoring in the unprofiled passes: the pass less the other stages (as for the headline line)
    score_ms = ms - (stage["select"] + stage["gather"] + stage["zero"])
    if not 0.0 < score_ms <= stage["score"]:
        score_ms = stage["score"]
    res = {"steps": percentiles(per), "score_us": score_ms * 1e3, "score_profiled_us": stage["score"] * 1e3,
           "algorithmic_bytes": pb,
           "score_algorithmic_bytes": sb, "hbm_frac": pb / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS,
           "score_hbm_frac": sb / (score_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS,
           "score_mfma_frac": flop / (score_ms * 1e-3) / 1e12 / 2500.0,
           "layer_tokens_per_s": B * len(rules) * L / (ms * 1e-3)}
    del q, k, v, out, ws, call
    torch.cuda.empty_cache()
    return res


def c1_measure(dev, steps=200, warmup=20):
    """Latency of one eviction call on the single-layer workload: L = 1024, SnapKV, budget 128,
    32 / 8 heads (and the same layer under H2O, StreamingLLM and Full); the pass is far below the
    HBM time scale (3.4 MB), so only its time is reported."""
    import torch
    import paper_2606_15157_amd as rkv
    from synth import prefill_layer_torch
    x = prefill_layer_torch(1, 0, batch=1, seq_len=1024, window=W, n_hh=16)
    out = {}
    for name, rule in (("snapkv", rkv.SNAPKV), ("h2o", rkv.H2O), ("streaming", rkv.STREAMING), ("full", rkv.FULL)):
        plan = rkv.Plan([rule], [128], window=W, pool_kernel=POOL)
        o = rkv.alloc_outputs(plan, 1, HKV, 1024, D, dev)
        ws = rkv.alloc_workspace(plan, 1, 1024, HQ, HKV, dev)
        call = rkv.PreparedPrefill(plan, [x["q"]], [x["k"]], [x["v"]], o, ws)
        per = time_steps(call, torch.cuda.current_stream(dev), steps, warmup)
        out[name] = percentiles(per)
        log(f"c1 {name}: median {out[name]['median_us']:.1f} us")
    return {"workload": "one layer, L=1024, batch 1, 32 q / 8 kv heads, d=128, w=32, pool 7, budget 128", **out}


def c3_measure(dev, steps=10, warmup=2):
    """Budget sweep on the 32-layer mixed route at L = 8192, batch 8 distinct sequences: average
    budgets 128 / 256 / 512 / 1024 / 2048 per layer, each the completed 512 vector rescaled to the
    new total (Section 3.3's sweep rule, b_min 48)."""
    import paper_2606_15157_amd as rkv
    from synth.workloads import mixed_route, pyramid_weights
    rules = mixed_route(N_LAYERS)
    b512 = rkv.allocate_budgets(pyramid_weights(N_LAYERS), N_LAYERS * 512, B_MIN)
    res = {}
    for avg in (128, 256, 512, 1024, 2048):
        budgets = rkv.allocate_budgets(b512, N_LAYERS * avg, B_MIN)
        r = run_route(dev, rules, budgets, 8, L_CTX, W, 3, steps, warmup, 16)
        res[str(avg)] = r
        log(f"c3 avg {avg}: {r['steps']['median_us']:.0f} us/pass, {r['hbm_frac']:.3f} of HBM peak")
    return {"workload": "32-layer mixed route, L=8192, batch 8, 32 q / 8 kv heads, d=128, w=32, pool 7", **res}


def c4_measure(dev, steps=5, warmup=2):
    """Long context: L = 32768, batch 4, w = 64, average budget 1024 (the completed 512 vector
    rescaled), all-SnapKV, all-H2O and the mixed route; 64 planted heavy hitters per head."""
    import paper_2606_15157_amd as rkv
    from synth.workloads import pyramid_weights, route_by_name
    b512 = rkv.allocate_budgets(pyramid_weights(N_LAYERS), N_LAYERS * 512, B_MIN)
    budgets = rkv.allocate_budgets(b512, N_LAYERS * 1024, B_MIN)
    res = {}
    for route in ("snapkv", "h2o", "mixed"):
        r = run_route(dev, route_by_name(route, N_LAYERS), budgets, 4, 32768, 64, 4, steps, warmup, 64)
        res[route] = r
        log(f"c4 {route}: {r['steps']['median_us']:.0f} us/pass, {r['hbm_frac']:.3f} of HBM peak")
    return {"workload": "32 layers, L=32768, batch 4, 32 q / 8 kv heads, d=128, w=64, pool 7, average budget 1024",
            **res}


def composition_measure(dev, steps=10, warmup=3):
    """Appendix E's composition as a tied both-phase plan (H2O on layers 0-15, TOVA on 16-31, 512
    positions per layer in both phases), batch 1 at the appendix's prompt lengths: the prefill
    eviction pass (H2O window scoring plus TOVA's last-query scoring, selection, gather) and the
    prefill-to-decode hand-off.  Eviction work only; the paper's table measures whole-model runs."""
    import torch
    import paper_2606_15157_amd as rkv
    from synth import prefill_layer_torch
    rules = [rkv.H2O] * 16 + [rkv.TOVA] * 16
    res = {}
    for L in (4096, 8192, 16384, 32768):
        plan = rkv.Plan.from_scoped_route(rules, [rkv.SCOPE_BOTH] * N_LAYERS, [512] * N_LAYERS, window=W)
        xs = [prefill_layer_torch(6, l, batch=1, seq_len=L, window=W, n_hh=16) for l in range(N_LAYERS)]
        q, k, v = [x["q"] for x in xs], [x["k"] for x in xs], [x["v"] for x in xs]
        del xs
        out = rkv.alloc_outputs(plan, 1, HKV, L, D, dev, acc_out=True)
        ws = rkv.alloc_workspace(plan, 1, L, HQ, HKV, dev)
        call = rkv.PreparedPrefill(plan, q, k, v, out, ws)
        stream = torch.cuda.current_stream(dev)
        per = time_steps(call, stream, steps, warmup)
        if rkv.prefill_check(ws) != 0:
            raise RuntimeError("composition pass reported a failure")
        out["io"] = call
        state = rkv.decode_init_from_prefill(plan, out)
        hand = time_steps(lambda st: rkv.decode_init_from_prefill(plan, out, state, stream=st), stream, steps, warmup)
        st_ = percentiles(per)
        res[str(L)] = {"prefill_pass": st_, "handoff": percentiles(hand),
                       "prompt_tokens_per_s": L / (st_["median_us"] * 1e-6)}
        log(f"composition L={L}: prefill eviction {st_['median_us']:.0f} us, hand-off "
            f"{res[str(L)]['handoff']['median_us']:.1f} us")
        del q, k, v, out, ws, call, state
        torch.cuda.empty_cache()
    return {"workload": "H2O 0-15 / TOVA 16-31 tied in both phases, 512 positions per layer, batch 1, "
                        "32 q / 8 kv heads, d=128", **res}


def copy_ceiling(dev, nbytes=1 << 30, reps=5):
    """A plain 1 GiB device-to-device copy (read + write bytes over its time): the HBM rate a
    streaming kernel reaches on this GPU, reported beside the 8 TB/s vendor peak."""
    import torch
    src = torch.empty(nbytes // 2, dtype=torch.bfloat16, device=dev).fill_(1.0)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del src, dst
    torch.cuda.empty_cache()
    return 2 * nbytes / (ms * 1e-3) / 1e9


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def kernel_source_hash():
    from paper_2606_15157_amd.pmc_summary import kernel_source_hash as source_hash
    return source_hash()


def traffic_record():
    """HBM bytes (read + write) per launch of the scoring kernel from the committed rocprofv3
    PMC summary, or None when it is missing or was taken on a different kernel source."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    rec = json.load(open(TRAFFIC_FILE))
    if rec.get("kernel_source_sha256") != kernel_source_hash():
        return None
    return rec.get("hbm_bytes_per_launch")


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--settle", type=int, default=100,
                    help="untimed passes of the headline route before the warm-up steps (power-state settling)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=20.0)
    ap.add_argument("--no-decode", action="store_true", help="skip the decode-step measurement")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the single-layer latency, batch-8 budget sweep and 32K long-context legs")
    ap.add_argument("--no-entropy", action="store_true", help="skip the entropy-profile measurement")
    ap.add_argument("--no-fullspan", action="store_true", help="skip the full-span H2O route measurement")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run one plain 1 GiB device copy (outside the timed region) so a "
                         "rocprofv3 --pmc run of this command can scale FETCH_SIZE / WRITE_SIZE")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported by this build "
              f"(the eviction path shards by KV head / sequence / layer with no exchange, but no "
              f"multi-GPU run is made here)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    import paper_2606_15157_amd as rkv
    from synth import prefill_layer
    from synth.workloads import mixed_route, pyramid_weights

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    rules = mixed_route(N_LAYERS)
    budgets = rkv.allocate_budgets(pyramid_weights(N_LAYERS), N_LAYERS * AVG_BUDGET, B_MIN)
    log(f"budgets {budgets}")
    t0 = time.perf_counter()
    xs = [prefill_layer(WORKLOAD_ID, 0, l, seq_len=L_CTX, n_q_heads=HQ, n_kv_heads=HKV, head_dim=D, window=W,
                        n_hh=16) for l in range(N_LAYERS)]
    log(f"generated inputs in {time.perf_counter() - t0:.1f} s")

    def to_dev(bits):
        return torch.from_numpy(np.ascontiguousarray(bits[None]).view(np.int16)).to(dev).view(torch.bfloat16)

    q = [to_dev(x["q"]) for x in xs]
    k = [to_dev(x["k"]) for x in xs]
    v = [to_dev(x["v"]) for x in xs]
    plan = rkv.Plan(rules, budgets, window=W, pool_kernel=POOL)
    out = rkv.alloc_outputs(plan, 1, HKV, L_CTX, D, dev)
    ws = rkv.alloc_workspace(plan, 1, L_CTX, HQ, HKV, dev)
    call = rkv.PreparedPrefill(plan, q, k, v, out, ws)
    stream = torch.cuda.current_stream(dev)

    # settle, then the W warm-up steps: after the first few passes under load the GPU's power
    # management slows this kernel by up to ~15 % for a few tens of passes before it settles
    # (kernel-trace durations 181 -> 207 -> 177 us), so that transient is run off untimed first
    for _ in range(args.settle):
        call(stream)
    for _ in range(args.warmup):
        call(stream)
    torch.cuda.synchronize()
    if rkv.prefill_check(ws) != 0:
        raise RuntimeError("scoring work items timed out during warm-up")

    # the timed region: K back-to-back steps between one pair of events
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    e0.record(stream)
    for _ in range(args.steps):
        call(stream)
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms_step = e0.elapsed_time(e1) / args.steps
    log(f"timed {args.steps} steps: {ms_step * 1e3:.1f} us/step (wall {wall / args.steps * 1e6:.1f} us/step)")
    # the spread of single steps, from another K steps with an event pair around each (the
    # events between the steps make these slightly slower than the back-to-back steps above)
    step_ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for a, b in step_ev:
        a.record(stream)
        call(stream)
        b.record(stream)
    torch.cuda.synchronize()
    step_stats = percentiles([a.elapsed_time(b) for a, b in step_ev])
    # cold steps: before each, a 512 MiB buffer is read (outside the events), so that the 256 MB
    # last-level cache holds none of the pass's inputs when it starts
    cold_buf = torch.ones(256 << 20, dtype=torch.bfloat16, device=dev)
    cold_ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for a, b in cold_ev:
        cold_buf.sum()
        a.record(stream)
        call(stream)
        b.record(stream)
    torch.cuda.synchronize()
    cold_stats = percentiles([a.elapsed_time(b) for a, b in cold_ev])
    del cold_buf
    log(f"cold steps (512 MiB read before each): median {cold_stats['median_us']:.1f} us")
    if rkv.prefill_check(ws) != 0:
        raise RuntimeError("scoring work items timed out in the timed region")

    if args.copy_calibration:
        # the source is filled first, then a 512 MiB buffer is written so that the copy reads
        # from HBM rather than from the 256 MB last-level cache
        src = torch.empty(COPY_CAL_BYTES // 2, dtype=torch.bfloat16, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        flush = torch.empty(256 << 20, dtype=torch.bfloat16, device=dev).fill_(0.0)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"copy calibration: {COPY_CAL_BYTES} bytes read and written once")
        del src, dst, flush

    # per-kernel durations: HIP events around every launch of each stage, over the same steps
    stage_ms = {}
    for name, st in (("score", rkv.STAGE_SCORE), ("select", rkv.STAGE_SELECT), ("gather", rkv.STAGE_GATHER),
                     ("zero", rkv.STAGE_ZERO)):
        rkv.profile_enable(st)
        for _ in range(args.steps):
            call(stream)
        torch.cuda.synchronize()
        n, tot = rkv.profile_read()
        rkv.profile_enable(-1)
        stage_ms[name] = tot / max(n, 1)
    log("stage us/launch: " + ", ".join(f"{kk} {vv * 1e3:.1f}" for kk, vv in stage_ms.items()))

    score_bytes, pass_bytes = algorithmic_bytes(rules, budgets)
    # the scoring kernel's duration in the unprofiled timed passes: the pass time less the other
    # three stages' own dispatch durations (those kernels time the same profiled or not; any gap
    # between launches is counted as scoring, so this bounds the duration from above).  Profiled
    # directly, the persistent scoring kernel runs 10-20 % slower (kept as score_profiled_us).
    score_ms = ms_step - (stage_ms["select"] + stage_ms["gather"] + stage_ms["zero"])
    if not 0.0 < score_ms <= stage_ms["score"]:
        score_ms = stage_ms["score"]
    log(f"scoring kernel in the timed passes: {score_ms * 1e3:.1f} us (profiled: {stage_ms['score'] * 1e3:.1f} us)")
    score_gbps = score_bytes / (score_ms * 1e-3) / 1e9
    score_flop = route_flop(rules, 1, L_CTX)
    pass_gbps = pass_bytes / (ms_step * 1e-3) / 1e9
    traffic = traffic_record()
    value = N_LAYERS * L_CTX / (ms_step * 1e-3)

    rec = {
        "metric": "KV tokens scored+compacted/s (32-layer 8K route); % of HBM peak",
        "value": value,
        "unit": "layer-tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "settle_passes": args.settle,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": "32-layer mixed route (StreamingLLM 0-1, SnapKV 2-15, H2O 16-27, SnapKV 28-31), "
                        "L=8192, batch 1, 32 q / 8 kv heads, d=128, window 32, pool 7, "
                        "PyramidKV ramp budgets summing to 32x512",
            "batch": 1, "seq_len": L_CTX, "n_layers": N_LAYERS, "n_q_heads": HQ, "n_kv_heads": HKV,
            "head_dim": D, "window": W, "pool_kernel": POOL, "aggregate_budget": sum(budgets),
        },
        "pass": {
            "algorithmic_bytes": pass_bytes,
            "achieved_GBps": pass_gbps,
            "hbm_frac": pass_gbps / HBM_PEAK_GBPS,
            "single_steps": {**step_stats, "note": "another K steps, each between its own pair of events"},
            "cold_steps": {**cold_stats, "note": "another K steps, each between its own pair of events, after a "
                                                "512 MiB read that leaves none of the inputs in the last-level cache"},
            "stage_us": {kk: vv * 1e3 for kk, vv in stage_ms.items()},
            "score_us_in_timed_passes": score_ms * 1e3,
        },
        "score_mfma": {
            "kernel": SCORE_KERNEL,
            "flop_per_launch": score_flop,
            "achieved_TFLOPs": score_flop / (score_ms * 1e-3) / 1e12,
            "peak_TFLOPs": 2500.0,
            "frac": score_flop / (score_ms * 1e-3) / 1e12 / 2500.0,
        },
        "roofline": {
            "kernel": SCORE_KERNEL,
            "bound": "hbm",
            "achieved": score_gbps,
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": score_gbps / HBM_PEAK_GBPS,
            "traffic": traffic,
            "algorithmic_bytes_per_launch": score_bytes,
            "timing": "the smaller of two upper bounds on the scoring kernel's duration in the timed "
                      "passes: their per-pass time (one HIP event pair around K back-to-back passes) less "
                      "the prepare, select and gather kernels' own durations (their dispatch timestamps, "
                      "HIP events, K passes each), and its own dispatch timestamps (score_profiled_us; "
                      "the persistent kernel runs 10-20 % slower while profiled); kernel trace in profiles/",
            "score_profiled_us": stage_ms["score"] * 1e3,
        },
    }
    del out, ws, call, q, k, v
    torch.cuda.empty_cache()
    rec["copy_ceiling_GBps"] = copy_ceiling(dev)
    log(f"copy ceiling: {rec['copy_ceiling_GBps']:.0f} GB/s")
    if not args.no_configs:
        rec["c1_latency"] = c1_measure(dev)
        rec["c3_budget_sweep"] = c3_measure(dev)
        rec["c4_long_context"] = c4_measure(dev)
        rec["h2o_tova_composition"] = composition_measure(dev)
    if not args.no_decode:
        rec["decode"] = decode_measure(dev)
    if not args.no_entropy:
        rec["entropy"] = entropy_measure(dev)
    if not args.no_fullspan:
        rec["h2o_full_span"] = fullspan_measure(dev)
    if not args.no_cpu_baseline:
        log("timing the CPU oracle ...")
        rec["cpu_baseline"] = cpu_baseline(xs, rules, budgets, args.cpu_seconds)
        rec["cpu_baseline"]["cpu_model"] = cpu_model()
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
