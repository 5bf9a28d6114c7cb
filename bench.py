#!/usr/bin/env python3
"""Decode-step benchmark of libckv on one MI355X.

One step = the whole hot path for every layer of a Llama-3-8B-shaped decode
batch: score every key of the context with the query (MFMA), select the
top-k positions per KV head, and attend over the selected K/V rows read in
place from HBM -- one fused `ckv_critical_kv_attn` call per layer, 32 layers.
Inputs are synthetic (seeded), resident in HBM before timing starts.

Prints ONE JSON line on stdout; progress goes to stderr.

    python bench.py [--gpus 1] [--steps 20] [--warmup 3]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = ("decode-step attention tokens/s at batch×context; "
          "achieved HBM GB/s + host GB/s")
HBM_PEAK_GBPS = 8000.0
COUNTERS = os.path.join(ROOT, "profiles", "critical_llama8b_counters.txt")


SECTIONS = ("main", "extras", "pipelined", "sweep", "host_link", "long128k", "dual64", "million",
            "cpu")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def median(xs):
    xs = sorted(xs)
    n = len(xs)
    return xs[n // 2] if n % 2 else 0.5 * (xs[n // 2 - 1] + xs[n // 2])


KERNEL_SOURCES = ("ckv_score.hpp", "ckv_device.hpp", "ckv_topk.hpp", "ckv_attn.hpp",
                  "ckv_kernels.hip")


def source_digest() -> str:
    """sha256 over the sources of the step's kernels (counters taken on other
    sources are stale)."""
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2607_26475_amd", "csrc", name), "rb") as f:
            h.update(name.encode())
            h.update(f.read())
    return h.hexdigest()


def read_counters(kernel):
    """HBM bytes per launch of the step's dominant kernel from the committed
    rocprofv3 counter summary, or None if absent, taken on other sources or
    for another kernel."""
    if not os.path.exists(COUNTERS):
        return None
    vals = {}
    for line in open(COUNTERS):
        if ":" in line:
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    if vals.get("source_sha256") != source_digest() or vals.get("kernel") != kernel:
        return None
    try:
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_name() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--layout", choices=("separate", "interleaved"), default="separate",
                    help="K and V caches as two arrays, or K|V interleaved per position")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-host-link", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the dual-token, chunked and graph sections "
                         "(the main step alone, e.g. for its kernel profile)")
    ap.add_argument("--no-pipeline", action="store_true",
                    help="skip the pipelined long-context measurement")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a 1 GiB device copy (known bytes) before timing, so "
                         "that counter runs can scale FETCH_SIZE/WRITE_SIZE")
    ap.add_argument("--sections", default=",".join(SECTIONS),
                    help="comma-separated sections to run (default: all of "
                         f"{','.join(SECTIONS)}); a kernel profile of one section "
                         "names it alone, e.g. --sections host_link")
    ap.add_argument("--loop-steps", type=int, default=20,
                    help="timed steps of each host-pinned decode loop (median reported)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              f"(asked for --gpus {args.gpus}, WORLD_SIZE {world}).", file=sys.stderr)
        return 2
    sections = [x for x in args.sections.split(",") if x]
    bad = [x for x in sections if x not in SECTIONS]
    if bad:
        print(f"unknown sections {bad}; choose from {SECTIONS}", file=sys.stderr)
        return 2
    for flag, names in ((args.no_cpu_baseline, ("cpu",)), (args.no_host_link, ("host_link",)),
                        (args.no_extras, ("extras",)),
                        (args.no_pipeline, ("long128k", "dual64", "million"))):
        if flag:
            sections = [x for x in sections if x not in names]

    import numpy as np
    import torch

    import paper_2607_26475_amd as ckv
    import synth

    assert torch.cuda.is_available(), "bench.py needs the GPU"
    dev = torch.device("cuda:0")
    _pipeline_streams(torch)  # first, so that the decode loops' streams get queues of their own
    w = synth.WORKLOADS["llama8b"]
    B, Hq, Hkv, d, n, k, L = (w.batch, w.q_heads, w.kv_heads, w.head_dim, w.max_ctx, w.k,
                              w.layers)
    scale = float(np.float32(1.0 / math.sqrt(d)))
    need_llama = [x for x in sections if x in ("main", "extras", "pipelined", "sweep", "cpu")]
    n_layers = L if any(x in sections for x in ("main", "extras", "pipelined", "sweep")) else (
        1 if need_llama else 0)

    log(f"generating {n_layers} layers of {w.name} inputs on {torch.cuda.get_device_name(0)}")
    t0 = time.time()
    layers = []
    for l in range(n_layers):
        t = synth.make_layer(w, seed=0, layer=l, device=dev)
        if args.layout == "interleaved":
            # the scoring pass reads the K half of each 512-byte row,
            # attention reads a selected row in one piece
            t["kv"] = synth.interleave_kv(t.pop("k"), t.pop("v"))
        del t["marked"]
        layers.append(t)
    torch.cuda.synchronize()
    log(f"  {time.time() - t0:.1f} s; {torch.cuda.memory_allocated() / 2**30:.1f} GiB resident")

    row = 2 * d if args.layout == "interleaved" else d
    s = ckv.shape_for(B, Hq, Hkv, n, key_row_stride=row, kv_row_stride=row)
    stream = torch.cuda.current_stream()
    if args.layout == "interleaved":
        kv_ptrs = [(t["kv"].data_ptr(), t["kv"].data_ptr() + 2 * d) for t in layers]
    else:
        kv_ptrs = [(t["k"].data_ptr(), t["v"].data_ptr()) for t in layers]

    if args.calibrate_copy:
        a = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        del a, b

    result = {
        "metric": METRIC, "value": None, "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": None,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "accumulate": "f32", "data": "synthetic",
        "config": {
            "workload": "Llama-3-8B-shaped decode, 32 layers: B16, 32 q / 8 KV heads, "
                        "head_dim 128, context 32768, k 2048 per KV head, K/V in HBM "
                        + ("(K|V interleaved per position)" if args.layout == "interleaved"
                           else "(separate K and V caches)"),
            "layout": args.layout,
            "batch": B, "context": n, "k": k, "layers": L, "q_heads": Hq,
            "kv_heads": Hkv, "head_dim": d, "placement": "hbm",
        },
        "sections": sections,
    }
    if "main" in sections:
        result.update(measure_main(torch, ckv, layers, kv_ptrs, s, w, scale, args, stream))
    if "extras" in sections:
        ws = ckv.workspace(s, k, ckv.ENTRY_CRITICAL_KV_ATTN)
        dual_token = measure_dual_token(torch, ckv, w, scale, stream)
        log(f"dual-token attention: co-batched {dual_token['co_batched_us']:.1f} us, two "
            f"launches {dual_token['two_launches_us']:.1f} us per layer")
        chunked = measure_chunked(torch, ckv, layers, kv_ptrs, s, w, scale, args.steps, stream)
        log(f"chunked (landmarks per {chunked['chunk']} rows): {chunked['ms_per_step']:.3f} "
            f"ms/step, {chunked['tokens_per_s']:.0f} tokens/s")
        idx = [torch.empty((B, Hkv, k), dtype=torch.int32, device=dev) for _ in range(L)]
        nsel = [torch.empty((B, Hkv), dtype=torch.int32, device=dev) for _ in range(L)]
        out = [torch.empty((B, Hq, d), dtype=torch.float32, device=dev) for _ in range(L)]
        for l, t in enumerate(layers):  # the eager reference of the graph's first replay
            kp, vp = kv_ptrs[l]
            ckv.critical_kv_attn(s, t["q"], None, kp, t["ctx_lens"], k, scale, kp, vp,
                                 ckv.SRC_DEVICE, None, None, None, idx[l], nsel[l], out[l],
                                 ws, stream)
        torch.cuda.synchronize()
        graph = measure_graph(torch, ckv, layers, kv_ptrs, s, w, scale, args.steps, idx, out)
        log(f"graph replay: {graph['ms_per_step']:.3f} ms/step, {graph['tokens_per_s']:.0f} "
            f"tokens/s, bit-identical {graph['bit_identical_to_eager']}")
        del idx, nsel, out, ws
        result.update(chunked=chunked, graph=graph, dual_token=dual_token)
    if "pipelined" in sections:
        pipelined_hbm = measure_pipelined_hbm(torch, ckv, layers, kv_ptrs, s, w, scale,
                                              args.steps, stream)
        log(f"pipelined, HBM: {pipelined_hbm['ms_per_step']:.3f} ms/step, "
            f"{pipelined_hbm['tokens_per_s']:.0f} tokens/s, per layer "
            f"{pipelined_hbm['per_layer_us']}")
        result.update(pipelined_hbm=pipelined_hbm)

    if "sweep" in sections and len(layers) == L:
        sweep = measure_attn_sweep(torch, ckv, layers, kv_ptrs, s, w, scale, stream)
        log("attention sweep: " + ", ".join(
            f"k{r['k']}: select_attn {r['select_attn_us']:.1f} us, attn {r['attn_us']:.1f} us"
            for r in sweep["points"]) + f"; fits {sweep.get('select_attn_fit')} "
            f"{sweep.get('attn_fit')}")
        result["attn_sweep"] = sweep
        cap = measure_read_cap(torch, ckv, layers, kv_ptrs, s, w, scale, stream)
        log("read cap (the selected rows read with each attention form's pattern, no "
            "arithmetic): " + ", ".join(f"{m} {r['us']:.1f} us ({r['frac_of_peak']:.2f})"
                                        for m, r in cap["forms"].items()))
        result["attn_read_cap"] = cap

    host_link = None
    if "host_link" in sections:
        host_link = measure_host_link(torch, ckv, dev)
        log(f"host link: {host_link}")
        result["host_link"] = host_link
    del layers[1:]  # keep layer 0 for the CPU baseline
    torch.cuda.empty_cache()
    pipeline = {}
    if "long128k" in sections:
        pipeline.update(measure_pipeline(torch, ckv, synth, dev, np, host_link,
                                         steps=args.loop_steps,
                                         runs=("plain", "corrected", "lowrank", "chunk8")))
        log(f"pipeline long128k: {pipeline}")
        torch.cuda.empty_cache()
    if "dual64" in sections:
        # the dual-token serving workload: 64 requests of ragged contexts
        pipeline["dual64"] = measure_pipeline(torch, ckv, synth, dev, np, host_link, "dual64",
                                              n_hbm=2, n_host=1, steps=args.loop_steps,
                                              runs=("plain",))
        log(f"pipeline dual64: {pipeline['dual64']}")
        torch.cuda.empty_cache()
    if "million" in sections:
        # the million-token single request
        pipeline["million"] = measure_pipeline(torch, ckv, synth, dev, np, host_link, "million",
                                               n_hbm=2, n_host=2, steps=args.loop_steps,
                                               runs=("plain", "chunk8"), layer_queries=True)
        log(f"pipeline million: {pipeline['million']}")
    if pipeline:
        result["pipeline"] = pipeline
    if "cpu" in sections:
        cpu = cpu_baseline(layers, w, scale, np)
        log(f"cpu baseline: {cpu}")
        result["cpu_baseline"] = cpu
    print(json.dumps(result), flush=True)
    return 0


def measure_main(torch, ckv, layers, kv_ptrs, s, w, scale, args, stream, stamp_every=31):
    """The headline: the Llama-8B same-step decode step, K steps timed by
    events on the compute stream (one more event after each step gives the
    per-step times and their median).  Inside the timed steps one launch in
    `stamp_every` of the dominant kernel carries dispatch-stamped events: its
    average duration there gives the roofline.  A stamped dispatch costs a few
    microseconds more than a plain one, so only a sample is stamped (one launch
    in 31: prime to the 32 layers, so the stamps move through all of them);
    the same steps are timed once more with no stamp at all."""
    B, Hq, Hkv, d, n, k, L = (w.batch, w.q_heads, w.kv_heads, w.head_dim, w.max_ctx, w.k,
                              w.layers)
    dev = torch.device("cuda:0")
    ws = ckv.workspace(s, k, ckv.ENTRY_CRITICAL_KV_ATTN)
    idx = [torch.empty((B, Hkv, k), dtype=torch.int32, device=dev) for _ in range(L)]
    nsel = [torch.empty((B, Hkv), dtype=torch.int32, device=dev) for _ in range(L)]
    out = [torch.empty((B, Hq, d), dtype=torch.float32, device=dev) for _ in range(L)]

    def step():
        for l, t in enumerate(layers):
            kp, vp = kv_ptrs[l]
            ckv.critical_kv_attn(s, t["q"], None, kp, t["ctx_lens"], k, scale, kp, vp,
                                 ckv.SRC_DEVICE, None, None, None, idx[l], nsel[l], out[l],
                                 ws, stream)

    def timed(steps):
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
        ev[0].record(stream)
        for i in range(steps):
            step()
            ev[i + 1].record(stream)
        torch.cuda.synchronize()
        per = [ev[i].elapsed_time(ev[i + 1]) for i in range(steps)]
        return ev[0].elapsed_time(ev[steps]) / steps, per

    log(f"warmup {args.warmup} steps")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # Breakdown (untimed): every kernel class stamped for a few steps.
    nb = 3
    ckv.profile_begin()
    timed(nb)
    kstats = ckv.profile_end()
    per_kernel = {name: {"launches": c, "avg_us": 1e3 * tot / c, "max_us": 1e3 * mx,
                         "ms_per_step": tot / nb}
                  for name, (c, tot, mx) in kstats.items()}
    dominant = max(kstats, key=lambda kname: kstats[kname][1])
    # Timed region: one launch in stamp_every of the dominant kernel carries
    # dispatch-stamped start/end events on `stream`.
    ckv.profile_begin([dominant], every=stamp_every)
    ms_step, per_step = timed(args.steps)
    dstats = ckv.profile_end()
    ms_plain, _ = timed(args.steps)  # same steps with no stamps at all (overhead check)
    # the same steps with the scoring launch and the selection and attention
    # launch apart (the two-launch form: the same index sets, the outputs
    # within fp32 rounding), for comparison
    ckv.set_one_launch_same_step(False)
    try:
        ms_two, _ = timed(args.steps)
    finally:
        ckv.set_one_launch_same_step(True)
    log(f"  {ms_step:.3f} ms/step, median {median(per_step):.3f} ({ms_plain:.3f} ms/step "
        f"unstamped, {ms_two:.3f} with the layer as two launches)")
    log("  per layer: " + ", ".join(f"{kname} {v['avg_us']:.1f} us"
                                   for kname, v in per_kernel.items()))
    assert all(torch.isfinite(o).all().item() for o in out[:2])

    tokens_per_s = B / (ms_step * 1e-3)
    launches, total_ms, _ = dstats[dominant]
    avg_s = total_ms / launches * 1e-3
    units = B * Hkv
    algo = {
        # key scan: every key of every unit once (n d bf16 per unit)
        "score": units * n * d * 2,
        # selected K and V rows once (2 k d bf16 per unit)
        "attn": units * k * 2 * d * 2,
        # the same rows, attended by the one-launch selection and attention
        # (its reads of the scores are implementation bytes)
        "select_attn": units * k * 2 * d * 2,
        # the layer in one launch: the key scan and the selected rows
        "critical": units * n * d * 2 + units * k * 2 * d * 2,
    }
    algo_bytes = algo.get(dominant)
    achieved = algo_bytes / avg_s / 1e9 if algo_bytes else None
    traffic = read_counters(dominant)
    roofline = {
        "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
        "frac": achieved / HBM_PEAK_GBPS if achieved else None, "traffic": traffic,
        "kernel": dominant, "algorithmic_bytes_per_launch": algo_bytes,
        "avg_launch_us": avg_s * 1e6, "stamped_launches": launches,
        "stamped": f"one launch in {stamp_every} inside the timed steps",
    }
    # every kernel of the step against the same peak, from the breakdown's
    # stamped durations (algorithmic bytes: keys for scoring, selected rows for
    # attention; the selection and the merge move implementation bytes only)
    for kname, v in per_kernel.items():
        if kname in algo:
            v["algorithmic_bytes"] = algo[kname]
            v["achieved_GBps"] = algo[kname] / (v["avg_us"] * 1e-6) / 1e9
            v["frac_of_peak"] = v["achieved_GBps"] / HBM_PEAK_GBPS
    step_bytes = L * (algo["score"] + algo["attn"])
    log(f"dominant kernel {dominant}: {avg_s * 1e6:.1f} us/launch, "
        f"{achieved:.0f} GB/s algorithmic")
    del idx, nsel, out, ws
    return {"value": tokens_per_s, "ms_per_step": ms_step,
            "ms_per_step_median": median(per_step), "ms_per_step_unstamped": ms_plain,
            "ms_per_step_two_launches": ms_two,
            "hbm_algorithmic_gbps_step": step_bytes / (ms_step * 1e-3) / 1e9,
            "kernels": per_kernel, "roofline": roofline}


def measure_attn_sweep(torch, ckv, layers, kv_ptrs, shape, w, scale, stream,
                       budgets=(512, 1024, 1536, 2048), reps=32):
    """The attention's time against its bytes at the Llama-8B shape (B16, 32 q
    / 8 KV heads, n 32768): budgets k from 512 to 2048 rows per KV head, so
    that the selected bytes grow while the grids keep their shape (up to
    2048 the one-launch kernel keeps one form: two workgroups per unit, each
    over the whole set with half the heads).  Two
    kernels: the same-step layer's one-launch selection and attention (over
    the 32 layers in turn, so that no call finds its rows in a cache), and the
    standalone attention over assembled buffers (distinct buffers totalling
    1 GiB per budget, for the same reason).  A line through the points, time
    = fixed + bytes / rate, splits a launch into what does not grow with the
    bytes (launch, selection, first round trip, the waves' merge, drain) and the
    streaming rate of the selected rows.  Dispatch-stamped kernel times.  The
    same-step calls run in the two-launch form here, so that the selection
    and attention launch is timed apart from the scoring."""
    ckv.set_one_launch_same_step(False)
    try:
        return _attn_sweep(torch, ckv, layers, kv_ptrs, shape, w, scale, stream, budgets, reps)
    finally:
        ckv.set_one_launch_same_step(True)


def _attn_sweep(torch, ckv, layers, kv_ptrs, shape, w, scale, stream, budgets, reps):
    import numpy as np
    dev = torch.device("cuda:0")
    B, Hq, Hkv, d = w.batch, w.q_heads, w.kv_heads, w.head_dim
    L = len(layers)
    points = []
    i32 = dict(dtype=torch.int32, device=dev)
    for k in budgets:
        ws = ckv.workspace(shape, k, ckv.ENTRY_CRITICAL_KV_ATTN)
        idx = [torch.empty((B, Hkv, k), **i32) for _ in range(L)]
        nsel = [torch.empty((B, Hkv), **i32) for _ in range(L)]
        out = torch.empty((B, Hq, d), device=dev)

        def same_step(l):
            kp, vp = kv_ptrs[l]
            ckv.critical_kv_attn(shape, layers[l]["q"], None, kp, layers[l]["ctx_lens"], k,
                                 scale, kp, vp, ckv.SRC_DEVICE, None, None, None, idx[l],
                                 nsel[l], out, ws, stream)
        for l in range(L):
            same_step(l)
        row_bytes = B * Hkv * k * 2 * d * 2
        nbuf = max(2, min(L, (1 << 30) // row_bytes))
        bufs = []
        for l in range(nbuf):
            kb = torch.empty((B, Hkv, k, d), dtype=torch.bfloat16, device=dev)
            vb = torch.empty_like(kb)
            ckv.gather_kv(shape, kv_ptrs[l][0], kv_ptrs[l][1], ckv.SRC_DEVICE, idx[l], nsel[l],
                          k, kb, vb, stream)
            bufs.append((kb, vb))
        wsa = ckv.workspace(shape, k, ckv.ENTRY_SPARSE_DECODE_ATTN)
        torch.cuda.synchronize()
        ckv.profile_begin(["select_attn", "attn", "combine"])
        for r in range(reps):
            same_step(r % L)
        for r in range(reps):
            kb, vb = bufs[r % nbuf]
            ckv.sparse_decode_attn(shape, layers[r % L]["q"], kb, vb, nsel[r % nbuf], k, scale,
                                   out, wsa, stream)
        st = ckv.profile_end()
        avg = {kname: 1e3 * tot / c for kname, (c, tot, _) in st.items()}
        points.append({"k": k, "row_bytes": row_bytes, "buffers": nbuf,
                       "select_attn_us": avg.get("select_attn", float("nan")),
                       "attn_us": avg.get("attn", float("nan")),
                       "combine_launches_us": avg.get("combine", float("nan"))})
        del ws, idx, nsel, out, bufs, wsa
        torch.cuda.empty_cache()
    res = {"points": points,
           "workload": "Llama-8B shape (B16, 32 q / 8 KV heads, head_dim 128, n 32768), "
                       f"budgets k {list(budgets)}; the same-step calls cycle over the {L} "
                       "layers, the standalone attention over distinct buffers of 1 GiB in all"}
    x = np.array([p["row_bytes"] for p in points], dtype=np.float64)
    for key in ("select_attn_us", "attn_us"):
        y = np.array([p[key] for p in points])
        if np.all(np.isfinite(y)):
            slope, icpt = np.polyfit(x, y, 1)
            res[key.replace("_us", "_fit")] = {
                "fixed_us": icpt, "marginal_GBps": 1e-3 / slope if slope > 0 else None,
                "marginal_frac_of_peak": (1e-3 / slope) / HBM_PEAK_GBPS if slope > 0 else None}
    return res


def measure_read_cap(torch, ckv, layers, kv_ptrs, shape, w, scale, stream, k=2048, reps=32):
    """What the memory system gives the attention's access pattern at the
    Llama-8B shape: the read-rate probe (ckv_probe_read_rows) reads the rows
    each layer's same-step selection chose (k 2048 per KV head, 128 MiB of K
    and V per launch) with the grid and load schedule of each attention form
    and no arithmetic, cycling the 32 distinct layers so that no launch finds
    its rows in a cache.  Dispatch-stamped kernel times."""
    dev = torch.device("cuda:0")
    B, Hq, Hkv, d = w.batch, w.q_heads, w.kv_heads, w.head_dim
    L = len(layers)
    i32 = dict(dtype=torch.int32, device=dev)
    ws = ckv.workspace(shape, k, ckv.ENTRY_CRITICAL_KV_ATTN)
    idx = [torch.empty((B, Hkv, k), **i32) for _ in range(L)]
    nsel = torch.empty((B, Hkv), **i32)
    out = torch.empty((B, Hq, d), device=dev)
    for l in range(L):
        kp, vp = kv_ptrs[l]
        ckv.critical_kv_attn(shape, layers[l]["q"], None, kp, layers[l]["ctx_lens"], k, scale,
                             kp, vp, ckv.SRC_DEVICE, None, None, None, idx[l], nsel, out, ws,
                             stream)
    row_bytes = B * Hkv * k * 2 * d * 2
    forms = {"standalone": ckv.PROBE_STANDALONE, "row_halves": ckv.PROBE_ROW_HALVES,
             "head_halves": ckv.PROBE_HEAD_HALVES}
    res = {}
    for name, mode in forms.items():
        sink = torch.empty(ckv.probe_sink_words(shape, k, mode), **i32)
        for l in range(4):  # warm
            ckv.probe_read_rows(shape, kv_ptrs[l][0], kv_ptrs[l][1], idx[l], k, mode, sink, stream)
        torch.cuda.synchronize()
        ckv.profile_begin(["probe"])
        for r in range(reps):
            l = r % L
            ckv.probe_read_rows(shape, kv_ptrs[l][0], kv_ptrs[l][1], idx[l], k, mode, sink, stream)
        st = ckv.profile_end()
        c, tot, mx = st["probe"]
        us = 1e3 * tot / c
        gbps = row_bytes / (us * 1e-6) / 1e9
        res[name] = {"us": us, "max_us": 1e3 * mx, "launches": c, "GBps": gbps,
                     "frac_of_peak": gbps / HBM_PEAK_GBPS}
        del sink
    del ws, idx
    torch.cuda.empty_cache()
    return {"forms": res, "bytes_per_launch": row_bytes,
            "workload": f"Llama-8B shape (B16, 32 q / 8 KV heads, n 32768), the same-step sets "
                        f"at k {k} of the {L} layers in turn"}


def measure_host_link(torch, ckv, dev):
    """Host-link rates: a contiguous pinned->device copy (the link's ceiling)
    and the zero-copy row gather of one long-context layer (B8, 8 KV heads,
    131072 positions, k 4096, K|V rows interleaved in pinned memory)."""
    import numpy as np
    mib = 1 << 20
    src = torch.empty(1024 * mib, dtype=torch.uint8, pin_memory=True)
    dst = torch.empty(1024 * mib, dtype=torch.uint8, device=dev)
    for _ in range(2):
        dst.copy_(src, non_blocking=True)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(5):
        dst.copy_(src, non_blocking=True)
    e1.record()
    torch.cuda.synchronize()
    copy_gbps = 5 * src.numel() / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del src, dst

    B, Hkv, n, k, d = 8, 8, 131072, 4096, 128
    kv = torch.empty((B, Hkv, n, 2, d), dtype=torch.bfloat16, pin_memory=True)
    rng = np.random.default_rng(0)
    idx = np.stack([np.sort(rng.choice(n, k, replace=False)) for _ in range(B * Hkv)])
    idx_t = torch.from_numpy(idx.astype(np.int32).reshape(B, Hkv, k)).to(dev)
    nsel = torch.full((B, Hkv), k, dtype=torch.int32, device=dev)
    kb = torch.empty((B, Hkv, k, d), dtype=torch.bfloat16, device=dev)
    vb = torch.empty_like(kb)
    s = ckv.shape_for(B, 32, Hkv, n, kv_row_stride=2 * d)
    base = kv.data_ptr()

    def gather():
        ckv.gather_kv(s, base, base + 2 * d, ckv.SRC_HOST_PINNED, idx_t, nsel, k, kb, vb)

    for _ in range(2):
        gather()
    torch.cuda.synchronize()
    ckv.profile_begin()
    reps = 20
    for _ in range(reps):
        gather()
    st = ckv.profile_end()
    c, tot, mx = st["gather"]
    gbytes = B * Hkv * k * 2 * d * 2
    gather_gbps = gbytes / (tot / c * 1e-3) / 1e9
    del kv
    return {"gather_GBps": gather_gbps, "h2d_copy_GBps": copy_gbps,
            "frac_of_copy": gather_gbps / copy_gbps, "bytes_per_gather": gbytes,
            "gathers": c, "avg_gather_us": 1e3 * tot / c, "max_gather_us": 1e3 * mx,
            "workload": "B8, 8 KV heads, n 131072, k 4096, 512-byte K|V rows, pinned host; "
                        "2 untimed and 20 timed gathers (the only gathers of "
                        "`bench.py --sections host_link`)"}


def measure_dual_token(torch, ckv, w, scale, stream, reps=50):
    """Sec. 5.2's co-batched attention at the Llama-8B shape (B16, 32 q / 8 KV
    heads, k 2048 gathered rows): the current and the speculative token in one
    launch against two attention calls, one per token.  Times per layer from
    events around `reps` repetitions, each layer on its own buffers (32 sets,
    so no repetition finds its rows in a cache)."""
    B, Hq, Hkv, d, k, L = w.batch, w.q_heads, w.kv_heads, w.head_dim, w.k, w.layers
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev)
    g.manual_seed(77)
    bf = lambda *shape: torch.randn(shape, generator=g, device=dev).to(torch.bfloat16)
    bufs = [(bf(B, Hkv, k, d), bf(B, Hkv, k, d)) for _ in range(L)]
    q1, q2 = bf(B, Hq, d), bf(B, Hq, d)
    kl, vl = bf(B, Hkv, 2, d), bf(B, Hkv, 2, d)
    n_sel = torch.full((B, Hkv), k, dtype=torch.int32, device=dev)
    o1, o2 = torch.empty((B, Hq, d), device=dev), torch.empty((B, Hq, d), device=dev)
    s = ckv.shape_for(B, Hq, Hkv, w.max_ctx)
    ws2 = ckv.workspace(s, k, ckv.ENTRY_DUAL_TOKEN_ATTN)
    ws1 = ckv.workspace(s, k, ckv.ENTRY_SPARSE_DECODE_ATTN)

    def co(l):
        ckv.dual_token_attn(s, q1, q2, bufs[l][0], bufs[l][1], n_sel, kl, vl, k, scale, o1, o2,
                            ws2, stream)

    def two(l):
        ckv.sparse_decode_attn(s, q1, bufs[l][0], bufs[l][1], n_sel, k, scale, o1, ws1, stream)
        ckv.sparse_decode_attn(s, q2, bufs[l][0], bufs[l][1], n_sel, k, scale, o2, ws1, stream)

    res = {}
    for name, fn in (("co_batched_us", co), ("two_launches_us", two)):
        for l in range(L):
            fn(l)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for r in range(reps):
            fn(r % L)
        e1.record(stream)
        torch.cuda.synchronize()
        res[name] = 1e3 * e0.elapsed_time(e1) / reps
    res["saving"] = 1.0 - res["co_batched_us"] / res["two_launches_us"]
    res["workload"] = ("B16, 32 q / 8 KV heads, k 2048 gathered rows per KV head; the two "
                       "tokens' own rows under the causal mask (co-batched only)")
    del bufs
    return res


def measure_chunked(torch, ckv, layers, kv_ptrs, shape, w, scale, steps, stream,
                    chunk=8):
    """The same Llama-8B step with chunk landmarks (the paper's index source):
    every layer scores the mean keys of 8-row chunks, selects k/8 chunks and
    attends over their rows in place.  Landmarks are built once beforehand (at
    prefill time, not timed): 1/8 of the keys' size."""
    B, Hq, Hkv, d, n, k = w.batch, w.q_heads, w.kv_heads, w.head_dim, w.max_ctx, w.k
    dev = torch.device("cuda:0")
    cmax = (n + chunk - 1) // chunk
    lms = []
    for l, t in enumerate(layers):
        lm = torch.empty((B, Hkv, cmax, d), dtype=torch.bfloat16, device=dev)
        ckv.chunk_landmarks(shape, chunk, kv_ptrs[l][0], t["ctx_lens"], lm, stream)
        lms.append(lm)
    i32 = dict(dtype=torch.int32, device=dev)
    cidx = torch.empty((B, Hkv, k // chunk), **i32)
    nch = torch.empty((B, Hkv), **i32)
    rows = [torch.empty((B, Hkv, k), **i32) for _ in layers]
    nrows = [torch.empty((B, Hkv), **i32) for _ in layers]
    out = [torch.empty((B, Hq, d), device=dev) for _ in layers]
    ws = ckv.workspace(shape, k, ckv.ENTRY_CRITICAL_KV_ATTN)

    def step():
        for l, t in enumerate(layers):
            kp, vp = kv_ptrs[l]
            ckv.chunked_kv_attn(shape, chunk, t["q"], None, lms[l], t["ctx_lens"], k, scale,
                                kp, vp, ckv.SRC_DEVICE, cidx, nch, rows[l], nrows[l], out[l],
                                ws, stream)

    for _ in range(3):
        step()
    torch.cuda.synchronize()
    ckv.profile_begin()
    step()
    torch.cuda.synchronize()
    per = {kname: round(1e3 * tot / c, 1) for kname, (c, tot, _) in ckv.profile_end().items()}
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    del lms
    return {"chunk": chunk, "ms_per_step": ms, "tokens_per_s": B / (ms * 1e-3),
            "per_layer_us": per, "landmark_bytes_per_layer": B * Hkv * cmax * d * 2,
            "workload": "the Llama-8B step above, chunk landmarks of 8 rows, k 2048 rows "
                        "(256 chunks) per KV head"}


def measure_graph(torch, ckv, layers, kv_ptrs, shape, w, scale, steps, ref_idx, ref_out):
    """The same Llama-8B step captured once into a HIP graph and replayed, as
    a serving loop would run it: the 128 launches of a step go to the device
    as one graph launch.  Every replay recomputes everything from the inputs;
    the first replay's index sets and outputs are checked bit for bit against
    the eager step's."""
    B, Hq, Hkv, d, k, L = w.batch, w.q_heads, w.kv_heads, w.head_dim, w.k, w.layers
    dev = torch.device("cuda:0")
    i32 = dict(dtype=torch.int32, device=dev)
    idx = [torch.empty((B, Hkv, k), **i32) for _ in range(L)]
    nsel = [torch.empty((B, Hkv), **i32) for _ in range(L)]
    out = [torch.empty((B, Hq, d), device=dev) for _ in range(L)]
    ws = ckv.workspace(shape, k, ckv.ENTRY_CRITICAL_KV_ATTN)

    def step():  # on the current stream: the capture stream inside the capture
        for l, t in enumerate(layers):
            kp, vp = kv_ptrs[l]
            ckv.critical_kv_attn(shape, t["q"], None, kp, t["ctx_lens"], k, scale, kp, vp,
                                 ckv.SRC_DEVICE, None, None, None, idx[l], nsel[l], out[l], ws)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()
    for o in out:
        o.fill_(float("nan"))
    graph.replay()
    torch.cuda.synchronize()
    same = all(torch.equal(idx[l], ref_idx[l]) and torch.equal(out[l], ref_out[l])
               for l in range(L))
    stream = torch.cuda.current_stream()
    for _ in range(3):
        graph.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        graph.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    del graph, idx, nsel, out, ws
    return {"ms_per_step": ms, "tokens_per_s": B / (ms * 1e-3), "bit_identical_to_eager": same,
            "workload": "the Llama-8B step above (same-step, K/V in HBM), one graph launch "
                        "per step"}


def measure_pipelined_hbm(torch, ckv, layers, kv_ptrs, shape, w, scale, steps, stream):
    """The Llama-8B step in the paper's pipelined form with the caches in HBM
    (Sec. 4.1: the set a layer attends over at step t was selected at step
    t-1 from the speculative token's query), run by the library's decode loop
    without buffers: per layer one launch attends with the current query over
    last step's set, read in place through its indices, and scores the keys
    with the speculative query; the selection then picks next step's set.
    Index sets alternate between two arrays per layer by step parity.  Queries
    are step-invariant: the current one is the layer's, the speculative one
    bf16(0.8 q + 0.6 noise).  A second run co-batches the two tokens (Sec.
    5.2): in the same launch the speculative token also attends over the set
    and both tokens over their own new rows (causal mask)."""
    B, Hq, Hkv, d, k, L = w.batch, w.q_heads, w.kv_heads, w.head_dim, w.k, w.layers
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev)
    g.manual_seed(4321)
    qs = [(0.8 * t["q"].float() + 0.6 * torch.randn(t["q"].shape, generator=g, device=dev))
          .to(torch.bfloat16) for t in layers]
    local = [(torch.randn((B, Hkv, 2, d), generator=g, device=dev).to(torch.bfloat16),
              torch.randn((B, Hkv, 2, d), generator=g, device=dev).to(torch.bfloat16))
             for _ in layers]
    i32 = dict(dtype=torch.int32, device=dev)
    idx = [[torch.empty((B, Hkv, k), **i32) for _ in range(L)] for _ in range(2)]
    nsel = [[torch.empty((B, Hkv), **i32) for _ in range(L)] for _ in range(2)]
    out = [torch.empty((B, Hq, d), device=dev) for _ in range(L)]
    out_spec = [torch.empty((B, Hq, d), device=dev) for _ in range(L)]
    ws = ckv.workspace(shape, k, ckv.ENTRY_DECODE_STEP)
    lens = layers[0]["ctx_lens"]
    assert all(torch.equal(t["ctx_lens"], lens) for t in layers)

    def one_run(two):
        io = [ckv.layer_array([{"q_att": t["q"], "q_sel": qs[l], "k_score": kv_ptrs[l][0],
                                "k_src": kv_ptrs[l][0], "v_src": kv_ptrs[l][1],
                                "idx_prev": idx[c][l], "n_sel_prev": nsel[c][l],
                                "idx_next": idx[1 - c][l], "n_sel_next": nsel[1 - c][l],
                                "out": out[l],
                                "k_local": local[l][0] if two else None,
                                "v_local": local[l][1] if two else None,
                                "out_spec": out_spec[l] if two else None}
                               for l, t in enumerate(layers)])
              for c in range(2)]
        pipe = ckv.Pipeline()
        cur = [0]

        def step():
            pipe.step(shape, io[cur[0]], lens, k, scale, ckv.SRC_DEVICE, None, None, ws, stream,
                      None)
            cur[0] ^= 1

        # bootstrap (the pre-decoding step): same-step selection into set 0
        for l, t in enumerate(layers):
            kp, vp = kv_ptrs[l]
            ckv.critical_kv_attn(shape, t["q"], qs[l], kp, t["ctx_lens"], k, scale, kp, vp,
                                 ckv.SRC_DEVICE, None, None, None, idx[0][l], nsel[0][l],
                                 out[l], ws, stream)
        for _ in range(3):
            step()
        torch.cuda.synchronize()
        ckv.profile_begin()
        step()
        torch.cuda.synchronize()
        per = {kname: round(1e3 * tot / c, 1) for kname, (c, tot, _) in ckv.profile_end().items()}
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps):
            step()
        e1.record(stream)
        torch.cuda.synchronize()
        pipe.close()
        ms = e0.elapsed_time(e1) / steps
        assert all(torch.isfinite(o).all().item() for o in out[:2])
        if two:
            assert all(torch.isfinite(o).all().item() for o in out_spec[:2])
        dual_bytes = B * Hkv * (w.max_ctx * d * 2 + k * 2 * d * 2)
        res = {"ms_per_step": ms, "tokens_per_s": B / (ms * 1e-3), "per_layer_us": per}
        if "dual" in per:
            res["dual_bytes_per_launch"] = dual_bytes
            res["dual_GBps"] = dual_bytes / (per["dual"] * 1e-6) / 1e9
            res["dual_frac_of_peak"] = res["dual_GBps"] / HBM_PEAK_GBPS
        return res

    res = one_run(False)
    res["workload"] = ("the Llama-8B step above, pipelined through the decode loop without "
                       "buffers: attention over last step's set read in place from HBM and "
                       "scoring with the speculative query in one launch per layer")
    res["two_tokens"] = one_run(True)
    res["two_tokens"]["workload"] = (
        "the same loop with both tokens attending in that launch (2G head rows: the current "
        "token over the set and its own row, the speculative token over the set and both "
        "rows, causal mask), outputs for both tokens per step")
    del qs, idx, nsel, out, out_spec, ws, local
    return res


_STREAMS = []


def _pipeline_streams(torch):
    """The compute and copy streams of every decode loop.  The runtime gives
    a stream its hardware queue at the stream's first use, a fresh one while
    fewer than its maximum exist (4 by default), else a shared one; a copy
    stream sharing the compute stream's queue would serialise the loop.  So
    the first call, made before anything else runs, puts one small kernel on
    the default stream, then on each of the two (three fresh queues)."""
    if not _STREAMS:
        cs, xs = torch.cuda.Stream(), torch.cuda.Stream()
        torch.zeros(1, device="cuda")
        for st in (cs, xs):
            with torch.cuda.stream(st):
                torch.zeros(1, device="cuda")
        torch.cuda.synchronize()
        _STREAMS.extend([cs, xs])
    return _STREAMS[0], _STREAMS[1]


def measure_pipeline(torch, ckv, synth, dev, np, host_link, wl="long128k", n_hbm=4, n_host=2,
                     steps=20, runs=("plain", "corrected", "lowrank"), layer_queries=False,
                     gather_width=0, warm=2, stamped=3):
    """The two-buffer decode loop of 32 layers on a host-pinned workload: the
    long-context one (B8, 32 q / 8 KV heads, n 131072, k 4096) or the
    dual-token one (B64, n_b ~ U{16384..65536}, k 2048); K|V rows in pinned
    host memory, scoring keys in HBM.  Layer inputs cycle over n_hbm distinct
    HBM and n_host distinct host layers (each far larger than any cache);
    queries are distinct per layer and step.  The speculative query of step t is 0.8 x the query of step
    t+1 plus 0.6 x noise (the dual workload's recipe).  Two runs over the same
    inputs: attention over the prefetched prediction, and with miss correction
    (each layer attends over its own query's set, misses fetched on the compute
    stream); a third run rebuilds the misses' keys in every layer from rank-32
    factors (per (request, KV head), one set per host layer) and fetches only
    their values.  Step time from events on the compute stream after it has
    joined the copy stream: the median over `steps` unstamped steady-state
    steps (events after every step), after `warm` untimed steps; a further
    `stamped` steps with every kernel stamped give the per-kernel times.
    layer_queries: every step's query of a layer is
    the workload's own query of that layer (the million-token keys cluster
    along it), instead of fresh draws per step."""
    w = synth.WORKLOADS[wl]
    B, Hq, Hkv, d, n, k, L = (w.batch, w.q_heads, w.kv_heads, w.head_dim, w.max_ctx, w.k,
                              w.layers)
    scale = float(np.float32(1.0 / math.sqrt(d)))
    kscore, hosts, lq = [], [], []
    for i in range(n_hbm):
        t = synth.make_layer(w, seed=0, layer=i, device=dev)
        if i < n_host:
            hosts.append(synth.host_kv(t["k"], t["v"]))
        kscore.append(t["k"])
        lq.append(t["q"])
        lens = t["ctx_lens"]
        del t
    torch.cuda.empty_cache()
    g = torch.Generator(device=dev)
    g.manual_seed(1234)
    total_steps = warm + steps + stamped
    if layer_queries:
        q = [[lq[l % n_hbm] for l in range(L)] for _ in range(total_steps + 1)]
    else:
        q = [[torch.randn((B, Hq, d), generator=g, device=dev).to(torch.bfloat16)
              for _ in range(L)] for _ in range(total_steps + 1)]
    qs = [[(0.8 * q[st + 1][l].float() + 0.6 * torch.randn((B, Hq, d), generator=g,
                                                           device=dev)).to(torch.bfloat16)
           for l in range(L)] for st in range(total_steps)]
    i32 = dict(dtype=torch.int32, device=dev)
    idx = [[torch.empty((B, Hkv, k), **i32) for _ in range(L)] for _ in range(2)]
    nsel = [[torch.empty((B, Hkv), **i32) for _ in range(L)] for _ in range(2)]
    idx_true = [torch.empty((B, Hkv, k), **i32) for _ in range(L)]
    n_true = [torch.empty((B, Hkv), **i32) for _ in range(L)]
    hits = [[torch.empty((B, Hkv), **i32) for _ in range(L)] for _ in range(total_steps)]
    out = [torch.empty((B, Hq, d), device=dev) for _ in range(L)]
    k_buf = [torch.empty((B, Hkv, k, d), dtype=torch.bfloat16, device=dev) for _ in range(2)]
    v_buf = [torch.empty_like(k_buf[0]) for _ in range(2)]
    shape = ckv.shape_for(B, Hq, Hkv, n, kv_row_stride=2 * d)
    ws = ckv.workspace(shape, k, ckv.ENTRY_DECODE_STEP)
    compute, copy = _pipeline_streams(torch)
    s1 = ckv.shape_for(B, Hq, Hkv, n)
    sc = torch.empty((B, Hkv, n), device=dev)
    wsel = ckv.workspace(s1, k, ckv.ENTRY_SELECT_TOPK)
    wchunk = ckv.workspace(s1, k, ckv.ENTRY_CRITICAL_KV_ATTN) if any(
        r.startswith("chunk") for r in runs) else None
    cidx = {int(r[len("chunk"):]): torch.empty((B, Hkv, k // int(r[len("chunk"):])), **i32)
            for r in runs if r.startswith("chunk")}
    nch = torch.empty((B, Hkv), **i32)

    lr_rank = 32
    lr = []

    lms = {}  # chunk landmarks per (chunk, HBM layer), built once (prefill-time work)

    def landmarks(chunk, i):
        if (chunk, i) not in lms:
            cmax = (n + chunk - 1) // chunk
            lm = torch.empty((B, Hkv, cmax, d), dtype=torch.bfloat16, device=dev)
            ckv.chunk_landmarks(s1, chunk, kscore[i], lens, lm)
            lms[(chunk, i)] = lm
        return lms[(chunk, i)]

    def run(corrected, lowrank=False, chunk=1):
        def io(step, cur):
            return [{"q_att": q[step][l], "q_sel": qs[step][l], "k_score": kscore[l % n_hbm],
                     "k_src": hosts[l % n_host].data_ptr(),
                     "v_src": hosts[l % n_host].data_ptr() + 2 * d,
                     "idx_prev": idx[cur][l], "n_sel_prev": nsel[cur][l],
                     "idx_next": idx[1 - cur][l], "n_sel_next": nsel[1 - cur][l],
                     "out": out[l],
                     "idx_true": idx_true[l] if corrected else None,
                     "n_true": n_true[l] if corrected else None,
                     "hits": hits[step][l] if corrected else None,
                     "lr_rank": lr_rank if lowrank else 0,
                     "lr_u": lr[l % n_host][0] if lowrank else None,
                     "lr_w": lr[l % n_host][1] if lowrank else None,
                     "chunk": chunk,
                     "landmarks": landmarks(chunk, l % n_hbm) if chunk > 1 else None}
                    for l in range(L)]

        # bootstrap selection (the pre-decoding step) into set 0
        for l in range(L):
            if chunk > 1:
                ckv.select_chunks(s1, chunk, q[0][l], landmarks(chunk, l % n_hbm), lens, k,
                                  scale, cidx[chunk], nch, idx[0][l], nsel[0][l], wchunk)
            else:
                ckv.score_keys(s1, q[0][l], kscore[l % n_hbm], lens, scale, sc)
                ckv.select_topk(s1, sc, lens, k, idx[0][l], nsel[0][l], wsel)
        torch.cuda.synchronize()
        pipe = ckv.Pipeline()
        if gather_width:
            pipe.set_gather_width(gather_width)
        copy.wait_stream(compute)
        pipe.prime(shape, k, io(0, 0), ckv.SRC_HOST_PINNED, k_buf, v_buf, copy)
        cur, st = 0, 0

        def one_step():
            nonlocal cur, st
            pipe.step(shape, io(st, cur), lens, k, scale, ckv.SRC_HOST_PINNED, k_buf, v_buf,
                      ws, compute, copy)
            cur, st = 1 - cur, st + 1

        for _ in range(warm):
            one_step()
        compute.wait_stream(copy)
        torch.cuda.synchronize()
        # timed, unstamped: an event on the compute stream after each step
        # (the copy stream keeps prefetching across step boundaries, as in
        # serving); the last event follows the compute stream's join with it
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 2)]
        first = st
        ev[0].record(compute)
        for i in range(steps):
            one_step()
            ev[i + 1].record(compute)
        compute.wait_stream(copy)
        ev[steps + 1].record(compute)
        torch.cuda.synchronize()
        per = [ev[i].elapsed_time(ev[i + 1]) for i in range(steps)]
        ms_mean = ev[0].elapsed_time(ev[steps + 1]) / steps
        ms = median(per)
        # breakdown (separate, untimed): every kernel stamped for a few steps
        ckv.profile_begin()
        for _ in range(stamped):
            one_step()
        compute.wait_stream(copy)
        torch.cuda.synchronize()
        stats = ckv.profile_end()
        pipe.close()
        host_bytes = L * B * Hkv * k * 2 * d * 2
        gather_ms = stats.get("gather", (0, 0.0, 0.0))[1] / stamped
        compute_ms = sum(v[1] for kname, v in stats.items() if kname != "gather") / stamped
        res = {"ms_per_step": ms, "ms_per_step_mean": ms_mean,
               "ms_per_step_min": min(per), "ms_per_step_max": max(per),
               "timed_steps": steps, "tokens_per_s": B / (ms * 1e-3),
               "host_bytes_per_step": host_bytes,
               "host_GBps_step": host_bytes / (ms * 1e-3) / 1e9,
               "stamped_steps": stamped,
               "gather_ms_per_step": gather_ms, "compute_kernels_ms_per_step": compute_ms,
               "kernels_ms_per_step": {kname: round(v[1] / stamped, 4)
                                       for kname, v in stats.items()},
               "overlap": (gather_ms + compute_ms) / ms,
               "refill_GBps": B * Hkv * k * 2 * d * 2 / (gather_ms / L * 1e-3) / 1e9,
               "gather_workgroups": gather_width or ("auto: 80" if n >= 64 * k else "auto: 256")}
        if corrected:  # the misses cross the link too, on the compute stream
            found = sum(int(hits[t][l].sum()) for t in range(first, first + steps)
                        for l in range(L))
            total = steps * L * B * Hkv * min(k, n)
            res["hit_rate"] = found / total
            # a rebuilt miss fetches its value only
            res["miss_bytes_per_step"] = (total - found) / steps * (1 if lowrank else 2) * d * 2
            res["host_bytes_per_step"] = host_bytes + res["miss_bytes_per_step"]
            res["host_GBps_step"] = res["host_bytes_per_step"] / (ms * 1e-3) / 1e9
        if host_link:
            res["frac_of_h2d_copy"] = res["host_GBps_step"] / host_link["h2d_copy_GBps"]
        return res

    res = run(False)
    for run_name in runs:
        if run_name.startswith("chunk"):  # chunk landmarks: contiguous-block refills
            c = int(run_name[len("chunk"):])
            r = run(False, chunk=c)
            r["chunk"] = c
            refill = r["gather_ms_per_step"] / L
            r["refill_us"] = 1e3 * refill
            r["refill_GBps"] = B * Hkv * k * 2 * d * 2 / (refill * 1e-3) / 1e9
            r["row_refill_GBps"] = res["refill_GBps"]
            res[run_name] = r
    ctx = (f"context {n}" if w.ctx_min == n else f"contexts U{{{w.ctx_min}..{n}}}")
    res["workload"] = (f"{wl} decode, {L} layers: B{B}, {Hq} q / {Hkv} KV heads, head_dim {d}, "
                       f"{ctx}, k {k}; K|V rows host-pinned, scoring keys in HBM; "
                       f"{n_hbm} HBM and {n_host} host layers cycled")
    if "corrected" in runs:
        res["corrected"] = run(True)
    if "lowrank" in runs:
        for i in range(n_host):
            lr.append(synth.low_rank_factors(w, lr_rank, seed=0, layer=i, device=dev))
        res["corrected_lowrank"] = run(True, lowrank=True)
        res["corrected_lowrank"]["rank"] = lr_rank
    del hosts, lr
    return res


def cpu_baseline(layers, w, scale, np):
    """The oracle (plain C, fp64, full sort) on the first layer of the same
    workload, every (request, KV head) unit, on this host's cores."""
    import oracle
    import synth
    o = oracle.get()
    try:
        cores = len(os.sched_getaffinity(0))
    except AttributeError:
        cores = os.cpu_count() or 1
    cores = max(1, min(cores, 16))
    t = layers[0]
    q = synth.to_u16(t["q"])
    if "kv" in t:
        K = synth.to_u16(t["kv"][:, :, :, 0].contiguous())
        V = synth.to_u16(t["kv"][:, :, :, 1].contiguous())
    else:
        K, V = synth.to_u16(t["k"]), synth.to_u16(t["v"])
    lens = t["ctx_lens"].cpu().numpy()
    so = o.shape(w.batch, w.q_heads, w.kv_heads, w.head_dim, w.max_ctx)
    # repeated until about 10 s of wall time: a bounded sample of the step
    runs, elapsed = 0, 0.0
    while elapsed < 10.0:
        t0 = time.perf_counter()
        o.critical_kv_attn(so, q, None, K, K, V, lens, w.k, scale, nthreads=cores)
        elapsed += time.perf_counter() - t0
        runs += 1
    sec_layer = elapsed / runs
    sec_step = sec_layer * w.layers
    # the tiny workload's layer (B1, 8/2 heads, n 4096, k 256) on one thread
    wt = synth.WORKLOADS["tiny"]
    tt = synth.make_layer(wt, seed=0)
    st = o.shape(wt.batch, wt.q_heads, wt.kv_heads, wt.head_dim, wt.max_ctx)
    qt, Kt, Vt = synth.to_u16(tt["q"]), synth.to_u16(tt["k"]), synth.to_u16(tt["v"])
    lt = tt["ctx_lens"].numpy()
    tiny_runs, t0 = 0, time.perf_counter()
    while time.perf_counter() - t0 < 1.0:
        o.critical_kv_attn(st, qt, None, Kt, Kt, Vt, lt, wt.k, scale, nthreads=1)
        tiny_runs += 1
    tiny_s = (time.perf_counter() - t0) / tiny_runs
    return {"value": w.batch / sec_step, "unit": "tokens/s", "cores": cores,
            "kind": "oracle", "cpu": cpu_name(), "seconds_per_step": sec_step,
            "sample": f"layer 0 of {w.layers}, all {w.units} (request, KV head) units, "
                      f"run {runs} times ({elapsed:.1f} s, {sec_layer:.2f} s each) and "
                      f"scaled x{w.layers} layers",
            "tiny_layer_one_thread_s": tiny_s,
            "tiny_sample": f"the tiny workload's layer (B1, 8/2 heads, n 4096, k 256) on one "
                           f"thread, {tiny_runs} runs"}


if __name__ == "__main__":
    sys.exit(main())
