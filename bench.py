"""Benchmark of the BACON prefill KV-compression pass on one MI355X.

One step = the whole pass of a prompt: bacon_begin_prompt and
bacon_compress_prompt over every layer (score -> calibrate -> select ->
compact per layer, the next layer's normaliser pass in the launch of this
layer's scoring pass); the per-layer calls (bacon_compress_layer) are timed
beside it,
on the 32K-token long-video GQA workload (32 layers, 32 query / 8 KV heads,
d = 128, window 32, budget 256, bf16).  Inputs are synthetic, seeded, and
resident in HBM before timing starts.

Prints one JSON line: keys scored per second (positions x KV heads x layers
per second), ms per step and per layer, a roofline entry for the dominant
kernel (its algorithmic bytes -- the per-layer bytes of the pass that the
launch completes: K read once, Q_win, E written -- over its mean launch time
from HIP events recorded around each launch on the pass's stream), the same
prompt call on every workload shape, and the fp64 CPU oracle timed on a
bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
COPY_BYTES = 1 << 30          # plain copy of the counter calibration (read once, written once)
METRIC = "KV compression pass ms/layer + keys scored/sec; HBM GB/s vs peak at N=32K"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def algorithmic_bytes(wl, persist_m=4):
    """Bytes a layer must move at minimum: K once, Q_win, the E history read and
    write, the gather of kept and window rows of K and V, and the indices."""
    es = wl.elem_size
    T, Hkv, d = wl.total_tokens, wl.num_kv_heads, wl.head_dim
    k_bytes = T * Hkv * d * es
    q_bytes = wl.batch * wl.window * wl.num_q_heads * d * es
    kept_rows = sum(b + wl.window for b in wl.budgets)
    gather = 2 * 2 * kept_rows * Hkv * d * es
    idx = 4 * sum(wl.budgets) * Hkv
    per_layer = []
    for l in range(wl.num_layers):
        ring = (min(persist_m, l) + 1) * T * Hkv * 4
        per_layer.append(k_bytes + q_bytes + ring + gather + idx)
    return {"k": k_bytes, "q": q_bytes, "layer_mean": float(np.mean(per_layer)),
            "layers": per_layer}


# Kernels (library timing names) by what they complete of a layer's pass.
# K passes that finish a layer's window score: its K read once, Q_win, E out.
SCORE_PASSES = ("window_score_calib_lse_kr", "window_score_calib_lse", "window_score_calib_kr",
                "window_score_calib", "window_score_single")
# Kernels whose work is only an intermediate of this design (a second read of
# K for the normalisers, the normaliser merge, pooled vectors, score keys and
# candidate lists): no algorithmic bytes of their own.
DESIGN_ONLY = ("window_lse_kr", "window_lse", "lse_merge", "segment_score", "segment_cand")


def kernel_bytes(name, wl, persist_m=4):
    """Algorithmic bytes (the per-layer units above) of the work one launch of
    a kernel of the measured path completes, mean over layers.  The launches
    of one layer add up to algorithmic_bytes()'s layer mean:
      K pass that finishes the window score   K + Q_win + E written
      calibration (segment_calib)             the earlier layers' E read for T
      final top-K and compaction              kept and window rows of K and V
                                              read and written, the indices
    A launch that holds the jobs of two layers (window_score_calib_lse*: pass 2
    of layer l with pass 1 of layer l+1) completes one layer's K pass."""
    ab = algorithmic_bytes(wl, persist_m)
    T, Hkv = wl.total_tokens, wl.num_kv_heads
    vec = T * Hkv * 4                                   # one fp32 value per (position, KV head)
    hist_reads = float(np.mean([min(persist_m, l) * vec for l in range(wl.num_layers)]))
    kept_rows = sum(b + wl.window for b in wl.budgets)
    if name in SCORE_PASSES:
        return ab["k"] + ab["q"] + vec
    if name in DESIGN_ONLY:
        return 0.0
    if name == "segment_calib":
        return hist_reads
    if name == "final_topk":
        return 2 * 2 * kept_rows * Hkv * wl.head_dim * wl.elem_size + 4 * sum(wl.budgets) * Hkv
    if name == "segment_calib_cand":                    # calibration, the previous layer's lists,
        return sum(kernel_bytes(k, wl, persist_m)      # the next layer's normaliser merge
                   for k in ("segment_calib", "segment_cand", "lse_merge"))
    if name == "segment_score_final":                   # scores, the previous layer's top-K
        return sum(kernel_bytes(k, wl, persist_m) for k in ("segment_score", "final_topk"))
    return 0.0


def design_bytes(name, wl, persist_m=4):
    """Bytes a launch moves in this design at minimum (beside the algorithmic
    ones): the dual launch reads two layers' K, pass 1 reads K again."""
    ab = algorithmic_bytes(wl, persist_m)
    vec = wl.total_tokens * wl.num_kv_heads * 4
    if name in ("window_score_calib_lse_kr", "window_score_calib_lse"):
        return 2 * (ab["k"] + ab["q"]) + 2 * vec
    if name in ("window_lse_kr", "window_lse"):
        return ab["k"] + ab["q"]
    if name in ("window_score_calib_kr", "window_score_calib", "window_score_single"):
        return ab["k"] + ab["q"] + 2 * vec
    return kernel_bytes(name, wl, persist_m)


def measured_traffic(kernel):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it
    was taken on the current kernel source."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path))
    except Exception:
        return None
    from paper_2606_14782_amd.counters import source_sha
    if rec.get("source_sha") != source_sha():
        return None
    k = rec.get("kernels", {}).get(kernel)
    return None if k is None else float(k["bytes_per_launch"])


def median_step_ms(fn, steps):
    """Median duration of `steps` calls of fn, each bracketed by HIP events on
    the current stream (no host synchronisation between calls)."""
    import torch
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    torch.cuda.synchronize()
    for e0, e1 in evs:
        e0.record()
        fn()
        e1.record()
    torch.cuda.synchronize()
    return float(np.median([e0.elapsed_time(e1) for e0, e1 in evs]))


def cpu_baseline(wl, budget_s, gpu_idx=None):
    """The fp64 oracle on this host, on layers 0.. of the same workload until
    about budget_s seconds have been spent (layers run in order)."""
    from oracle import ref
    from paper_2606_14782_amd import inputs
    ref.build(force=False)
    threads = min(os.cpu_count() or 1, 16)
    ref.set_threads(threads)
    used = min(threads, wl.batch * wl.num_kv_heads)
    p = ref.Prompt.for_workload(wl)
    spent, layers = 0.0, 0
    kept, differing = 0, 0
    while layers < wl.num_layers and spent < budget_s:
        x = inputs.layer_inputs(wl, layers)
        t0 = time.perf_counter()
        r = p.layer(layers, x["q_win"], x["k"])
        spent += time.perf_counter() - t0
        if gpu_idx is not None and layers < len(gpu_idx):
            # kept positions of each (sequence, KV head) that the GPU's set
            # and the oracle's do not share (near ties of the K-th score)
            off = 0
            for b in range(wl.batch):
                for h in range(wl.num_kv_heads):
                    K = int(wl.budgets[b])
                    o = set(r["idx"][off:off + K].tolist()) - {-1}
                    g = set(gpu_idx[layers][off:off + K].tolist()) - {-1}
                    kept += len(o)
                    differing += len(o - g)
                    off += K
        layers += 1
    keys = wl.total_tokens * wl.num_kv_heads * layers
    # the same oracle on one thread, on the first layer of a fresh prompt
    ref.set_threads(1)
    p1 = ref.Prompt.for_workload(wl)
    x = inputs.layer_inputs(wl, 0)
    t0 = time.perf_counter()
    p1.layer(0, x["q_win"], x["k"])
    one = time.perf_counter() - t0
    ref.set_threads(threads)
    return {"value": keys / spent, "unit": "keys/s", "cores": used, "kind": "oracle",
            "sample": f"layers 0-{layers - 1} of the {wl.num_layers}-layer workload "
                      f"({spent:.1f} s, OpenMP over (sequence, KV head))",
            "ms_per_layer": 1e3 * spent / layers,
            "one_thread": {"value": wl.total_tokens * wl.num_kv_heads / one, "unit": "keys/s",
                           "ms_per_layer": 1e3 * one, "sample": "layer 0"},
            "cpu_model": _cpu_model(),
            "kept_vs_gpu": None if gpu_idx is None else {
                "layers": min(layers, len(gpu_idx)), "kept": kept, "differing": differing}}


def prompt_rate(idx, steps, warmup):
    """The prompt call (bacon_begin_prompt + bacon_compress_prompt over every
    layer) on workload idx at its full shape: median step over `steps`."""
    import torch
    from paper_2606_14782_amd import bacon, inputs
    wl = inputs.workload(idx)
    dev = torch.device("cuda:0")
    tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    qs, ks, vs = [], [], []
    for l in range(wl.num_layers):
        x = inputs.layer_inputs(wl, l)
        qs.append(torch.from_numpy(x["q_win"]).to(dev).to(tdt))
        ks.append(torch.from_numpy(x["k"]).to(dev).to(tdt))
        vs.append(torch.from_numpy(x["v"]).to(dev).to(tdt))
    batch = bacon.BatchLayout(wl.cu_seqlens, wl.budgets_arr)
    ctx = bacon.Context(wl.num_layers, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.window,
                        wl.batch, wl.total_tokens, wl.dtype,
                        bacon.default_params(pool_kernel=wl.pool_kernel))
    outs = None

    def step():
        nonlocal outs
        ctx.bacon_begin_prompt(batch)
        outs = ctx.bacon_compress_prompt(0, batch, qs, ks, vs, outs=outs)

    for _ in range(warmup):
        step()
    ms = median_step_ms(step, steps)
    ab = algorithmic_bytes(wl)
    us_layer = 1e3 * ms / wl.num_layers
    keys = wl.total_tokens * wl.num_kv_heads / (us_layer * 1e-6)
    del qs, ks, vs, outs, ctx
    torch.cuda.empty_cache()
    return {"workload": wl.name, "layers": wl.num_layers, "us_per_layer": us_layer,
            "keys_per_s": keys, "bytes_per_layer": ab["layer_mean"],
            "hbm_frac": ab["layer_mean"] / (us_layer * 1e-6) / 1e9 / HBM_PEAK_GBS,
            "steps": steps}


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", type=int, default=3, help="workload index (default: 32K video)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the prompt call on the other workload shapes")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain fp32 copy of COPY_BYTES (read and written once) whose "
                         "HBM counters scale the kernels' counters")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported: the pass shards "
              f"by KV head with no exchange, so N GPUs each run this one-GPU workload on "
              f"H_kv/N heads.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2606_14782_amd import bacon, inputs

    wl = inputs.workload(args.workload)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    log(f"workload {wl.name}: generating {wl.num_layers} layers")
    batch = bacon.BatchLayout(wl.cu_seqlens, wl.budgets_arr)
    qs, ks, vs = [], [], []
    tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    for l in range(wl.num_layers):
        x = inputs.layer_inputs(wl, l)
        if l % 8 == 7:
            log(f"  layer {l + 1}/{wl.num_layers} generated")
        qs.append(torch.from_numpy(x["q_win"]).to(dev).to(tdt))
        ks.append(torch.from_numpy(x["k"]).to(dev).to(tdt))
        vs.append(torch.from_numpy(x["v"]).to(dev).to(tdt))
    params = bacon.default_params(pool_kernel=wl.pool_kernel)
    ctx = bacon.Context(wl.num_layers, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.window,
                        wl.batch, wl.total_tokens, wl.dtype, params)
    n_idx = batch.idx_count(wl.num_kv_heads)
    rows = batch.kept_rows(wl.window)
    outs = [(torch.empty(n_idx, dtype=torch.int32, device=dev),
             torch.empty((rows, wl.num_kv_heads, wl.head_dim), dtype=tdt, device=dev),
             torch.empty((rows, wl.num_kv_heads, wl.head_dim), dtype=tdt, device=dev))
            for _ in range(wl.num_layers)]

    def step():
        ctx.bacon_begin_prompt(batch)
        ctx.bacon_compress_prompt(0, batch, qs, ks, vs, outs=outs)

    def step_layers():
        ctx.bacon_begin_prompt(batch)
        for l in range(wl.num_layers):
            ctx.bacon_compress_layer(l, batch, qs[l], ks[l], vs[l], out=outs[l])

    if args.copy_calibration:
        n = COPY_BYTES // 4
        src = torch.randn(n, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        del src, dst
        log(f"copy calibration: {COPY_BYTES} bytes read and written, 3 launches")

    log("warmup")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    gpu_idx = [o[0].cpu().numpy() for o in outs[:8]]

    log(f"timing {args.steps} steps")
    # each step bracketed by events on the stream (no host sync between
    # steps); the headline is the median step, the wall clock is kept beside it
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for e0, e1 in evs:
        e0.record()
        step()
        e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    step_ms = sorted(e0.elapsed_time(e1) for e0, e1 in evs)
    ms_step = float(np.median(step_ms))
    ms_step_wall = 1e3 * wall / args.steps

    # one layer alone (a fresh prompt's layer 0), host-synchronised: latency
    single = []
    for _ in range(20):
        ctx.bacon_begin_prompt(batch)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        ctx.bacon_compress_layer(0, batch, qs[0], ks[0], vs[0], out=outs[0])
        torch.cuda.synchronize()
        single.append(time.perf_counter() - t1)
    single_us = 1e6 * float(np.median(single))

    # Same region again with HIP events around every launch (on the pass's stream).
    ctx.bacon_profile_enable(True)
    torch.cuda.synchronize()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    kt = ctx.bacon_profile_read()
    ctx.bacon_profile_enable(False)
    per_kernel = {k: {"launches": n, "avg_us": 1e3 * ms / n, "algorithmic_bytes": kernel_bytes(k, wl),
                      "design_bytes": design_bytes(k, wl)} for k, (n, ms) in kt.items()}
    dom = max((k for k in per_kernel if kernel_bytes(k, wl) > 0),
              key=lambda k: per_kernel[k]["avg_us"])
    kbytes = kernel_bytes(dom, wl)
    achieved = kbytes / (per_kernel[dom]["avg_us"] * 1e-6) / 1e9
    traffic = measured_traffic(dom)
    for k in per_kernel:
        per_kernel[k]["measured_traffic"] = measured_traffic(k)

    # The per-layer calls over the same prompt (no next-layer pass in the
    # scoring launch), for comparison.
    for _ in range(args.warmup):
        step_layers()
    ms_step_layers = median_step_ms(step_layers, args.steps)

    # The same pass with the window-row normalisers supplied, as a prefill
    # attention that returns its softmax normalisers would (the first K pass and
    # the merge are skipped); reported beside the headline, never as it.
    lses = []
    for l in range(wl.num_layers):
        _, _, lse = ctx.bacon_score(l, batch, qs[l], ks[l], want_lse=True)
        lses.append(lse)
    torch.cuda.synchronize()

    def step_lse():
        ctx.bacon_begin_prompt(batch)
        ctx.bacon_compress_prompt(0, batch, qs, ks, vs, lses=lses, outs=outs)

    for _ in range(args.warmup):
        step_lse()
    ms_step_lse = median_step_ms(step_lse, args.steps)

    ab = algorithmic_bytes(wl)
    ms_layer = ms_step / wl.num_layers
    keys_step = wl.total_tokens * wl.num_kv_heads * wl.num_layers
    pass_gbs = ab["layer_mean"] / (ms_layer * 1e-3) / 1e9

    result = {
        "metric": METRIC,
        "value": keys_step / (ms_step * 1e-3),
        "unit": "keys/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "ms_per_layer": ms_layer,
        "ms_per_step_wall_mean": ms_step_wall,
        "timing": f"median of {args.steps} prompt steps, each bracketed by HIP events on the "
                  f"pass's stream (one stream)",
        "qk_scores_per_s": wl.num_q_heads * wl.window * wl.total_tokens * wl.num_layers
                           / (ms_step * 1e-3),
        "single_layer_us": single_us,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic: seeded N(0,1) Q/K/V, frame-periodic low-rank K component, "
                "planted query-aligned evidence keys (no checkpoint or dataset)",
        "config": {"workload": f"{wl.name}: {wl.num_layers} layers, {wl.num_q_heads}/"
                               f"{wl.num_kv_heads} heads, d={wl.head_dim}, N="
                               f"{wl.seq_lens[0] if wl.batch == 1 else list(wl.seq_lens)}, "
                               f"W={wl.window}, pool {wl.pool_kernel}, budget "
                               f"{list(set(wl.budgets))}",
                   "batch": wl.batch, "tokens": wl.total_tokens, "layers": wl.num_layers},
        "pass_hbm": {"bytes_per_layer": ab["layer_mean"], "achieved_GBs": pass_gbs,
                     "frac_of_peak": pass_gbs / HBM_PEAK_GBS},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": traffic, "kernel": dom,
                     "bytes_per_launch": kbytes,
                     "bytes_note": "algorithmic bytes of the work the launch completes: one "
                                   "layer's K read once, Q_win and E written",
                     "design_bytes_per_launch": design_bytes(dom, wl),
                     "traffic_over_algorithmic": None if traffic is None else traffic / kbytes,
                     "avg_us": per_kernel[dom]["avg_us"]},
        "kernels": per_kernel,
        "per_layer_calls": {
            "note": "bacon_compress_layer called for each layer (pass 1 of a layer in its own "
                    "launch)",
            "ms_per_layer": ms_step_layers / wl.num_layers,
            "value": keys_step / (ms_step_layers * 1e-3), "unit": "keys/s"},
        "supplied_lse": {
            "note": "window-row softmax normalisers given by the prefill attention "
                    "(bacon_compress_prompt with lse); the first K pass and the merge are "
                    "skipped",
            "ms_per_layer": ms_step_lse / wl.num_layers,
            "value": keys_step / (ms_step_lse * 1e-3), "unit": "keys/s"},
    }
    if not args.no_configs:
        del qs, ks, vs, outs, lses
        torch.cuda.empty_cache()
        configs = []
        for i in range(5):
            if i == args.workload:
                configs.append({"workload": wl.name, "layers": wl.num_layers,
                                "us_per_layer": 1e3 * ms_layer,
                                "keys_per_s": wl.total_tokens * wl.num_kv_heads / (ms_layer * 1e-3),
                                "bytes_per_layer": ab["layer_mean"],
                                "hbm_frac": pass_gbs / HBM_PEAK_GBS, "steps": args.steps})
                continue
            log(f"workload {i}: prompt call")
            configs.append(prompt_rate(i, min(args.steps, 20), 2))
        result["configs"] = configs
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle)")
        result["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds, gpu_idx)
    print(json.dumps(result))


if __name__ == "__main__":
    main()
