#!/usr/bin/env python3
"""Throughput of the ECOKV prefill eviction pass on one MI355X.

Workload: a 28-layer stack shaped like a 7B multimodal LLM (28 query / 4 KV
heads, head_dim 128, bf16) at N = 32768 tokens per layer, window w = 4, a
per-head budget of 20 % (10 % and 40 % reported alongside, under
other_budgets), synthetic keys
with 75 % near-duplicate "visual" tokens.  One step = score -> select ->
compact over all 28 layers (three library calls, inputs resident in HBM).

Prints one JSON line: tokens scored+evicted per second per layer, the
roofline of the dominant kernel (live HIP-event timing) and the CPU oracle
timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, vendor figure


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--budget-frac", type=float, default=0.2)
    ap.add_argument("--tokens", type=int, default=32768)
    ap.add_argument("--layers", type=int, default=28)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-layers", type=int, default=28)
    ap.add_argument("--config", choices=sorted(CONFIGS),
                    help="time only this configuration's pass (one JSON line; with --counter-run: its counter "
                         "workload) -- for profiling one configuration at a time")
    ap.add_argument("--prefill", action="store_true",
                    help="with --config stack28: the prefill's cache write (ecokv_prefill_write) from token-major "
                         "rows, then the pass with the handed-over sums (score_pre, select, compact)")
    ap.add_argument("--counter-run", action="store_true",
                    help="run a few passes and a 1 GiB copy for rocprofv3 --pmc, then exit")
    ap.add_argument("--traffic-summary", nargs=3, metavar=("FETCH_DIR", "WRITE_DIR", "COMMAND"),
                    help="turn two rocprofv3 --pmc outputs (FETCH_SIZE, WRITE_SIZE) of --counter-run into "
                         "the traffic summary text (CPU only)")
    return ap.parse_args()


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


# Stage names the library times (ECOKV_STAGE_TIMING=1) and the kernels behind them.
STAGE_KERNELS = {
    "sweep1_stream": ["k_fs1s"], "sweep1_block": ["k_fs1", "k_pass1"], "reduce1": ["k_reduce1"],
    "sweep2_stream": ["k_fs2s"], "sweep2_block": ["k_fs2", "k_pass2"], "epilogue": ["k_epi_unit"],
    "epilogue1": ["k_epi1"], "epilogue2": ["k_epi2"],
    "select": ["k_select_reg", "k_select", "k_sel_digit", "k_sel_count", "k_sel_emit"], "compact": ["k_compact"], "vnorm": ["k_vnorm"],
    "dquant": ["k_dquant", "k_dquant_reg"], "decode": ["k_decode_mx", "k_decode"], "decode_merge": ["k_decode_merge"],
    "prefill_sweep": [], "prefill_reduce": [], "prefill_copy": [],
}
BF16_MFMA_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix peak, vendor figure
COPY_BYTES = 1 << 30  # size of the calibration copy in --counter-run
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic_stack28.txt")


def stage_of_kernel(kname):
    import re
    m = re.search(r"::(k_\w+?)(<|\()", kname)
    if not m:
        return None
    # the prefill cache write's forms of sweep 1 and its reduction, and its copies
    if m.group(1) in ("k_fs1s", "k_reduce1") and ", true>" in kname:
        return "prefill_sweep" if m.group(1) == "k_fs1s" else "prefill_reduce"
    if m.group(1) == "k_rows_copy":
        return "prefill_copy"
    for st, ks in STAGE_KERNELS.items():
        if m.group(1) in ks:
            return st
    return None


def source_digest():
    """sha256 over the kernel sources (csrc); stored traffic figures are valid only for this digest."""
    import hashlib
    h = hashlib.sha256()
    d = os.path.join(ROOT, "paper_2609_06663_amd", "csrc")
    for f in sorted(os.listdir(d)):
        if f.endswith((".hip", ".h")):
            h.update(f.encode())
            with open(os.path.join(d, f), "rb") as fh:
                h.update(fh.read())
    return h.hexdigest()[:16]


def stored_traffic(stage):
    """HBM bytes per launch of `stage` from the committed counter summary, or None if the
    summary is missing or the sources changed since the counters were taken."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    digest, val = None, None
    with open(TRAFFIC_FILE) as fh:
        for line in fh:
            parts = line.split()
            if len(parts) >= 2 and parts[0] == "source_digest:":
                digest = parts[1]
            if len(parts) >= 6 and parts[0] == "stage:" and parts[1] == stage:
                val = float(parts[5])
    if digest != source_digest():
        return None
    return val


# The configurations of the benchmark: workload builder, selection mode, label.
CONFIGS = {
    "stack28": ("stack28", "per_head", "28-layer GQA stack (28q/4kv, head_dim 128, bf16), N=32768, window 4, "
                                       "budget 20 % per head"),
    "layer7b": ("layer7b", "per_head", "one 7B-MLLM layer (28q/4kv, head_dim 128, bf16), N=8192, window 8, "
                                       "budget 20 % per head"),
    "mha64k": ("mha64k", "per_head", "one 32-head MHA layer (head_dim 128, bf16), N=65536, window 8, "
                                     "budget 2048 per head"),
    "varlen": ("varlen", "layer_flat", "one layer over 8 packed sequences of 4k-32k tokens (28q/4kv, head_dim "
                                       "128, bf16), window 4, layer-flat budget 15 % of each sequence"),
}


def timed(fn, reps, stream):
    """Average milliseconds of fn() over reps calls, bracketed by events on `stream`."""
    import torch
    fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def stage_us(fn, reps):
    """Microseconds per call of fn() in every library stage (all its launches in
    the call together; "launches" gives how many per call)."""
    import torch
    import paper_2609_06663_amd as P
    os.environ["ECOKV_STAGE_TIMING"] = "1"
    P.ecokv_stage_times()
    for _ in range(reps):
        fn()
    torch.cuda.synchronize()
    st = P.ecokv_stage_times()
    os.environ["ECOKV_STAGE_TIMING"] = "0"
    out = {k: round(v[0] / reps * 1e3, 2) for k, v in st.items()}
    for k, v in st.items():
        if v[1] != reps:
            out[f"{k}_launches"] = round(v[1] / reps, 2)
    return out


def pass_leg(name, steps, to_dev, wl=None):
    """One configuration's pass (score, select, compact): per-pass time, per-kernel
    times, algorithmic bytes and the fraction of the HBM peak."""
    import torch
    import workloads as W
    import paper_2609_06663_amd as P
    from paper_2609_06663_amd.pipeline import EvictionPass
    builder, mode, label = CONFIGS[name]
    if wl is None:
        t0 = time.time()
        wl = W.CONFIG_BUILDERS[builder]()
        log(f"{name}: generated in {time.time() - t0:.1f}s")
    Kx, Vx, Qx = to_dev(wl.K), to_dev(wl.V), to_dev(wl.Q)
    sh = P.Shape(wl.L, wl.Hq, wl.Hkv, wl.D, wl.w, wl.cu_seqlens)
    epx = EvictionPass(sh, wl.budget, P.LAYER_FLAT if mode == "layer_flat" else P.PER_HEAD, P.Params(),
                       torch.bfloat16, "cuda")
    stream = torch.cuda.current_stream()
    for _ in range(3):
        epx.run(Kx, Vx, Qx)
    ms = timed(lambda: epx.run(Kx, Vx, Qx), steps, stream)
    kern = stage_us(lambda: epx.run(Kx, Vx, Qx), steps)
    epx.check()
    tot, B = wl.cu_seqlens[-1], len(wl.cu_seqlens) - 1
    nbytes = (wl.L * wl.Hkv * tot * wl.D * 2 + wl.L * wl.Hq * B * wl.w * wl.D * 2
              + 4 * epx.n_idx * wl.D * 2 + 4 * epx.n_idx)
    out = {"workload": label, "layers": wl.L, "q_heads": wl.Hq, "kv_heads": wl.Hkv, "sequences": B,
           "tokens": tot, "entries": epx.n_idx, "ms_per_pass": round(ms, 4),
           "tokens_per_s_per_layer": round(tot / (ms / 1e3 / wl.L), 1),
           "algorithmic_bytes": nbytes, "achieved_GBs": round(nbytes / (ms / 1e3) / 1e9, 1),
           "frac_of_hbm_peak": round(nbytes / (ms / 1e3) / 1e9 / HBM_PEAK_GBS, 4), "kernels_us": kern}
    # the same pass when the prefill's cache write (ecokv_prefill_write) has
    # handed over the first sweep's sums: K read once
    pre, producer = prefill_inputs(epx, Kx, Vx, Qx)
    ms_pre = timed(lambda: epx.run(Kx, Vx, Qx, pre=pre), steps, stream)
    ms_prod = timed(producer, steps, stream)
    epx.check()
    out["with_prefill_sums"] = {"ms_per_pass": round(ms_pre, 4), "frac_of_hbm_peak":
                                round(nbytes / (ms_pre / 1e3) / 1e9 / HBM_PEAK_GBS, 4),
                                "producer_ms": round(ms_prod, 4)}
    del epx, Kx, Vx, Qx, pre, producer
    torch.cuda.empty_cache()
    return out


def main():
    args = parse()
    if args.traffic_summary:
        label = CONFIGS[args.config or "stack28"][2]
        if args.prefill:
            label += "; the prefill's cache write from token-major rows (ecokv_prefill_write), then the pass " \
                     "with its sums (ecokv_score_pre, select, compact)"
        traffic_summary(*args.traffic_summary, label=label)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the eviction pass is per (layer, KV head) and this "
              "build has no multi-GPU path; run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import workloads as W
    import paper_2609_06663_amd as P
    from paper_2609_06663_amd.pipeline import EvictionPass, LayerwiseEviction

    dev = torch.device("cuda:0")

    def to_dev(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)

    if args.config and args.config != "stack28":
        if args.counter_run:
            wl_c = W.CONFIG_BUILDERS[CONFIGS[args.config][0]]()
            sh = P.Shape(wl_c.L, wl_c.Hq, wl_c.Hkv, wl_c.D, wl_c.w, wl_c.cu_seqlens)
            mode_c = P.LAYER_FLAT if CONFIGS[args.config][1] == "layer_flat" else P.PER_HEAD
            ep_c = EvictionPass(sh, wl_c.budget, mode_c, P.Params(), torch.bfloat16, "cuda")
            counter_run(ep_c, to_dev(wl_c.K), to_dev(wl_c.V), to_dev(wl_c.Q))
            return
        print(json.dumps({"config": args.config, **pass_leg(args.config, args.steps, to_dev)}), flush=True)
        return

    T, L = args.tokens, args.layers
    log(f"generating stack: {L} layers x 4 KV heads x {T} tokens (bf16)")
    t0 = time.time()
    wl = W.stack28(T=T, budget_frac=args.budget_frac, L=L)
    log(f"generated in {time.time() - t0:.1f}s")

    K, V, Q = to_dev(wl.K), to_dev(wl.V), to_dev(wl.Q)
    shape = P.Shape(wl.L, wl.Hq, wl.Hkv, wl.D, wl.w, wl.cu_seqlens)
    b = wl.budget[0]
    ep = EvictionPass(shape, [b], P.PER_HEAD, P.Params(), torch.bfloat16, "cuda")
    stream = torch.cuda.current_stream()

    if args.counter_run:
        counter_run(ep, K, V, Q, prefill=args.prefill)
        return

    log(f"warmup {args.warmup}")
    for _ in range(args.warmup):
        ep.run(K, V, Q)
    torch.cuda.synchronize()

    if args.config == "stack28":
        if args.prefill:
            pre, producer = prefill_inputs(ep, K, V, Q)
            ms_prod = timed(producer, args.steps, stream)
            ms = timed(lambda: ep.run(K, V, Q, pre=pre), args.steps, stream)
            kern = stage_us(lambda: (producer(), ep.run(K, V, Q, pre=pre)), args.steps)
            print(json.dumps({"config": "stack28", "prefill": True, "producer_ms": round(ms_prod, 4),
                              "ms_per_pass": round(ms, 4), "kernels_us": kern}), flush=True)
            return
        print(json.dumps({"config": "stack28", **pass_leg("stack28", args.steps, to_dev, wl=wl)}), flush=True)
        return

    log(f"timing {args.steps} steps")
    # an event between consecutive steps as well, for the median step time
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    evs[0].record(stream)
    for i in range(args.steps):
        ep.run(K, V, Q)
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    ms_per_step = evs[0].elapsed_time(evs[-1]) / args.steps
    step_ms = sorted(evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps))
    median_ms = step_ms[len(step_ms) // 2] if len(step_ms) % 2 else 0.5 * (step_ms[len(step_ms) // 2 - 1] +
                                                                           step_ms[len(step_ms) // 2])
    t_layer_s = ms_per_step / 1e3 / L
    value = T / t_layer_s

    # Per-call timing over the same stream (each call bracketed by events).
    log("per-call timing")
    calls = {"score": lambda: ep.score(K, Q), "select": lambda: ep.select(), "compact": lambda: ep.compact(K, V)}
    per_call_ms = {}
    for name, fn in calls.items():
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        fn()
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(args.steps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        per_call_ms[name] = e0.elapsed_time(e1) / args.steps

    # Per-kernel durations: a second timed region with the library's own HIP events
    # around every launch, recorded on the stream the kernel runs on.
    log("per-kernel timing")
    os.environ["ECOKV_STAGE_TIMING"] = "1"
    P.ecokv_stage_times()  # drop anything recorded before
    for _ in range(args.steps):
        ep.run(K, V, Q)
    torch.cuda.synchronize()
    stages = P.ecokv_stage_times()
    os.environ["ECOKV_STAGE_TIMING"] = "0"

    e = 2
    Hkv, Hq, D, w = wl.Hkv, wl.Hq, wl.D, wl.w
    n_idx = ep.n_idx
    P_ = T - w
    bytes_k = L * Hkv * T * D * e
    bytes_q = L * Hq * w * D * e
    bytes_scores = L * Hkv * P_ * 4
    bytes_gather = 4 * n_idx * D * e
    bytes_idx = 4 * n_idx
    algo = {
        # what each call must move at minimum
        "score": bytes_k + bytes_q + bytes_scores,
        "select": bytes_scores + bytes_idx,
        "compact": bytes_gather + bytes_idx,
    }
    # what each kernel must move at minimum (scratch between kernels is not counted)
    stage_algo = {
        "sweep1_stream": bytes_k + bytes_q, "sweep1_block": bytes_k + bytes_q,
        "sweep2_stream": bytes_k + bytes_q, "sweep2_block": bytes_k + bytes_q,
        "reduce1": 0, "epilogue": bytes_scores,
        "epilogue1": 0, "epilogue2": bytes_scores, "select": bytes_scores + bytes_idx,
        "compact": bytes_gather + bytes_idx,
    }
    # window logits q.k for every (window row, key): the contraction the sweeps run on the matrix cores
    window_flops = 2 * L * Hq * w * T * D
    pass_bytes = bytes_k + bytes_q + bytes_gather + bytes_idx  # per-layer formula x L
    kernels = {}
    for name, (ms, n) in stages.items():
        avg_s = ms / n / 1e3
        ab = stage_algo.get(name, 0)
        kernels[name] = {"avg_us": round(avg_s * 1e6, 2), "launches": n, "algorithmic_bytes": ab,
                         "GBs": round(ab / avg_s / 1e9, 1) if ab else None}
    dom = max(kernels, key=lambda k: kernels[k]["avg_us"])
    dom_s = kernels[dom]["avg_us"] / 1e6
    dom_gbs = stage_algo[dom] / dom_s / 1e9
    traffic = stored_traffic(dom)
    roofline = {
        "bound": "hbm",
        "kernel": dom,
        "achieved": round(dom_gbs, 1),
        "peak": HBM_PEAK_GBS,
        "unit": "GB/s",
        "frac": round(dom_gbs / HBM_PEAK_GBS, 4),
        "traffic": None if traffic is None else int(traffic),
        "algorithmic_bytes": stage_algo[dom],
        "avg_launch_us": kernels[dom]["avg_us"],
    }
    pass_gbs = pass_bytes / (ms_per_step / 1e3) / 1e9
    mfma = {}
    for name in ("sweep1_stream", "sweep2_stream"):
        if name in kernels:
            tf = window_flops / (kernels[name]["avg_us"] / 1e6) / 1e12
            mfma[name] = {"window_flops": window_flops, "achieved_tflops": round(tf, 1),
                          "peak_tflops": BF16_MFMA_PEAK_TFLOPS, "frac": round(tf / BF16_MFMA_PEAK_TFLOPS, 4)}

    # Budgets per (layer, KV head): the PyramidKV layer schedule (beta 20) with
    # the same tokens per head over the stack, select + compact on the scores
    # of the pass above (outputs fit the uniform-budget buffers: same total).
    log("per-(layer, head) budgets: PyramidKV schedule")
    per_layer = P.ecokv_pyramid_budgets(L, L * b, 20.0, w)
    hbud = [bl for bl in per_layer for _ in range(Hkv)]
    n_h = P.ecokv_index_count_mode(shape, P.HEAD_BUDGETS, hbud)
    assert n_h <= ep.n_idx
    ws_h = torch.zeros(P.ecokv_select_workspace_size(shape, P.HEAD_BUDGETS), dtype=torch.uint8, device=dev)
    h_calls = {
        "select": lambda: P.ecokv_select(ep.scores, shape, P.HEAD_BUDGETS, hbud, ep.idx, ep.counts, ep.offsets,
                                         ws_h),
        "compact": lambda: P.ecokv_compact(K, V, shape, P.HEAD_BUDGETS, hbud, ep.idx, None, None, ep.Kc, ep.Vc),
    }
    head_budgets = {"schedule": "PyramidKV, beta 20", "budget_first_layer": per_layer[0],
                    "budget_last_layer": per_layer[-1], "entries": n_h}
    for name, fn in h_calls.items():
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(args.steps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        head_budgets[f"{name}_ms"] = round(e0.elapsed_time(e1) / args.steps, 4)
    h_gather = 4 * n_h * D * e + 4 * n_h
    head_budgets["compact_algorithmic_bytes"] = h_gather
    head_budgets["compact_GBs"] = round(h_gather / (head_budgets["compact_ms"] / 1e3) / 1e9, 1)

    # Value-norm importance (S_imp = pooled attention x |v_i|_2): the score
    # call with V, on the same stack; one extra pass reads V.
    log("value-norm importance")
    pv = P.Params(imp_mode=P.IMP_ATTN_VNORM)
    ws_v = torch.empty(P.ecokv_workspace_size(shape, pv), dtype=torch.uint8, device=dev)

    def score_v():
        P.ecokv_score_v(K, V, Q, shape, pv, ep.scores, ep.lambda_, ep.stats, ws_v)

    score_v()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        score_v()
    e1.record(stream)
    torch.cuda.synchronize()
    os.environ["ECOKV_STAGE_TIMING"] = "1"
    P.ecokv_stage_times()
    for _ in range(args.steps):
        score_v()
    torch.cuda.synchronize()
    vstages = P.ecokv_stage_times()
    os.environ["ECOKV_STAGE_TIMING"] = "0"
    del ws_v
    bytes_v = L * Hkv * P_ * D * e  # the non-window value rows
    vn_s = vstages["vnorm"][0] / vstages["vnorm"][1] / 1e3
    value_norm = {"score_ms": round(e0.elapsed_time(e1) / args.steps, 4),
                  "score_ms_attention_only": round(per_call_ms["score"], 4),
                  "vnorm_kernel_us": round(vn_s * 1e6, 2),
                  "vnorm_algorithmic_bytes": bytes_v + 2 * bytes_scores,
                  "vnorm_GBs": round((bytes_v + 2 * bytes_scores) / vn_s / 1e9, 1)}

    # Alternatives of Sec. 6.3 / Appendix D / Appendix B.6: the score call with
    # each option, and the quantile kernel of the winsorised / MAD forms.
    log("normalisation / redundancy / centroid alternatives")
    alternatives = {"score_ms_default": round(per_call_ms["score"], 4)}
    alt_opts = {
        "winsorised_1pct": P.Params(norm_mode=P.NORM_WINSOR, winsor_q=0.01),
        "mad": P.Params(norm_mode=P.NORM_MAD),
        "r_std": P.Params(redundancy=P.RED_STD),
        "prefix_centroid": P.Params(centroid_scope=P.CENTROID_PREFIX),
    }
    for name, pa in alt_opts.items():
        ws_a = torch.empty(P.ecokv_workspace_size(shape, pa), dtype=torch.uint8, device=dev)

        def score_a():
            P.ecokv_score(K, Q, shape, pa, ep.scores, ep.lambda_, ep.stats, ws_a)

        score_a()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(args.steps):
            score_a()
        e1.record(stream)
        torch.cuda.synchronize()
        alternatives[f"score_ms_{name}"] = round(e0.elapsed_time(e1) / args.steps, 4)
        if name == "mad":
            os.environ["ECOKV_STAGE_TIMING"] = "1"
            P.ecokv_stage_times()
            for _ in range(args.steps):
                score_a()
            torch.cuda.synchronize()
            st_a = P.ecokv_stage_times()
            os.environ["ECOKV_STAGE_TIMING"] = "0"
            alternatives["dquant_mad_us"] = round(st_a["dquant"][0] / st_a["dquant"][1] * 1e3, 2)
        del ws_a

    # The pass with the first sweep's results handed over by the prefill's
    # KV-cache write (ecokv_prefill_write): the new K and V rows arrive
    # token-major, as a projection writes them, and the producer moves them
    # into the head-major cache while it accumulates the key sums and the
    # window rows' softmax statistics; the pass then reads K once.  The
    # producer's cost beyond a plain cache write is measured against the
    # library's own copy of V in the same call (the same rows moved the same
    # way, without the sweep) and against torch's transposing copy.
    log("prefill cache write with the first sweep, then the pass reading K once")
    G_, R_ = Hq // Hkv, (Hq // Hkv) * w
    U_ = L * Hkv
    Kn = K.transpose(1, 2).contiguous()  # [L][T][Hkv][D]
    Vn = V.transpose(1, 2).contiguous()
    Kc_, Vc_ = torch.empty_like(K), torch.empty_like(V)
    pre = torch.empty(U_ * (2 * D + 2 * R_), dtype=torch.float32, device=dev)
    ws_p = torch.empty(P.ecokv_prefill_workspace_size(shape), dtype=torch.uint8, device=dev)

    def producer():
        P.ecokv_prefill_write(Kn, Vn, Q, shape, P.Params(), Kc_, Vc_, pre, ws_p)

    def plain_write():
        Kc_.view(L, Hkv, T, D).copy_(Kn.view(L, T, Hkv, D).transpose(1, 2))
        Vc_.view(L, Hkv, T, D).copy_(Vn.view(L, T, Hkv, D).transpose(1, 2))

    ms_plain = timed(plain_write, args.steps, stream)
    ms_prod = timed(producer, args.steps, stream)
    assert torch.equal(Kc_, K) and torch.equal(Vc_, V), "the producer's cache differs from the rows it was given"
    os.environ["ECOKV_STAGE_TIMING"] = "1"
    P.ecokv_stage_times()
    for _ in range(args.steps):
        producer()
    torch.cuda.synchronize()
    pstages = P.ecokv_stage_times()
    os.environ["ECOKV_STAGE_TIMING"] = "0"
    p_us = {k: round(v[0] / v[1] * 1e3, 2) for k, v in pstages.items()}
    ms_pre = timed(lambda: ep.run(Kc_, Vc_, Q, pre=pre), args.steps, stream)
    ms_pre_score = timed(lambda: ep.score(Kc_, Q, pre=pre), args.steps, stream)
    # the sweep's cost beyond moving the same rows: the K sweep-with-copy minus
    # the plain copy of V (same bytes, same layout move), plus the reduction
    extra_us = p_us.get("prefill_sweep", 0.0) + p_us.get("prefill_reduce", 0.0) - p_us.get("prefill_copy_v", 0.0)
    kv_bytes = 2 * bytes_k
    with_pre = {"ms_per_step": round(ms_pre, 4), "score_ms": round(ms_pre_score, 4),
                "tokens_per_s_per_layer": round(T / (ms_pre / 1e3 / L), 1),
                "pass_frac_of_hbm_peak": round(pass_bytes / (ms_pre / 1e3) / 1e9 / HBM_PEAK_GBS, 4),
                "pre_from": "ecokv_prefill_write (timed below)",
                "producer": {"ms_per_call": round(ms_prod, 4), "kernels_us": p_us,
                             "algorithmic_bytes": 2 * kv_bytes + bytes_q,
                             "GBs": round((2 * kv_bytes + bytes_q) / (ms_prod / 1e3) / 1e9, 1),
                             "torch_transpose_copy_ms": round(ms_plain, 4),
                             "extra_over_plain_copy_us": round(extra_us, 2)},
                "producer_plus_pass_ms": round(ms_prod + ms_pre, 4),
                "plain_write_plus_two_sweep_pass_ms": round(ms_plain + ms_per_step, 4),
                "pass_frac_counting_producer_extra": round(
                    pass_bytes / ((ms_pre + max(extra_us, 0.0) / 1e3) / 1e3) / 1e9 / HBM_PEAK_GBS, 4)}
    del Kn, Vn, Kc_, Vc_, pre, ws_p
    torch.cuda.empty_cache()

    # Decode attention over the compressed cache the pass just wrote: one new
    # query per (layer, query head), all kept rows of its KV head.
    log("decode attention over the compressed cache")
    gq = torch.Generator(device="cpu").manual_seed(5)
    Qd = torch.randn((L, Hq, 1, D), generator=gq).to(torch.bfloat16).to(dev)
    Od = torch.empty((L, Hq, 1, D), dtype=torch.float32, device=dev)
    lsed = torch.empty((L, Hq, 1), dtype=torch.float32, device=dev)
    ws_d = torch.empty(max(P.ecokv_decode_workspace_size(shape, b), 256), dtype=torch.uint8, device=dev)

    def decode():
        P.ecokv_decode(Qd, ep.Kc, ep.Vc, shape, ep.counts, ep.offsets, b, Od, lsed, ws_d)

    decode()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        decode()
    e1.record(stream)
    torch.cuda.synchronize()
    os.environ["ECOKV_STAGE_TIMING"] = "1"
    P.ecokv_stage_times()
    for _ in range(args.steps):
        decode()
    torch.cuda.synchronize()
    dstages = P.ecokv_stage_times()
    os.environ["ECOKV_STAGE_TIMING"] = "0"
    dk_s = dstages["decode"][0] / dstages["decode"][1] / 1e3
    bytes_dec = 2 * n_idx * D * e + 2 * L * Hq * D * e  # Kc, Vc and the queries
    decode_att = {"call_ms": round(e0.elapsed_time(e1) / args.steps, 4),
                  "decode_kernel_us": round(dk_s * 1e6, 2),
                  "merge_kernel_us": round(dstages["decode_merge"][0] / dstages["decode_merge"][1] * 1e3, 2),
                  "algorithmic_bytes": bytes_dec,
                  "decode_GBs": round(bytes_dec / dk_s / 1e9, 1),
                  "frac_of_hbm_peak": round(bytes_dec / dk_s / 1e9 / HBM_PEAK_GBS, 4)}
    del ws_d

    # the stack's other two budgets (10 % and 40 % per head): the same pass, timed the same way
    log("10 % and 40 % budgets")
    other_budgets = {}
    for frac in (0.1, 0.4):
        bb = int(frac * T)
        ep2 = EvictionPass(shape, [bb], P.PER_HEAD, P.Params(), torch.bfloat16, "cuda")
        ep2.run(K, V, Q)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(args.steps):
            ep2.run(K, V, Q)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / args.steps
        pb = bytes_k + bytes_q + 4 * ep2.n_idx * D * e + 4 * ep2.n_idx
        other_budgets[f"budget_{int(frac * 100)}pct"] = {
            "budget_per_head": bb, "ms_per_step": round(ms, 4), "tokens_per_s_per_layer": T / (ms / 1e3 / L),
            "algorithmic_bytes": pb, "frac_of_hbm_peak": round(pb / (ms / 1e3) / 1e9 / HBM_PEAK_GBS, 4)}
        del ep2

    # the other configurations, each as its own pass: one 8192-token layer, one
    # 32-head 65536-token layer, and the head-adaptive batch (8 packed
    # sequences of 4k-32k tokens, layer-flat selection with H_kv floor(0.15 T_s)
    # places per sequence)
    log("one 8192-token layer")
    layer_8k = pass_leg("layer7b", args.steps, to_dev)
    log("one 32-head 65536-token layer")
    mha_64k = pass_leg("mha64k", args.steps, to_dev)
    log("layer-flat selection over 8 packed sequences")
    layer_flat_varlen = pass_leg("varlen", args.steps, to_dev)

    # the same stack as L single-layer calls on one stream (one call per layer
    # as its prefill finishes)
    log(f"{L} single-layer calls")
    shape1 = P.Shape(1, Hq, Hkv, D, w, wl.cu_seqlens)
    ep1 = EvictionPass(shape1, [b], P.PER_HEAD, P.Params(), torch.bfloat16, "cuda")
    Ks, Vs, Qs = [K[l:l + 1] for l in range(L)], [V[l:l + 1] for l in range(L)], [Q[l:l + 1] for l in range(L)]
    for l in range(L):
        ep1.run(Ks[l], Vs[l], Qs[l])
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        for l in range(L):
            ep1.run(Ks[l], Vs[l], Qs[l])
    e1.record(stream)
    torch.cuda.synchronize()
    ms1 = e0.elapsed_time(e1) / args.steps
    per_layer_calls = {"ms_per_step": round(ms1, 4), "us_per_layer": round(ms1 * 1e3 / L, 2),
                       "tokens_per_s_per_layer": round(T / (ms1 / 1e3 / L), 1)}
    # the same calls alternating over two streams (one workspace each): one
    # layer's latency-bound kernels overlap the next layer's sweeps
    log(f"{L} single-layer calls on two streams")
    lw = LayerwiseEviction(shape1, [b], L)

    def two_streams():
        lw.run_layers(range(L), Ks, Vs, Qs)
        lw.wait()

    for _ in range(3):
        two_streams()
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(args.steps):
        two_streams()
    e1.record(stream)
    torch.cuda.synchronize()
    ms2 = e0.elapsed_time(e1) / args.steps
    per_layer_calls["two_streams_ms_per_step"] = round(ms2, 4)
    per_layer_calls["two_streams_us_per_layer"] = round(ms2 * 1e3 / L, 2)
    del ep1, lw, Ks, Vs, Qs
    # a call per group of consecutive layers (as a prefill can issue every few
    # layers), alternating over two streams
    for k in (2, 4, 7):
        if L % k:
            continue
        log(f"{L // k} calls of {k} layers on two streams")
        shapek = P.Shape(k, Hq, Hkv, D, w, wl.cu_seqlens)
        lwk = LayerwiseEviction(shapek, [b], L)
        Kg = [K[c * k:(c + 1) * k] for c in range(L // k)]
        Vg = [V[c * k:(c + 1) * k] for c in range(L // k)]
        Qg = [Q[c * k:(c + 1) * k] for c in range(L // k)]

        def groups():
            lwk.run_layers(range(L // k), Kg, Vg, Qg)
            lwk.wait()

        msk = timed(groups, args.steps, stream)
        lwk.check()
        per_layer_calls[f"groups_of_{k}_two_streams_us_per_layer"] = round(msk * 1e3 / L, 2)
        del lwk, Kg, Vg, Qg

    # a plain device copy of 1 GiB (torch's copy kernel), for the bandwidth the
    # memory system gives an ordinary streaming kernel next to the 8 TB/s peak
    log("copy bandwidth")
    src = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device=dev).fill_(1.0)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(10):
        dst.copy_(src)
    e1.record(stream)
    torch.cuda.synchronize()
    copy_ms = e0.elapsed_time(e1) / 10
    copy_bw = {"bytes_per_copy": 2 * COPY_BYTES, "GBs": round(2 * COPY_BYTES / (copy_ms / 1e3) / 1e9, 1),
               "frac_of_hbm_peak": round(2 * COPY_BYTES / (copy_ms / 1e3) / 1e9 / HBM_PEAK_GBS, 4)}
    del src, dst

    cpu = cpu1 = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(wl, args.cpu_sample_layers)
        cpu1 = cpu_baseline_one_thread()

    out = {
        "metric": "tokens scored+evicted/sec per layer (all heads) at N=32k; % of HBM roofline",
        "value": round(value, 1),
        "unit": "tokens/s per layer",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": f"{L}-layer GQA stack (28q/4kv, head_dim 128, bf16), N={T} tokens per layer, "
                        f"window {w}, budget {b} tokens per head ({args.budget_frac:.0%}), per-head top-k",
            "layers": L, "q_heads": Hq, "kv_heads": Hkv, "head_dim": D, "tokens": T, "window": w,
            "budget_per_head": b, "layers_per_call": L,
        },
        "roofline": roofline,
        "cpu_baseline": cpu,
        "cpu_baseline_one_thread": cpu1,
        "median_ms_per_step": round(median_ms, 4),
        "pass": {"algorithmic_bytes": pass_bytes, "achieved_GBs": round(pass_gbs, 1),
                 "frac_of_hbm_peak": round(pass_gbs / HBM_PEAK_GBS, 4),
                 "t_layer_us": round(t_layer_s * 1e6, 3)},
        "per_layer_calls": per_layer_calls,
        "copy_bandwidth": copy_bw,
        "per_call_ms": {k: round(v, 4) for k, v in per_call_ms.items()},
        "per_call_algorithmic_bytes": algo,
        "kernels": kernels,
        "mfma_window_gemm": mfma,
        "head_budgets": head_budgets,
        "value_norm": value_norm,
        "alternatives": alternatives,
        "decode_attention": decode_att,
        "with_prefill_sums": with_pre,
        "layer_8k": layer_8k,
        "mha_64k": mha_64k,
        "layer_flat_varlen": layer_flat_varlen,
        "other_budgets": other_budgets,
    }
    print(json.dumps(out), flush=True)


def prefill_inputs(ep, K, V, Q):
    """Token-major copies of K and V, a cache to write, `pre`, and the producer call
    (ecokv_prefill_write) that fills the cache and `pre` from them."""
    import torch
    import paper_2609_06663_amd as P
    c = ep.shape.c
    L, Hkv, D, w, Hq = c.num_layers, c.num_kv_heads, c.head_dim, c.window, c.num_q_heads
    R = Hq // Hkv * w
    Kn = K.view(L, Hkv, -1, D).transpose(1, 2).contiguous()
    Vn = V.view(L, Hkv, -1, D).transpose(1, 2).contiguous()
    Kc, Vc = torch.empty_like(K), torch.empty_like(V)
    pre = torch.empty(L * Hkv * c.num_seqs * (2 * D + 2 * R), dtype=torch.float32, device=K.device)
    ws = torch.empty(P.ecokv_prefill_workspace_size(ep.shape), dtype=torch.uint8, device=K.device)

    def producer():
        P.ecokv_prefill_write(Kn, Vn, Q, ep.shape, P.Params(), Kc, Vc, pre, ws)

    producer()
    torch.cuda.synchronize()
    return pre, producer


def counter_run(ep, K, V, Q, prefill=False):
    """Workload for rocprofv3 --pmc: three passes (with prefill: three cache writes
    from token-major rows, then three passes with the handed-over sums), then three
    copies of COPY_BYTES."""
    import torch
    if prefill:
        pre, producer = prefill_inputs(ep, K, V, Q)
        for _ in range(3):
            producer()
        torch.cuda.synchronize()
        for _ in range(3):
            ep.run(K, V, Q, pre=pre)
        del producer
    else:
        for _ in range(3):
            ep.run(K, V, Q)
    torch.cuda.synchronize()
    src = torch.ones(COPY_BYTES // 2, dtype=torch.bfloat16, device=K.device)
    dst = torch.empty_like(src)
    for _ in range(3):
        torch.neg(src, out=dst)  # reads and writes COPY_BYTES each
    torch.cuda.synchronize()
    log("counter run done")


def _counter_rows(d):
    import csv
    import glob
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {d}")
    rows = []
    for f in files:
        with open(f, newline="") as fh:
            rows.extend(csv.DictReader(fh))
    return rows


def traffic_summary(fetch_dir, write_dir, command, label):
    """FETCH_SIZE and WRITE_SIZE (KiB per dispatch) per stage, scaled by the same counters
    on a plain copy of COPY_BYTES, into the text that stored_traffic() reads."""
    per = {}
    for ctr, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        copies = []
        for r in _counter_rows(d):
            if r.get("Counter_Name") != ctr:
                continue
            kname = r.get("Kernel_Name", "")
            val = float(r["Counter_Value"]) * 1024.0
            if "neg" in kname and "kernel" in kname:
                copies.append(val)
                continue
            st = stage_of_kernel(kname)
            if st:
                per.setdefault(st, {}).setdefault(ctr, {}).setdefault(kname, []).append(val)
        if not copies:
            raise SystemExit(f"{ctr}: copy kernel not found")
        per.setdefault("_copy", {})[ctr] = copies
    cf = COPY_BYTES / (sum(per["_copy"]["FETCH_SIZE"]) / len(per["_copy"]["FETCH_SIZE"]))
    cw = COPY_BYTES / (sum(per["_copy"]["WRITE_SIZE"]) / len(per["_copy"]["WRITE_SIZE"]))
    print(f"HBM traffic per launch from rocprofv3 counters: {label}")
    print(f"command: {command}")
    print("FETCH_SIZE and WRITE_SIZE are KiB per dispatch; each is scaled by copy_bytes / counter "
          f"on torch.neg over {COPY_BYTES} bytes (reads and writes that many bytes)")
    print(f"copy_factor_fetch: {cf:.4f}")
    print(f"copy_factor_write: {cw:.4f}")
    print(f"source_digest: {source_digest()}")
    print("# stage: name  fetch_bytes  write_bytes  =  scaled_total_bytes  (per call: each kernel's average "
          "over its dispatches, summed over the stage's kernels)")

    def per_call(d):
        return sum(sum(v) / len(v) for v in d.values())

    for st in STAGE_KERNELS:
        if st not in per or "FETCH_SIZE" not in per[st] or "WRITE_SIZE" not in per[st]:
            continue
        f = per_call(per[st]["FETCH_SIZE"]) * cf
        w = per_call(per[st]["WRITE_SIZE"]) * cw
        print(f"stage: {st} {f:.0f} {w:.0f} = {f + w:.0f}")


def cpu_baseline(wl, sample_layers):
    """The CPU oracle (score, select, compact) on the first layers of the same stack."""
    import numpy as np
    import oracle
    oracle.build(force=False)
    try:
        ncpu = len(os.sched_getaffinity(0))
    except AttributeError:
        ncpu = os.cpu_count() or 1
    # the host cores this process may use: its CPU affinity, or the thread
    # count the machine assigns it (OMP_NUM_THREADS) when that is smaller
    omp = int(os.environ.get("OMP_NUM_THREADS", "0") or 0)
    threads = max(1, min(ncpu, omp) if omp > 0 else ncpu)
    Ls = min(sample_layers, wl.L)
    K, V, Q = wl.K[:Ls], wl.V[:Ls], wl.Q[:Ls]
    log(f"cpu baseline: oracle on {Ls} layers x {wl.Hkv} heads with {threads} threads, repeated for >= 10 s")
    reps, dt = 0, 0.0
    while dt < 10.0 and reps < 64:
        t0 = time.perf_counter()
        S, _ = oracle.score(K, Q, Ls, wl.Hq, wl.Hkv, wl.cu_seqlens, wl.D, wl.w, nthreads=threads)
        idx, counts, offsets = oracle.select(S, Ls, wl.Hkv, wl.cu_seqlens, wl.w, wl.budget, oracle.PER_HEAD,
                                             nthreads=threads)
        oracle.compact(K, V, Ls, wl.Hkv, wl.cu_seqlens, wl.D, idx, counts, offsets)
        dt += time.perf_counter() - t0
        reps += 1
    T = wl.cu_seqlens[-1]
    used = min(threads, Ls * wl.Hkv)
    return {"value": round(T * reps / (dt / Ls), 1), "unit": "tokens/s per layer", "cores": used, "kind": "oracle",
            "sample": f"first {Ls} of {wl.L} layers ({Ls * wl.Hkv} (layer, head) units of {T} tokens), "
                      f"score+select+compact, fp64, {reps} repetitions, {dt:.2f}s wall",
            "host_cpus": {"affinity": ncpu, "os_cpu_count": os.cpu_count(), "OMP_NUM_THREADS": omp or None}}


def cpu_baseline_one_thread():
    """The CPU oracle on one thread, on one 8192-token layer of the same head shape (28q/4kv, D 128)."""
    import workloads as W
    import oracle
    wl = W.layer7b()
    T = wl.cu_seqlens[-1]
    log(f"cpu baseline: oracle on one {T}-token layer with 1 thread, repeated for >= 3 s")
    reps, dt = 0, 0.0
    while dt < 3.0 and reps < 64:
        t0 = time.perf_counter()
        S, _ = oracle.score(wl.K, wl.Q, wl.L, wl.Hq, wl.Hkv, wl.cu_seqlens, wl.D, wl.w, nthreads=1)
        idx, counts, offsets = oracle.select(S, wl.L, wl.Hkv, wl.cu_seqlens, wl.w, wl.budget, oracle.PER_HEAD,
                                             nthreads=1)
        oracle.compact(wl.K, wl.V, wl.L, wl.Hkv, wl.cu_seqlens, wl.D, idx, counts, offsets)
        dt += time.perf_counter() - t0
        reps += 1
    return {"value": round(T * reps / (dt / wl.L), 1), "unit": "tokens/s per layer", "cores": 1, "kind": "oracle",
            "sample": f"one layer of {wl.Hkv} KV heads x {T} tokens (28 query heads, window {wl.w}, budget "
                      f"{wl.budget[0]}), score+select+compact, fp64, {reps} repetitions, {dt:.2f}s wall"}


if __name__ == "__main__":
    main()
