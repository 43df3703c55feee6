#!/usr/bin/env python3
"""Benchmark the slot-scoring step of Zarya's slotted speculative decoding on one MI355X.

A step (Sec. 5.2 of the paper: draft phase, slot confidence, slot selection)
is, on one batch of synthetic input already resident in HBM:

  1. zarya_slot_attn        DIFFUSION pass (draft) over the prefix cache
  2. zarya_slot_confidence  LM-head confidence of every draft token
  3. zarya_select_slots     the workload's selection rule (below)

Headline workload (the JSON line's `value`): qwen4b -- the 4B-scale
long-context layer, B=8, Hq/Hkv=32/8, D=128, P=16384, S=8, L=16, H=2560,
V=151936, bf16; selection: threshold 0.9 on the first-token confidence
(Sec. 5.2, Sec. 6).  The same line carries the qwen0.6b (B=16, 16/8 heads,
P=2048, S=8, L=8, H=1024; threshold 0.9) and qwen1.7b (B=32, 16/8 heads,
P=4096, S=16, L=4, H=2048; top-4 slots by mean max-prob) steps under
`workloads`, each with its own rooflines.  Three copies of every input are
rotated so that neither the KV cache nor the LM head is served from the
256 MB Infinity Cache.

Every measurement first runs its own work back to back, untimed, for
--spin-up seconds (the GPU clock settles after idle gaps), then its warm-up
steps, then the timed steps.  Times come from HIP events recorded on the
stream the library launches on (torch's current stream); `roofline` is the dominant kernel's
(slot_confidence, against the bf16 MFMA peak) and `roofline_slot_attn` the
attention's, against both the HBM and the MFMA peak.  The float64 CPU oracle
is timed on the host cores as a reference baseline.
"""

from __future__ import annotations

import argparse
import hashlib
import itertools
import json
import os
import re
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0
PEAK_BF16_TFLOPS = 2500.0
METRIC = "slot-scoring steps/s, draft tokens/s; slot_attn HBM GB/s & conf MFMA % @1 MI355X"
HEADLINE = "qwen4b"
SUB_WORKLOADS = ["qwen0.6b", "qwen1.7b"]
# selection of each workload's step: (slot confidence rule, selection rule, threshold, k)
SELECTION = {
    "qwen0.6b": ("first_token", "threshold", 0.9, 1),
    "qwen1.7b": ("mean", "top_k", 0.9, 4),
    "qwen4b": ("first_token", "threshold", 0.9, 1),
}
# which peak bounds the attention of each workload (algorithmic flops / bytes against the ridge point)
ATTN_BOUND = {"qwen0.6b": "hbm", "qwen1.7b": "hbm", "qwen4b": "mfma"}
COUNTERS = os.path.join(ROOT, "profiles", "hbm_traffic_{}.md")
# Seconds of untimed back-to-back work before each measurement's warm-up steps
# (--spin-up).  After an idle gap (input generation, the CPU oracle) the GPU
# clock needs tens of milliseconds of load to settle: at qwen4b the first 10
# steps after 3 s idle averaged 1.46 ms, the next three blocks of 10
# 1.06 / 1.02 / 1.01 ms, and every later block 0.98-0.99 ms.
SPIN_UP_S = 0.25


def spin_up(fn, seconds):
    """Call fn() back to back until `seconds` of wall time have passed (the
    device is synchronised every 8 calls); returns the number of calls."""
    import torch

    n = 0
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(8):
            fn()
        n += 8
        torch.cuda.synchronize()
    return n


def quantile(sorted_vals, q):
    """Linear-interpolation quantile of an already sorted list."""
    x = q * (len(sorted_vals) - 1)
    i = int(x)
    j = min(i + 1, len(sorted_vals) - 1)
    return sorted_vals[i] + (sorted_vals[j] - sorted_vals[i]) * (x - i)


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


KERNEL_SOURCES = {
    "slot_confidence": ("slot_conf.hip", "common.hpp", "kernels.hpp"),
    "slot_attn": ("slot_attn.hip", "common.hpp", "kernels.hpp"),
}


def source_hash(op):
    """sha256 of the sources an op's kernels are built from (ties committed
    counter readings to the kernel version they were taken on)."""
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[op]:
        with open(os.path.join(ROOT, "paper_2609_19868_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(workload, op):
    """HBM bytes per launch of `op` from the committed rocprofv3 counter
    summary of `workload`, or None when absent or taken on other sources."""
    path = COUNTERS.format(workload)
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(rf"^source_sha256\[{re.escape(op)}\]:\s*(\S+)", text, re.M)
    t = re.search(rf"^traffic_bytes\[{re.escape(op)}\]:\s*([0-9.eE+]+)", text, re.M)
    if not m or not t or m.group(1) != source_hash(op):
        return None
    return float(t.group(1))


def cpu_baseline(wl, x, c, sel):
    """The float64 oracle as it stands, on this host's cores: the whole step
    (attention of every head, confidence of every row over the whole
    vocabulary, selection).  One run, or the median of three when one run
    takes under 8 s, so the leg stays within about 10-30 s."""
    import numpy as np
    from threadpoolctl import threadpool_info

    import oracle
    import workloads as W

    xf = {k: W.as_f64(v, wl.dtype) for k, v in x.items()}
    hf = W.as_f64(c["hidden"], wl.dtype)
    wf = W.as_f64(c["w_vocab"], wl.dtype)
    conf_rule = oracle.CONF_MEAN if sel[0] == "mean" else oracle.CONF_FIRST_TOKEN
    rule = oracle.SELECT_TOP_K if sel[1] == "top_k" else oracle.SELECT_THRESHOLD
    times = []
    while len(times) < (3 if not times or times[0] < 8.0 else 1):
        t0 = time.perf_counter()
        oracle.slot_attention(xf["q"], xf["k_cache"], xf["v_cache"], xf["k_slot"], xf["v_slot"], wl.prefix_len,
                              wl.n_slots, wl.slot_len, wl.scale, oracle.PASS_DIFFUSION)
        r = oracle.slot_confidence(hf, wf)
        oracle.select_slots(r["max_prob"].reshape(wl.batch, wl.n_slots, wl.slot_len).astype(np.float32), None,
                            conf_rule, rule, sel[2], sel[3])
        times.append(time.perf_counter() - t0)
        log(f"cpu oracle step {len(times) - 1}: {times[-1]:.2f} s")
    pools = threadpool_info()
    threads = max([d.get("num_threads", 1) for d in pools] + [1])
    blas = ",".join(sorted({d.get("internal_api", "?") for d in pools if d.get("user_api") == "blas"})) or "none"
    t = statistics.median(times)
    return {
        "value": 1.0 / t,
        "unit": "steps/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"the whole {wl.name} step once per run (attention of all {wl.batch}x{wl.n_q_heads} heads x "
                  f"{wl.T} tokens over P={wl.prefix_len}, confidence of all {wl.M} rows over {wl.vocab} ids, "
                  f"selection), float64 numpy, median of {len(times)} run(s); host has "
                  f"{len(os.sched_getaffinity(0))} usable cores, BLAS {blas} with {threads} threads",
        "seconds_per_step": t,
        "draft_tokens_per_s": wl.M / t,
    }


def attn_work(wl):
    """Algorithmic bytes and flops of one DIFFUSION-pass slot_attn launch."""
    B, Hq, Hkv, D, P, T, L = wl.batch, wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.prefix_len, wl.T, wl.slot_len
    nbytes = (2 * B * Hkv * P * D * 2  # prefix K and V, once per GQA group
              + 2 * B * Hq * T * D * 2  # Q in, O out
              + 2 * B * Hkv * T * D * 2  # the draft tokens' own K and V
              + B * Hq * T * 4)  # LSE
    flops = 4.0 * B * Hq * T * (P + L) * D  # QK^T and PV over the prefix and the row's own slot
    return nbytes, flops


def measure_workload(name, steps, warmup, extras, want_cpu, spin_s=SPIN_UP_S):
    """Time the scoring step of one workload; returns its record (and runs the
    extras that belong to it)."""
    import numpy as np
    import torch

    import paper_2609_19868_amd as Z
    import workloads as W
    from paper_2609_19868_amd import _lib

    dev = torch.device("cuda:0")
    wl = W.WORKLOADS[name]
    B, Hq, Hkv, D, P, S, L, H, V = (wl.batch, wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.prefix_len, wl.n_slots,
                                    wl.slot_len, wl.hidden, wl.vocab)
    T, M = wl.T, wl.M
    sel = SELECTION[name]
    conf_rule = Z.SLOT_CONF_MEAN if sel[0] == "mean" else Z.SLOT_CONF_FIRST_TOKEN
    rule = Z.SELECT_TOP_K if sel[1] == "top_k" else Z.SELECT_THRESHOLD

    log(f"generating {name} inputs")
    x = W.attention_inputs(wl)
    c = W.confidence_inputs(wl)

    def dev_bf16(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)

    base = {k: dev_bf16(v) for k, v in x.items()}
    base["hidden"] = dev_bf16(c["hidden"])
    base["w_vocab"] = dev_bf16(c["w_vocab"])
    n_sets = 3
    sets = [base] + [{k: v.clone() for k, v in base.items()} for _ in range(n_sets - 1)]

    out = torch.empty((B, Hq, T, D), dtype=torch.bfloat16, device=dev)
    lse = torch.empty((B, Hq, T), dtype=torch.float32, device=dev)
    desc = Z.slot_attn_desc(base["q"], base["k_cache"], base["k_slot"], S, L, Z.PASS_DIFFUSION)
    plan = _lib.slot_attn_plan(desc)
    attn_ws = torch.empty(max(1, _lib.slot_attn_workspace_size(desc)), dtype=torch.uint8, device=dev)
    conf_out = {
        "max_prob": torch.empty(M, dtype=torch.float32, device=dev),
        "argmax": torch.empty(M, dtype=torch.int32, device=dev),
        "lse": torch.empty(M, dtype=torch.float32, device=dev),
    }
    conf_ws = torch.empty(_lib.slot_confidence_workspace_size(_lib.ConfDesc(n_rows=M, hidden=H, vocab=V, dtype=1)),
                          dtype=torch.uint8, device=dev)
    sel_out = (torch.empty((B, S), dtype=torch.float32, device=dev), torch.empty((B, S), dtype=torch.int32, device=dev),
               torch.empty((B,), dtype=torch.int32, device=dev))

    def step(s, pass_, evs=None):
        if evs:
            evs[0].record()
        Z.slot_attn(s["q"], s["k_cache"], s["v_cache"], s["k_slot"], s["v_slot"], S, L, pass_=pass_, out=out, lse=lse,
                    workspace=attn_ws)
        if evs:
            evs[1].record()
        Z.slot_confidence(s["hidden"], s["w_vocab"], out=conf_out, workspace=conf_ws)
        if evs:
            evs[2].record()
        Z.select_slots(conf_out["max_prob"].view(B, S, L), None, conf_rule, rule, sel[2], sel[3], out=sel_out)
        if evs:
            evs[3].record()

    def timed(pass_, K, Wm):
        """K steps timed as a whole (no events between the kernels, which
        would add their own packets to the timed stream), then K more with
        events around each kernel for the per-kernel breakdown."""
        ctr = itertools.count()
        spin_up(lambda: step(sets[next(ctr) % n_sets], pass_), spin_s)
        for i in range(Wm):
            step(sets[i % n_sets], pass_)
        torch.cuda.synchronize()
        t_start, t_end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t_start.record()
        for i in range(K):
            step(sets[i % n_sets], pass_)
        t_end.record()
        torch.cuda.synchronize()
        total_ms = t_start.elapsed_time(t_end)
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(K)]
        for i in range(K):
            step(sets[i % n_sets], pass_, evs[i])
        torch.cuda.synchronize()
        per = [[e[j].elapsed_time(e[j + 1]) for j in range(3)] for e in evs]
        return total_ms / K, [statistics.mean(p[j] for p in per) for j in range(3)], \
            [statistics.median(p[j] for p in per) for j in range(3)], \
            [[quantile(sorted(p[j] for p in per), q) for q in (0.1, 0.9)] for j in range(3)]

    log(f"{name}: timing {steps} steps after {warmup} warm-up steps (DIFFUSION pass)")
    ms_step, mean_ms, med_ms, pct_ms = timed(Z.PASS_DIFFUSION, steps, warmup)
    attn_ms, conf_ms, sel_ms = mean_ms
    log(f"{name}: step {ms_step * 1e3:.1f} us: slot_attn {attn_ms * 1e3:.1f} us, slot_confidence "
        f"{conf_ms * 1e3:.1f} us, select_slots {sel_ms * 1e3:.1f} us")

    attn_bytes, attn_flops = attn_work(wl)
    conf_flops = 2.0 * M * V * H
    conf_tflops = conf_flops / (conf_ms * 1e-3) / 1e12
    attn_gbps = attn_bytes / (attn_ms * 1e-3) / 1e9
    attn_tflops = attn_flops / (attn_ms * 1e-3) / 1e12
    sel_desc = (f"top-{sel[3]} slots by mean max-prob" if sel[1] == "top_k"
                else f"threshold {sel[2]} on the {sel[0].replace('_', '-')} confidence")
    rec = {
        "workload": f"{name}: B={B} Hq/Hkv={Hq}/{Hkv} D={D} P={P} S={S} L={L} H={H} V={V}; step = slot_attn "
                    f"(DIFFUSION) + slot_confidence + select_slots ({sel_desc})",
        "steps_per_s": 1e3 / ms_step,
        "ms_per_step": ms_step,
        "draft_tokens_per_s": B * S * L * 1e3 / ms_step,
        "kernel_us": {"slot_attn": attn_ms * 1e3, "slot_confidence": conf_ms * 1e3, "select_slots": sel_ms * 1e3},
        "kernel_us_median": {"slot_attn": med_ms[0] * 1e3, "slot_confidence": med_ms[1] * 1e3,
                             "select_slots": med_ms[2] * 1e3},
        "kernel_us_p10_p90": {k: [pct_ms[j][0] * 1e3, pct_ms[j][1] * 1e3]
                              for j, k in enumerate(("slot_attn", "slot_confidence", "select_slots"))},
        "roofline": {
            "bound": "mfma",
            "kernel": "slot_confidence (GEMM + fused reduction; launch to launch on its stream)",
            "achieved": conf_tflops,
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": conf_tflops / PEAK_BF16_TFLOPS,
            "traffic": measured_traffic(name, "slot_confidence"),
            "algorithmic_flops_per_launch": conf_flops,
        },
        "roofline_slot_attn": {
            "bound": ATTN_BOUND[name],
            "hbm": {"achieved": attn_gbps, "peak": PEAK_HBM_GBPS, "unit": "GB/s", "frac": attn_gbps / PEAK_HBM_GBPS,
                    "algorithmic_bytes_per_launch": attn_bytes},
            "mfma": {"achieved": attn_tflops, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": attn_tflops / PEAK_BF16_TFLOPS, "algorithmic_flops_per_launch": attn_flops},
            "traffic": measured_traffic(name, "slot_attn"),
            "plan": plan,
        },
    }
    if "graph" in extras:
        log(f"{name}: timing the same step replayed from HIP graphs")
        rec["graph_step"] = graph_step(step, sets, steps, spin_s)
    if "ar_infill" in extras:
        log(f"{name}: timing the AR_INFILL (verification) pass")
        ms_ar, mean_ar, _, _ = timed(Z.PASS_AR_INFILL, max(10, steps // 2), 3)
        rec["ar_infill_pass"] = {"steps_per_s": 1e3 / ms_ar, "slot_attn_us": mean_ar[0] * 1e3}
    if "verification" in extras:
        log(f"{name}: timing the verification step")
        rec["verification_step"] = verification_step(dev, wl, sets[0], conf_out, sel_out, max(10, steps // 2), spin_s)
    if "sampled" in extras:
        log(f"{name}: timing the sampled LM-head reduction (Gumbel-max, T = 1)")
        rec["sampled_draft"] = sampled_draft(dev, wl, sets, max(10, steps // 2), conf_ms, spin_s)
    if "mode_a" in extras:
        log("timing a Mode A denoising step")
        rec["mode_a_step"] = mode_a_step(dev, sets[0]["w_vocab"], max(10, steps // 4), spin_s)
    del sets, base
    torch.cuda.empty_cache()
    if "single" in extras:
        log(f"{name}: timing the single-sequence step (batch 1)")
        rec["single_sequence_step"] = single_sequence_step(dev, wl, max(20, steps // 2), spin_s)
    if want_cpu:
        log(f"{name}: timing the float64 CPU oracle (reference baseline)")
        rec["cpu_baseline"] = cpu_baseline(wl, x, c, sel)
    return rec


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--spin-up", type=float, default=SPIN_UP_S,
                    help="seconds of untimed work before each measurement's warm-up steps (GPU clock settling)")
    ap.add_argument("--workload", default=HEADLINE, choices=["qwen0.6b", "qwen1.7b", "qwen4b"],
                    help="workload of the headline value")
    ap.add_argument("--only", action="store_true", help="time the headline workload only (no sub-workloads)")
    ap.add_argument("--no-cpu-baseline", action="store_true", help="skip the CPU oracle leg")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the graph, AR_INFILL, verification, sampling, Mode A, batch-1 and layout timings")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy (scale reference for HBM byte counters)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures the slot-scoring step on one GPU only; the multi-GPU sharding is designed "
              "but not built (run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch

    dev = torch.device("cuda:0")
    if args.copy_calibration:
        copy_calibration(dev, args.steps)
        return

    def extras_of(name):
        if args.no_extras:
            return set()
        if name == args.workload:
            return {"graph", "ar_infill", "sampled"}
        if name == "qwen0.6b":
            return {"verification", "sampled", "mode_a", "single"}
        return set()

    head = measure_workload(args.workload, args.steps, args.warmup, extras_of(args.workload),
                            not args.no_cpu_baseline, args.spin_up)
    subs = {}
    if not args.only:
        for name in SUB_WORKLOADS + [HEADLINE]:
            if name != args.workload and name not in subs:
                subs[name] = measure_workload(name, args.steps, args.warmup, extras_of(name), False, args.spin_up)

    result = {
        "metric": METRIC,
        "value": head["steps_per_s"],
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "clock_spin_up_s": args.spin_up,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) activations and KV cache, N(0,0.02^2) LM head, rounded to bf16)",
        "config": {
            "workload": head["workload"],
            "parallelism": "single GPU",
        },
        "draft_tokens_per_s": head["draft_tokens_per_s"],
        "roofline": head["roofline"],
        "roofline_slot_attn": head["roofline_slot_attn"],
    }
    if "cpu_baseline" in head:
        result["cpu_baseline"] = head.pop("cpu_baseline")
    for k in ("kernel_us", "kernel_us_median", "kernel_us_p10_p90", "graph_step", "ar_infill_pass",
              "sampled_draft"):
        if k in head:
            result[k] = head[k]
    if subs:
        result["workloads"] = subs
    if not args.no_extras:
        result["layout_attention"] = layout_attention(dev, max(5, args.steps // 10), args.spin_up)
    print(json.dumps(result), flush=True)


def graph_step(step, sets, K, spin_s):
    """The scoring step captured once per input copy in a HIP graph
    (torch.cuda.CUDAGraph over the library's launches) and replayed: the same
    kernels without the host-side launch path between them."""
    import torch

    import paper_2609_19868_amd as Z

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for s in sets:
            step(s, Z.PASS_DIFFUSION)
    torch.cuda.current_stream().wait_stream(side)
    graphs = []
    for s in sets:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step(s, Z.PASS_DIFFUSION)
        graphs.append(g)
    ctr = itertools.count()
    spin_up(lambda: graphs[next(ctr) % len(graphs)].replay(), spin_s)
    for g in graphs:
        g.replay()
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for i in range(K):
        graphs[i % len(graphs)].replay()
    t1.record()
    torch.cuda.synchronize()
    us = t0.elapsed_time(t1) / K * 1e3
    return {"step_us": us, "steps_per_s": 1e6 / us}


def verification_step(dev, wl, s, conf_out, sel_out, K, spin_s):
    """The step after scoring (Sec. 5.2 "Verification phase", "KV cache
    update"): AR_INFILL attention of the draft tokens, confidence of the draft
    ids (the scoring step's argmax) as targets, acceptance of the selected
    slots, and the append of the accepted tokens to a cache with room for them.
    The prefix lengths are reset between steps, outside the timed events."""
    import torch

    import paper_2609_19868_amd as Z

    B, Hq, Hkv, D, P, S, L = wl.batch, wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.prefix_len, wl.n_slots, wl.slot_len
    T = wl.T
    kc = torch.empty((B, Hkv, P + T, D), dtype=torch.bfloat16, device=dev)
    vc = torch.empty_like(kc)
    kc[:, :, :P].copy_(s["k_cache"][:, :, :P])
    vc[:, :, :P].copy_(s["v_cache"][:, :, :P])
    plens0 = torch.full((B,), P, dtype=torch.int32, device=dev)
    plens = plens0.clone()
    targets = conf_out["argmax"].clone()
    out = torch.empty((B, Hq, T, D), dtype=torch.bfloat16, device=dev)
    lse = torch.empty((B, Hq, T), dtype=torch.float32, device=dev)
    tout = {k: torch.empty_like(conf_out[k]) for k in ("max_prob", "argmax", "lse")}
    tout["target_prob"] = torch.empty_like(conf_out["max_prob"])
    acc_out = (torch.empty((B, S, L), dtype=torch.uint8, device=dev), torch.empty((B, S), dtype=torch.int32, device=dev),
               torch.empty((B,), dtype=torch.int32, device=dev))
    # random LM-head weights make every probability tiny: threshold 0 accepts every
    # token of the selected slots, which is the copy-heavy end of the append
    thr = 0.0
    selected = sel_out[1]

    def one(evs=None):
        if evs:
            evs[0].record()
        Z.slot_attn(s["q"], kc, vc, s["k_slot"], s["v_slot"], S, L, pass_=Z.PASS_AR_INFILL, prefix_len=P,
                    out=out, lse=lse, prefix_lens=plens)
        if evs:
            evs[1].record()
        Z.slot_confidence(s["hidden"], s["w_vocab"], target_ids=targets, out=tout)
        if evs:
            evs[2].record()
        Z.verify_accept(tout["target_prob"].view(B, S, L), selected, thr, Z.ACCEPT_PREFIX, out=acc_out)
        if evs:
            evs[3].record()
        Z.kv_append(kc, vc, plens, s["k_slot"], s["v_slot"], acc_out[0], selected)
        if evs:
            evs[4].record()

    def reset_and_run():
        plens.copy_(plens0)
        one()

    spin_up(reset_and_run, spin_s)
    for _ in range(3):
        reset_and_run()
    torch.cuda.synchronize()
    # steps run back to back (the reset is a copy on the same stream, between
    # the timed events); the host reads the events and counts once at the end
    ev_steps = []
    appended = []
    for _ in range(K):
        plens.copy_(plens0)
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(5)]
        one(evs)
        ev_steps.append(evs)
        appended.append((plens - plens0).float().mean())
    torch.cuda.synchronize()
    per = [[evs[j].elapsed_time(evs[j + 1]) * 1e3 for j in range(4)] for evs in ev_steps]
    appended = [float(a) for a in appended]
    m = [statistics.mean(p[j] for p in per) for j in range(4)]
    return {"slot_attn_ar_infill_us": m[0], "slot_confidence_targets_us": m[1], "verify_accept_us": m[2],
            "kv_append_us": m[3], "step_us": sum(m), "steps_per_s": 1e6 / sum(m),
            "tokens_appended_per_row": statistics.mean(appended), "token_threshold": thr}


def sampled_draft(dev, wl, sets, K, greedy_ms, spin_s):
    """Drafting with temperature (Sec. 5.2 "Sampling from categorical
    distribution"): the LM-head reduction with Gumbel-max sampling fused in,
    timed alone on the scoring step's hidden states, one Philox offset per
    step."""
    import torch

    import paper_2609_19868_amd as Z
    from paper_2609_19868_amd import _lib

    M, H, V = wl.M, wl.hidden, wl.vocab
    out = {k: torch.empty(M, dtype=torch.float32, device=dev) for k in ("sample_prob", "max_prob", "lse")}
    out["sample_id"] = torch.empty(M, dtype=torch.int32, device=dev)
    ws = torch.empty(_lib.slot_sample_workspace_size(_lib.ConfDesc(n_rows=M, hidden=H, vocab=V, dtype=1)),
                     dtype=torch.uint8, device=dev)
    ctr = itertools.count()

    def sample_once():
        i = next(ctr)
        Z.slot_sample(sets[i % len(sets)]["hidden"], sets[i % len(sets)]["w_vocab"], 1.0, 2024, i, out=out,
                      workspace=ws)

    spin_up(sample_once, spin_s)
    for _ in range(3):
        sample_once()
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(K)]
    for i in range(K):
        s = sets[i % len(sets)]
        evs[i][0].record()
        Z.slot_sample(s["hidden"], s["w_vocab"], 1.0, 2024, 100 + i, out=out, workspace=ws)
        evs[i][1].record()
    torch.cuda.synchronize()
    us = statistics.mean(a.elapsed_time(b) for a, b in evs) * 1e3
    return {"slot_sample_us": us, "tflops": 2.0 * M * V * H / (us * 1e-6) / 1e12,
            "uniforms_per_s": M * V / (us * 1e-6), "vs_greedy_reduction": us / (greedy_ms * 1e3)}


def mode_a_step(dev, w_vocab, K, spin_s):
    """One denoising step of Mode A (Sec. 5.1) at the modeA workload: causal
    attention of the 4 tokens revealed at the previous step and the 256 masked
    ones after a 2048-token prompt, Gumbel-max sampling of the masked rows,
    the reveal of the 4 most confident, and the cache append of the previous
    step's 4.  The prefix lengths are reset between steps, outside the timed
    events."""
    import numpy as np
    import torch

    import paper_2609_19868_amd as Z
    import workloads as W

    wl = W.WORKLOADS["modeA"]
    B, Hq, Hkv, D, P, R = wl.batch, wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.prefix_len, wl.T
    k_prev = W.MODE_A_REVEALED
    Nt = R - k_prev
    x = W.attention_inputs(wl)

    def dev_bf16(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)

    xd = {k: dev_bf16(v) for k, v in x.items()}
    kc = torch.empty((B, Hkv, P + k_prev, D), dtype=torch.bfloat16, device=dev)
    vc = torch.empty_like(kc)
    kc[:, :, :P].copy_(xd["k_cache"])
    vc[:, :, :P].copy_(xd["v_cache"])
    del xd["k_cache"], xd["v_cache"]
    rng = np.random.default_rng(wl.seed + 7_000_000)
    hidden = dev_bf16(W.bf16_bits(rng.standard_normal((B * Nt, wl.hidden), dtype=np.float32)))
    plens0 = torch.full((B,), P, dtype=torch.int32, device=dev)
    plens = plens0.clone()
    out = torch.empty((B, Hq, R, D), dtype=torch.bfloat16, device=dev)
    lse = torch.empty((B, Hq, R), dtype=torch.float32, device=dev)
    samp = {k: torch.empty(B * Nt, dtype=torch.float32, device=dev) for k in ("sample_prob", "max_prob", "lse")}
    samp["sample_id"] = torch.empty(B * Nt, dtype=torch.int32, device=dev)
    mask0 = torch.ones((B, Nt), dtype=torch.uint8, device=dev)
    mask = mask0.clone()
    kk = torch.full((B,), k_prev, dtype=torch.int32, device=dev)
    rev = (torch.empty((B, Nt), dtype=torch.int32, device=dev), torch.empty((B,), dtype=torch.int32, device=dev))
    acc = torch.zeros((B, R, 1), dtype=torch.uint8, device=dev)
    acc[:, :k_prev] = 1
    order = torch.arange(R, dtype=torch.int32, device=dev).repeat(B, 1).contiguous()

    # the first-hitting sampler's order: reveal uniformly random positions,
    # then sample only those rows (their hidden-row indices, b * Nt + position)
    samp_sel = {k: torch.empty(B * k_prev, dtype=torch.float32, device=dev)
                for k in ("sample_prob", "max_prob", "lse")}
    samp_sel["sample_id"] = torch.empty(B * k_prev, dtype=torch.int32, device=dev)
    row_base = (torch.arange(B, dtype=torch.int32, device=dev) * Nt).view(B, 1)
    sel_rows = torch.empty(B * k_prev, dtype=torch.int32, device=dev)

    def one(step, rule, evs=None):
        if evs:
            evs[0].record()
        Z.slot_attn(xd["q"], kc, vc, xd["k_slot"], xd["v_slot"], R, 1, pass_=Z.PASS_AR_INFILL,
                    cross_slot=Z.CROSS_SLOT_CAUSAL, prefix_len=P, out=out, lse=lse, prefix_lens=plens)
        if evs:
            evs[1].record()
        if rule == Z.REVEAL_CONFIDENCE:
            Z.slot_sample(hidden, w_vocab, 1.0, 2025, step, out=samp)
            if evs:
                evs[2].record()
            Z.mdm_reveal(mask, kk, rule, conf=samp["sample_prob"].view(B, Nt), out=rev)
            if evs:
                evs[3].record()
        else:
            Z.mdm_reveal(mask, kk, rule, seed=2026, offset=step, out=rev)
            if evs:
                evs[2].record()
            # row indices of the revealed positions (index arithmetic on 64 ints, outside the sampled rows' work)
            torch.add(rev[0][:, :k_prev], row_base, out=sel_rows.view(B, k_prev))
            Z.slot_sample(hidden, w_vocab, 1.0, 2025, step, rows=sel_rows, out=samp_sel)
            if evs:
                evs[3].record()
        Z.kv_append(kc, vc, plens, xd["k_slot"], xd["v_slot"], acc, order)
        if evs:
            evs[4].record()

    result = {"workload": f"modeA: B={B} Hq/Hkv={Hq}/{Hkv} D={D} P={P} rows={R} ({k_prev} revealed + {Nt} masked) "
                          f"H={wl.hidden} V={wl.vocab}"}
    for rule, name in ((Z.REVEAL_CONFIDENCE, "confidence"), (Z.REVEAL_RANDOM, "random")):
        ctr = itertools.count()

        def reset_and_run():
            plens.copy_(plens0)
            mask.copy_(mask0)
            one(next(ctr), rule)

        spin_up(reset_and_run, spin_s)
        for _ in range(3):
            reset_and_run()
        torch.cuda.synchronize()
        ev_steps = []
        for i in range(K):  # back to back; the resets run between the timed events
            plens.copy_(plens0)
            mask.copy_(mask0)
            evs = [torch.cuda.Event(enable_timing=True) for _ in range(5)]
            one(100 + i, rule, evs)
            ev_steps.append(evs)
        torch.cuda.synchronize()
        per = [[evs[j].elapsed_time(evs[j + 1]) * 1e3 for j in range(4)] for evs in ev_steps]
        m = [statistics.mean(p[j] for p in per) for j in range(4)]
        if rule == Z.REVEAL_CONFIDENCE:
            parts = {"slot_attn_causal_us": m[0], "slot_sample_all_masked_us": m[1], "mdm_reveal_us": m[2]}
        else:
            parts = {"slot_attn_causal_us": m[0], "mdm_reveal_us": m[1], "slot_sample_revealed_us": m[2]}
        result[name] = {**parts, "kv_append_us": m[3], "step_us": sum(m),
                        "revealed_tokens_per_s": B * k_prev * 1e6 / sum(m)}
    return result


def copy_calibration(dev, K):
    """A plain copy of known size: read 1 GiB, write 1 GiB, K times.  Under
    rocprofv3 --pmc its FETCH_SIZE / WRITE_SIZE per dispatch give the factor
    between the counters' reading and the bytes actually moved."""
    import torch

    n = 1 << 30
    src = torch.randint(0, 255, (n,), dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(K):
        dst.copy_(src)
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / K
    print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "us": ms * 1e3,
                      "gbps": 2 * n / (ms * 1e-3) / 1e9}), flush=True)


def single_sequence_step(dev, wl, K, spin_s):
    """The scoring step of one sequence (batch 1 of the same model and slot
    shape): the latency a single request sees.  Its 64 draft rows take the
    reduction's 64-row tile.  Inputs rotate over three copies of W."""
    import numpy as np
    import torch

    import paper_2609_19868_amd as Z
    import workloads as W

    w1 = wl.replace(batch=1, seed=wl.seed + 11)
    x = W.attention_inputs(w1)
    c = W.confidence_inputs(w1)

    def dev_bf16(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)

    xd = {k: dev_bf16(v) for k, v in x.items()}
    h = dev_bf16(c["hidden"])
    ws = [dev_bf16(c["w_vocab"])]
    ws += [ws[0].clone() for _ in range(2)]
    S, L = w1.n_slots, w1.slot_len

    def one(i, evs=None):
        if evs:
            evs[0].record()
        Z.slot_attn(xd["q"], xd["k_cache"], xd["v_cache"], xd["k_slot"], xd["v_slot"], S, L,
                    pass_=Z.PASS_DIFFUSION)
        if evs:
            evs[1].record()
        r = Z.slot_confidence(h, ws[i % 3])
        if evs:
            evs[2].record()
        Z.select_slots(r["max_prob"].view(1, S, L), threshold=0.9)
        if evs:
            evs[3].record()

    ctr = itertools.count()
    spin_up(lambda: one(next(ctr)), spin_s)
    for i in range(5):
        one(i)
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for i in range(K):
        one(i)
    t1.record()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(K)]
    for i in range(K):
        one(i, evs[i])
    torch.cuda.synchronize()
    m = [statistics.mean(e[j].elapsed_time(e[j + 1]) * 1e3 for e in evs) for j in range(3)]
    us = t0.elapsed_time(t1) / K * 1e3

    # The same step captured in HIP graphs (one per W copy) and replayed: the
    # host-side launch cost of the three calls leaves the critical path.
    graphs = []
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for i in range(3):
            one(i)
    torch.cuda.current_stream().wait_stream(side)
    for i in range(3):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            one(i)
        graphs.append(g)
    torch.cuda.synchronize()
    ctr = itertools.count()
    spin_up(lambda: graphs[next(ctr) % 3].replay(), spin_s)
    for i in range(3):
        graphs[i].replay()
    torch.cuda.synchronize()
    t0.record()
    for i in range(K):
        graphs[i % 3].replay()
    t1.record()
    torch.cuda.synchronize()
    us_graph = t0.elapsed_time(t1) / K * 1e3
    return {"workload": f"{wl.name} shapes at batch 1 ({S * L} draft rows)", "step_us": us,
            "steps_per_s": 1e6 / us, "slot_attn_us": m[0], "slot_confidence_us": m[1], "select_slots_us": m[2],
            "graph_step_us": us_graph, "graph_steps_per_s": 1e6 / us_graph}


def layout_attention(dev, K, spin_s):
    """Causal attention over the reordered training layout (B=8, 16/8 heads,
    N=4096 = 128 slots x 32 tokens, every slot AR_INFILL with earlier slots
    visible), through zarya_slot_attn with cross_slot = CAUSAL and no prefix."""
    import numpy as np
    import torch

    import workloads as W
    import paper_2609_19868_amd as Z

    wl = W.WORKLOADS["layout"]
    log("generating layout-attention inputs")
    x = W.attention_inputs(wl)
    xd = {k: torch.from_numpy(np.ascontiguousarray(v).view(np.int16)).view(torch.bfloat16).to(dev) for k, v in x.items()}
    out = torch.empty_like(xd["q"])
    run = lambda: Z.slot_attn(xd["q"], None, None, xd["k_slot"], xd["v_slot"], wl.n_slots, wl.slot_len,
                              pass_=Z.PASS_AR_INFILL, cross_slot=Z.CROSS_SLOT_CAUSAL, out=out, want_lse=False)
    spin_up(run, spin_s)
    for _ in range(2):
        run()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(K):
        run()
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / K
    N = wl.T
    flops = 4.0 * wl.batch * wl.n_q_heads * wl.head_dim * (N * (N + 1) / 2)  # causal QK^T + PV
    tf = flops / (ms * 1e-3) / 1e12
    return {"us": ms * 1e3, "tflops": tf, "frac_bf16_peak": tf / PEAK_BF16_TFLOPS,
            "shape": "B=8 Hq/Hkv=16/8 D=128 N=4096 (128 slots x 32), causal"}


if __name__ == "__main__":
    main()
