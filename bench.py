"""Benchmark of the split-expert MoE layer on one MI355X.

Default workload: the Mixtral-8x7B-shaped MoE layer (d=4096, F=14336, E=8,
top-2, bf16 weights, fp32 accumulation), decode batch 1, split ratio r=0.5
with the top segments of experts 0-3 cached in the VRAM pool, a staging
buffer of K=2 whole-expert slots (the paper's buffer), every other segment in
pinned host RAM.  One step = one decode token through the whole hot path:
routing + next-layer prediction, grouping, residency resolution and miss
transfers, resident-segment FFN, streamed-segment FFN, combine and the
prefetch pass.  Each token meets the layer as a layer of a deep stack does:
the staging buffer holds none of the layer's segments when its routing
arrives (the other layers' misses cycle the buffer between two visits), so
the step time is the layer's steady state and not a matter of which tokens
fall into the timed window.  Tokens are independent N(0,1) rows, resident
in HBM before timing starts.

Prints one JSON line: value = MoE-layer latency in us per layer (lower is
better); plus the expert FFN kernel's roofline from HIP events over the
timed region, H2D bandwidth and overlap figures from the same events, the
hit path (every missing segment already staged), an all-resident (r=1)
variant that isolates the HBM-bound expert read, the Mixtral-shaped
32-layer stack at a 12 GiB budget (where cross-layer prefetch moves bytes),
and the CPU oracle timed on a bounded sample.
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

HBM_PEAK_GBPS = 8000.0
GIB = 1 << 30
PROFILES = os.path.join(ROOT, "profiles")
CALIB_BYTES = 256 << 20   # device-to-device copy that calibrates the PMC byte counters
FFN_KERNELS = ("ffn_chunk_kernel", "ffn_q_kernel", "mma_gateup", "mma_down")


def kernel_sources_sha():
    """Hash of the kernel and runtime sources (the runtime picks grids, task
    lists and splits): PMC traffic figures hold only for them."""
    import hashlib
    h = hashlib.sha256()
    for f in ("kernels.hip", "kernels.h", "runtime.hip"):
        with open(os.path.join(ROOT, "paper_2509_08342_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def pmc_profile_path(workload):
    return os.path.join(PROFILES, "ffn_%s_pmc.md" % workload)


def traffic_from_profile(workload):
    """(HBM bytes per FFN launch, algorithmic weight bytes per FFN launch of
    the same profiled run) from the committed PMC summary of this workload,
    or None when there is none or the sources changed since."""
    path = pmc_profile_path(workload)
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for line in f:
            if ":" in line and line.startswith("- ") and "`" in line:
                k, v = line[2:].split(":", 1)
                vals[k.strip().strip("`")] = v.strip().strip("`")
    if vals.get("kernels_sha256") != kernel_sources_sha():
        return None
    try:
        return int(vals["ffn_traffic_bytes_per_launch"]), int(vals["ffn_algorithmic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None

# name -> (shape, tokens per step, split ratio, per-layer budget in top
# segments (None: whole budget of the reference config), which tops to cache,
# staging-buffer slots: decode K whole experts, the paper's buffer; prefill
# the library's default 2K, so one expert's copies overlap another's compute)
def _workloads():
    import dataclasses
    import synth
    ds1 = dataclasses.replace(synth.DEEPSEEK, n_layers=1)
    qw1 = dataclasses.replace(synth.QWEN3, n_layers=1)
    return {
        # Mixtral-8x7B-shaped layer, decode batch 1, r = .5, tops of experts 0-3
        "mixtral-decode": dict(shape=synth.MIXTRAL, T=1, r=0.5, budget=lambda tb: 4 * tb,
                               tops=lambda rig: [0, 1, 2, 3], slots=2),
        # the same layer with 2-bit expert codes (the paper's HQQ Mixtral setting)
        "mixtral-q2-decode": dict(shape=synth.MIXTRAL_Q2, T=1, r=0.5, budget=lambda tb: 4 * tb,
                                  tops=lambda rig: [0, 1, 2, 3], slots=2),
        # DeepSeek-V2-Lite-shaped layer: 4 GiB over 26 layers at r = .5 (19 tops)
        "deepseek-decode": dict(shape=ds1, T=1, r=0.5, budget=lambda tb: (4 * GIB) // 26,
                                tops=lambda rig: list(range(19)), slots=6),
        "deepseek-prefill": dict(shape=ds1, T=512, r=0.5, budget=lambda tb: (4 * GIB) // 26,
                                 tops=lambda rig: list(range(19)), slots=0),
        # Qwen3-30B-A3B-shaped layer: 8 GiB over 48 layers at r = .5 (37 tops),
        # the Zipf-hot experts cached
        "qwen-decode16": dict(shape=qw1, T=16, r=0.5, budget=lambda tb: (8 * GIB) // 48,
                              tops=lambda rig: list(np.argsort(-rig.biases[0], kind="stable")[:37]), slots=0),
        "qwen-prefill": dict(shape=qw1, T=2048, r=0.5, budget=lambda tb: (8 * GIB) // 48,
                             tops=lambda rig: list(np.argsort(-rig.biases[0], kind="stable")[:37]), slots=0),
    }

# stacked workloads: shape, total budget V_e, uniform r (or "mixed": r by layer
# index mod 3 over {.25, .5, .75}), prefill tokens (0: none), decode batch
def _stacks():
    import synth
    return {
        # t_moe_us: the layer with every expert resident at the decode batch
        # (measured on this GPU), the configurator's T_comp^moe
        "mixtral-stack": dict(shape=synth.MIXTRAL_STACK, budget=12 * GIB, r=0.5, prefill=0, T=1, n_sets=4,
                              t_moe_us=208.0),
        "mixtral-stack-mixed": dict(shape=synth.MIXTRAL_STACK, budget=12 * GIB, r="mixed", prefill=0, T=1,
                                    n_sets=4, t_moe_us=208.0),
        # 2-bit expert codes (the paper's HQQ Mixtral): 2 GiB keeps two tops
        # per layer at r = .5, as 12 GiB does for the bf16 stack
        "mixtral-q2-stack": dict(shape=synth.MIXTRAL_Q2_STACK, budget=2 * GIB, r=0.5, prefill=0, T=1, n_sets=4,
                                 t_moe_us=70.0),
        "deepseek-stack": dict(shape=synth.DEEPSEEK, budget=4 * GIB, r=0.5, prefill=512, T=1, n_sets=4,
                               t_moe_us=117.0),
        "qwen-stack": dict(shape=synth.QWEN3, budget=8 * GIB, r=0.5, prefill=2048, T=16, n_sets=4,
                           t_moe_us=305.0),
    }


# decoder loops: the MoE stack with Mixtral's attention and head, a prompt
# (time to first token), then greedy decode (time per output token); the
# cache is warmed by a first generation with LCP replacement
def _decoders():
    import synth
    return {
        "mixtral-decoder": dict(shape=synth.MIXTRAL_STACK, attn=synth.MIXTRAL_ATTN, budget=12 * GIB, r=0.5,
                                prompt=512, n_sets=4, t_moe_us=208.0),
        "mixtral-q2-decoder": dict(shape=synth.MIXTRAL_Q2_STACK, attn=synth.MIXTRAL_ATTN, budget=2 * GIB, r=0.5,
                                   prompt=512, n_sets=4, t_moe_us=70.0),
        # the budget of the paper's Mixtral TPOT comparison (Sec. 4.2): 160 of
        # the 256 experts; r = 5/8 caches every expert's top at that budget
        "mixtral-q2-decoder-160": dict(shape=synth.MIXTRAL_Q2_STACK, attn=synth.MIXTRAL_ATTN,
                                       budget=160 * synth.MIXTRAL_Q2_STACK.expert_bytes, r=0.625,
                                       prompt=512, n_sets=4, t_moe_us=70.0),
    }


METRIC = "MoE-layer decode µs/layer + achieved HBM GB/s; H2D overlap % at fixed VRAM budget"
KERNEL_KINDS = ("router", "group", "predict", "ffn_resident", "ffn_streamed", "ffn_down", "combine")
COPY_KINDS = ("copy_miss", "copy_prefetch")


# ------------------------------------------------------------ interval math

def _union(iv):
    iv = sorted((a, b) for a, b in iv if b > a)
    out = []
    for a, b in iv:
        if out and a <= out[-1][1]:
            out[-1][1] = max(out[-1][1], b)
        else:
            out.append([a, b])
    return out


def _length(u):
    return sum(b - a for a, b in u)


def _intersect(u, v):
    i = j = 0
    tot = 0.0
    while i < len(u) and j < len(v):
        a, b = max(u[i][0], v[j][0]), min(u[i][1], v[j][1])
        if b > a:
            tot += b - a
        if u[i][1] < v[j][1]:
            i += 1
        else:
            j += 1
    return tot


def analyse(tl, steps, ms_per_step, router_starts=True):
    by = {}
    for r in tl:
        by.setdefault(r["kind"], []).append(r)
    kern = {}
    for k in KERNEL_KINDS:
        rs = by.get(k, [])
        dur = sum(r["t1_ms"] - r["t0_ms"] for r in rs)
        kern[k] = dict(launches=len(rs), total_ms=dur, bytes=sum(r["bytes"] for r in rs))
    # per-step latency: from a step's routing launch to its last record
    # (single-layer workloads: one routing launch per step)
    starts = sorted(r["t0_ms"] for r in by.get("router", [])) if router_starts else []
    step_ms = []
    for i, t0 in enumerate(starts):
        t1 = starts[i + 1] if i + 1 < len(starts) else float("inf")
        ends = [r["t1_ms"] for r in tl if t0 <= r["t0_ms"] < t1]
        step_ms.append(max(ends) - t0)
    copies = [r for k in COPY_KINDS for r in by.get(k, [])]
    copy_u = _union([(r["t0_ms"], r["t1_ms"]) for r in copies])
    kern_u = _union([(r["t0_ms"], r["t1_ms"]) for k in KERNEL_KINDS for r in by.get(k, [])])
    copy_t, kern_t = _length(copy_u), _length(kern_u)
    both = _intersect(copy_u, kern_u)
    copy_bytes = sum(r["bytes"] for r in copies)
    t_layer = ms_per_step * steps
    eta = None
    if copy_t > 0 and kern_t > 0:
        eta = (kern_t + copy_t - t_layer) / min(kern_t, copy_t)
    return dict(
        kernels=kern,
        copy_ms=copy_t, kernel_ms=kern_t, copy_bytes=copy_bytes,
        h2d_gbps=(copy_bytes / (copy_t * 1e-3) / 1e9) if copy_t > 0 else None,
        hidden_frac=(both / copy_t) if copy_t > 0 else None,
        compute_hidden_frac=(both / kern_t) if kern_t > 0 else None,
        overlap_eta=eta,
        step_us=({q: round(float(np.percentile(step_ms, p)) * 1e3, 1) for q, p in (("p10", 10), ("p50", 50), ("p90", 90))}
                 if step_ms else None),
        miss_bytes=sum(r["bytes"] for r in by.get("copy_miss", [])),
        prefetch_bytes=sum(r["bytes"] for r in by.get("copy_prefetch", [])),
    )


PCIE_GEN5_X16_GBPS = 32.0 * 16 * 128 / 130 / 8  # 63.0 GB/s per direction: 32 GT/s x 16 lanes, 128b/130b


def copy_roofline(tl):
    """Host-to-device segment copies (the copy kernel or the DMA engines):
    bytes per copy / average copy duration against the PCIe 5.0 x16 link."""
    rs = [r for r in tl if r["kind"] in COPY_KINDS]
    dur = sum(r["t1_ms"] - r["t0_ms"] for r in rs)
    if not rs or dur <= 0:
        return None
    b = sum(r["bytes"] for r in rs)
    gbps = b / (dur * 1e-3) / 1e9
    return dict(bound="pcie", achieved=round(gbps, 2), peak=round(PCIE_GEN5_X16_GBPS, 2), unit="GB/s",
                frac=round(gbps / PCIE_GEN5_X16_GBPS, 4), launches=len(rs),
                avg_launch_us=round(dur / len(rs) * 1e3, 2), bytes_per_launch=int(b / len(rs)))


def ffn_roofline(an):
    """Expert FFN kernels (resident and streamed launches are the same
    kernel; the prefill path adds the down projection): weight bytes read per
    launch / average launch duration."""
    ks = [an["kernels"]["ffn_resident"], an["kernels"]["ffn_streamed"], an["kernels"]["ffn_down"]]
    n = sum(k["launches"] for k in ks)
    ms_tot = sum(k["total_ms"] for k in ks)
    b = sum(k["bytes"] for k in ks)
    if n == 0 or ms_tot <= 0:
        return None
    gbps = b / (ms_tot * 1e-3) / 1e9
    return dict(bound="hbm", achieved=round(gbps, 1), peak=HBM_PEAK_GBPS, unit="GB/s",
                frac=round(gbps / HBM_PEAK_GBPS, 4), traffic=None,
                launches=n, avg_launch_us=round(ms_tot / n * 1e3, 2),
                bytes_per_launch=int(b / n))


MFMA_BF16_PEAK_TFLOPS = 2500.0  # dense bf16 matrix-core peak of MI355X


def mfma_roofline(an, shape, T, steps):
    """Matrix-core FFN kernels of the prefill path (gate/up and down launches):
    algorithmic flops (6 d F per token and selected expert, plus the shared
    experts' 6 d F_sh per token) over their summed launch durations, against
    the bf16 dense peak and against the attainable bound min(peak, flops per
    weight byte x 8 TB/s), where the weight bytes are those the launches
    read.  None when the forwards took the decode path."""
    ks = [an["kernels"]["ffn_resident"], an["kernels"]["ffn_streamed"], an["kernels"]["ffn_down"]]
    if an["kernels"]["ffn_down"]["launches"] == 0:
        return None
    ms_tot = sum(k["total_ms"] for k in ks)
    b = sum(k["bytes"] for k in ks)
    if ms_tot <= 0 or b <= 0:
        return None
    flops_step = 6.0 * shape.d_model * (shape.d_ff * T * shape.top_k + shape.d_ff_shared * T * shape.n_shared)
    flops = flops_step * steps
    tflops = flops / (ms_tot * 1e-3) / 1e12
    intensity = flops / b
    hbm_tflops = intensity * HBM_PEAK_GBPS * 1e9 / 1e12
    attainable = min(MFMA_BF16_PEAK_TFLOPS, hbm_tflops)
    return dict(bound="mfma" if MFMA_BF16_PEAK_TFLOPS < hbm_tflops else "hbm", achieved=round(tflops, 1),
                peak=MFMA_BF16_PEAK_TFLOPS, unit="TFLOP/s", frac=round(tflops / MFMA_BF16_PEAK_TFLOPS, 4),
                attainable=round(attainable, 1), attainable_frac=round(tflops / attainable, 4),
                flop_per_weight_byte=round(intensity, 1), flops_per_step=flops_step,
                launches=sum(k["launches"] for k in ks))


def _read(path):
    try:
        with open(path) as f:
            return f.read().strip()
    except OSError:
        return None


def platform_info():
    """The machine the figures come from: GPU name, architecture and CU
    count, its current and peak engine / memory clocks (sysfs DPM tables,
    else rocm-smi), the PCIe link's current and maximum speed and width, and
    the host CPU model with the cores this process may use.  Read from sysfs,
    /proc and a rocm-smi child process; a field that cannot be read is None."""
    import subprocess
    import torch
    info = {}
    try:
        pr = torch.cuda.get_device_properties(0)
        info["gpu"] = {"name": pr.name, "arch": pr.gcnArchName, "compute_units": pr.multi_processor_count,
                       "memory_gib": round(pr.total_memory / GIB, 1)}
        bdf = "%04x:%02x:%02x.0" % (pr.pci_domain_id, pr.pci_bus_id, pr.pci_device_id)
        dev = "/sys/bus/pci/devices/" + bdf
        info["pcie"] = {"bdf": bdf, "current_link_speed": _read(dev + "/current_link_speed"),
                        "current_link_width": _read(dev + "/current_link_width"),
                        "max_link_speed": _read(dev + "/max_link_speed"),
                        "max_link_width": _read(dev + "/max_link_width")}
        clocks = {}
        for key, fname in (("sclk", "pp_dpm_sclk"), ("mclk", "pp_dpm_mclk")):
            table = _read(dev + "/" + fname)
            if table:
                lines = [l for l in table.splitlines() if l.strip()]
                cur = [l for l in lines if l.rstrip().endswith("*")]
                clocks[key] = {"current": cur[0].split(":", 1)[1].strip(" *") if cur else None,
                               "levels": [l.split(":", 1)[1].strip(" *") for l in lines]}
        if not clocks:
            try:
                r = subprocess.run(["rocm-smi", "--showclocks"], capture_output=True, text=True, timeout=30)
                clocks["rocm_smi"] = [l.strip() for l in r.stdout.splitlines() if "clk" in l.lower()][:8]
            except (OSError, subprocess.SubprocessError):
                pass
        info["clocks"] = clocks or None
    except Exception as e:  # reporting only: never fail the benchmark
        info["error"] = repr(e)[:200]
    cpuinfo = _read("/proc/cpuinfo") or ""
    models = [l.split(":", 1)[1].strip() for l in cpuinfo.splitlines() if l.startswith("model name")]
    info["cpu"] = {"model": models[0] if models else None, "logical_cpus": os.cpu_count(),
                   "usable_cpus": len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else None}
    try:
        r = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=30)
        want = {"Model name": "lscpu_model", "Socket(s)": "sockets", "Core(s) per socket": "cores_per_socket",
                "Thread(s) per core": "threads_per_core", "CPU(s)": "cpus", "CPU max MHz": "max_mhz"}
        for line in r.stdout.splitlines():
            k, _, v = line.partition(":")
            if k.strip() in want and v.strip():
                info["cpu"][want[k.strip()]] = v.strip()
    except (OSError, subprocess.SubprocessError):
        pass
    return info


# ------------------------------------------------------------------ timing

def run_steps(rig, hs, steps, warmup, flags, timeline=True, cold=False, T=1, before_timed=None, per_step=None):
    """Time `steps` batches of T tokens through layer 0.  cold=True drops the
    staging buffer before every batch, so each pays all of its misses, as a
    layer of a deep stack does.  per_step: a list that receives each timed
    step's span in ms (between HIP events recorded after consecutive
    forwards on the compute stream)."""
    import torch
    from paper_2509_08342_amd import moesplit as ms
    stream = torch.cuda.current_stream()
    y, idx, w = rig.outputs(T)
    # every pass starts from an empty staging buffer, so passes over the same
    # tokens start from the same state
    ms.ms_drop_buffer(rig.ctx)
    for i in range(warmup):
        if cold:
            ms.ms_drop_buffer(rig.ctx)
        rig.forward(0, hs[i % len(hs)], T, y, idx, w, flags, stream)
    ms.ms_sync(rig.ctx)
    torch.cuda.synchronize()
    ms.ms_reset_stats(rig.ctx)
    if before_timed is not None:
        before_timed()
    if timeline:
        # room for every record of the timed steps (events are created up front)
        cap = min(1 << 16, max(1024, steps * (4 * rig.shape.n_experts + 64)))
        ms.ms_timeline_begin(rig.ctx, stream, cap)
    evs = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    if per_step is not None:
        evs.append(torch.cuda.Event(enable_timing=True))
        evs[-1].record(stream)
    for i in range(steps):
        if cold:
            ms.ms_drop_buffer(rig.ctx)
        rig.forward(0, hs[(warmup + i) % len(hs)], T, y, idx, w, flags, stream)
        if per_step is not None:
            evs.append(torch.cuda.Event(enable_timing=True))
            evs[-1].record(stream)
    ms.ms_sync(rig.ctx)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    if per_step is not None:
        per_step.extend(a.elapsed_time(b) for a, b in zip(evs, evs[1:]))
    tl = ms.ms_timeline_end(rig.ctx) if timeline else []
    st = ms.ms_stats(rig.ctx, 0)
    return (t1 - t0) * 1e3 / steps, tl, st


def run_hit_path(rig, hs, steps, T=1):
    """The layer when every selected expert's missing segment is already in
    the staging buffer (a prediction that was right and a prefetch that had
    time to land): per step, the buffer is emptied and the token run once
    untimed to stage its misses, then run again between two HIP events on
    the compute stream.  Returns the per-step times in ms and the buffer
    hits of the timed forwards, or (None, 0) when a batch misses more experts
    than the buffer has slots (the staged segments of one expert are then
    overwritten by another's, and the path does not exist)."""
    import torch
    from paper_2509_08342_amd import moesplit as ms
    stream = torch.cuda.current_stream()
    y, idx, w = rig.outputs(T)
    per = []
    hits = 0
    for i in range(steps):
        ms.ms_drop_buffer(rig.ctx)
        rig.forward(0, hs[i % len(hs)], T, y, idx, w, 0, stream)
        ms.ms_sync(rig.ctx)
        torch.cuda.synchronize()
        before = ms.ms_stats(rig.ctx, 0)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        rig.forward(0, hs[i % len(hs)], T, y, idx, w, 0, stream)
        e1.record(stream)
        ms.ms_sync(rig.ctx)
        torch.cuda.synchronize()
        after = ms.ms_stats(rig.ctx, 0)
        if after["bytes_miss"] != before["bytes_miss"]:
            return None, 0
        hits += after["buffer_hits"] - before["buffer_hits"]
        per.append(e0.elapsed_time(e1))
    return per, hits


def h2d_link_peak_gbps():
    import torch
    n = 1 << 30
    hbuf = torch.empty(n, dtype=torch.uint8, pin_memory=True)
    dbuf = torch.empty(n, dtype=torch.uint8, device="cuda")
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        dbuf.copy_(hbuf, non_blocking=True)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(s)
        for _ in range(3):
            dbuf.copy_(hbuf, non_blocking=True)
        e1.record(s)
    torch.cuda.synchronize()
    ms_ = e0.elapsed_time(e1) / 3
    del hbuf, dbuf
    return n / (ms_ * 1e-3) / 1e9


def cpu_baseline_q(rig, hf_list, budget_s):
    """The b-bit oracle, one thread: routing of each batch, then each row's
    selected experts over the first eighth of their units (dequantizing only
    those), scaled by eight; as many batches as fit in about budget_s."""
    import oracle
    from oracle import quant
    s = rig.shape
    frac = 8
    hi = (s.d_ff // frac) // 64 * 64
    T = hf_list[0].shape[0]
    rows = list(range(min(T, 16)))
    experts = rig.layer_experts(0)
    t0 = time.perf_counter()
    n = 0
    for hf in hf_list:
        logits = oracle.router_logits(hf, rig.routers[0], rig.biases[0])
        idx = oracle.topk(logits, s.top_k)
        w = oracle.gate_weights(logits, idx, s.renormalize)
        for t in rows:
            y = np.zeros(s.d_model)
            for k in range(s.top_k):
                q = experts[int(idx[t, k])]
                y += w[t, k] * quant.expert_range(hf[t], q.codes, q.meta, q.bits, s.d_model, s.d_ff, 0, hi)
        n += 1
        if time.perf_counter() - t0 > budget_s:
            break
    dt = time.perf_counter() - t0
    scale = (T / len(rows)) * (s.d_ff / hi)
    return dict(value=round(dt / n * scale * 1e6, 1), unit="us/layer", cores=1, kind="oracle",
                sample="%d batches of %d token(s) of the %s layer (router on all rows, %d experts per row "
                "on %d rows over %d of %d units, dequantized per call, fp64, scaled to the batch and the "
                "whole expert)" % (n, T, s.name, s.top_k, len(rows), hi, s.d_ff))


def cpu_baseline(rig, hf_list, budget_s):
    """The oracle as it stands on as many batches of the same layer as fit
    in about budget_s seconds.  Decode batches (up to 16 tokens): one thread,
    every row.  Prefill batches: the unchanged oracle called from one thread
    per usable host core on disjoint blocks of 16 rows (its C expert loops
    release the interpreter lock), routing on all rows in each call, and the
    time scaled to the whole batch."""
    import oracle
    from concurrent.futures import ThreadPoolExecutor
    s = rig.shape
    if getattr(s, "expert_bits", 0):
        return cpu_baseline_q(rig, hf_list, budget_s)
    T = hf_list[0].shape[0]
    per = 16
    n_thr = 1 if T <= per else max(1, len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity")
                                   else (os.cpu_count() or 1))
    n_rows = min(T, per * n_thr)
    blocks = [list(range(i, min(i + per, n_rows))) for i in range(0, n_rows, per)]

    def run(hf, rows):
        oracle.moe_layer(hf, rig.routers[0], rig.layer_experts(0), s.top_k, renormalize=s.renormalize,
                         bias=rig.biases[0], shared=rig.shared[0], tokens=rows)

    t0 = time.perf_counter()
    n = 0
    with ThreadPoolExecutor(len(blocks)) as ex:
        for hf in hf_list:
            list(ex.map(lambda rows: run(hf, rows), blocks))
            n += 1
            if time.perf_counter() - t0 > budget_s:
                break
    dt = time.perf_counter() - t0
    scale = T / n_rows
    where = ("every row, one thread" if len(blocks) == 1 and n_rows == T else
             "%d rows in %d threads of up to %d rows, scaled to the batch" % (n_rows, len(blocks), per))
    return dict(value=round(dt / n * scale * 1e6, 1), unit="us/layer", cores=len(blocks), kind="oracle",
                sample="%d batches of %d token(s) of the %s layer (router on all rows, %d experts per row on %s; "
                "experts in fp64)" % (n, T, s.name, s.top_k, where))


def log(msg):
    print("[bench] " + msg, file=sys.stderr, flush=True)


# ------------------------------------------------------- rocprofv3 summaries

def _read_rows(d, suffix):
    import csv
    import glob
    rows = []
    for f in sorted(glob.glob(os.path.join(d, "**", "*" + suffix), recursive=True)):
        with open(f, newline="") as fh:
            rows.extend(csv.DictReader(fh))
    if not rows:
        raise SystemExit("no *%s under %s" % (suffix, d))
    return rows


def _counter_by_dispatch(d):
    """{dispatch id: (kernel name, counter value)} from a --pmc run of one counter."""
    out = {}
    for r in _read_rows(d, "counter_collection.csv"):
        did = int(r["Dispatch_Id"])
        name, val = r["Kernel_Name"], float(r["Counter_Value"])
        prev = out.get(did)
        out[did] = (name, val + (prev[1] if prev else 0.0))
    return out


def pmc_summary(fetch_dir, write_dir, workload, out, cmd_fetch, cmd_write, pass_log=None):
    """FETCH_SIZE and WRITE_SIZE (KiB per dispatch) of the FFN kernels in the
    timed steps of a --pmc-pass run, each scaled by the same counter on the
    calibration copy of CALIB_BYTES (the largest __amd_rocclr_copyBuffer
    dispatch, issued just before the timed steps).  pass_log: the JSON line
    the --pmc-pass run printed, whose algorithmic FFN bytes of the same
    dispatches are recorded beside the counted traffic."""
    alg = None
    if pass_log:
        with open(pass_log) as f:
            for line in f:
                if line.startswith("{") and "pmc_pass" in line:
                    rec = json.loads(line)
                    if rec.get("ffn_launches"):
                        alg = (rec["ffn_launches"], rec["ffn_algorithmic_bytes"])
    res = {}
    for label, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        by = _counter_by_dispatch(d)
        copies = [(v[1], did) for did, v in by.items() if "copyBuffer" in v[0]]
        cal_kib, cal_id = max(copies)
        factor = cal_kib * 1024.0 / CALIB_BYTES
        kern = {}
        for did, (name, val) in by.items():
            if did <= cal_id:
                continue
            short = name.split("(")[0].replace("void ", "")
            k = kern.setdefault(short, [0, 0.0])
            k[0] += 1
            k[1] += val
        res[label] = dict(cal_kib=cal_kib, factor=factor, kern=kern)
    f_fac, w_fac = res["FETCH_SIZE"]["factor"], res["WRITE_SIZE"]["factor"]
    names = sorted(set(res["FETCH_SIZE"]["kern"]) | set(res["WRITE_SIZE"]["kern"]))
    ffn_n, ffn_bytes = 0, 0.0
    lines = ["# FFN kernels, %s workload: HBM traffic from rocprofv3 counters" % workload, "",
             "Commands (from the repository root, on one MI355X):", "",
             "    " + cmd_fetch, "    " + cmd_write, "",
             "Calibration: a device-to-device copy of %d bytes (torch copy_, the runtime's "
             "copyBuffer kernel) issued right before the timed steps; each counter is divided "
             "by what it reads for that copy per byte moved." % CALIB_BYTES, "",
             "| counter | calibration copy reads (KiB) | factor (counter bytes per byte moved) |",
             "|---|---|---|",
             "| FETCH_SIZE | %.0f | %.4f |" % (res["FETCH_SIZE"]["cal_kib"], f_fac),
             "| WRITE_SIZE | %.0f | %.4f |" % (res["WRITE_SIZE"]["cal_kib"], w_fac), "",
             "Dispatches after the calibration copy (warm-up excluded), scaled bytes per dispatch:", "",
             "| kernel | dispatches | fetch MB/dispatch | write MB/dispatch |", "|---|---|---|---|"]
    for n in names:
        fk = res["FETCH_SIZE"]["kern"].get(n, [0, 0.0])
        wk = res["WRITE_SIZE"]["kern"].get(n, [0, 0.0])
        cnt = max(fk[0], wk[0])
        fb = fk[1] * 1024.0 / f_fac / max(fk[0], 1)
        wb = wk[1] * 1024.0 / w_fac / max(wk[0], 1)
        lines.append("| `%s` | %d | %.3f | %.3f |" % (n, cnt, fb / 1e6, wb / 1e6))
        if any(k in n for k in FFN_KERNELS):
            ffn_n += cnt
            ffn_bytes += (fb + wb) * cnt
    per = int(ffn_bytes / max(ffn_n, 1))
    lines += ["", "Figures bench.py reads (valid while the kernel and runtime sources hash the same):", "",
              "- `workload`: `%s`" % workload,
              "- `ffn_dispatches`: `%d`" % ffn_n,
              "- `ffn_traffic_bytes_per_launch`: `%d`" % per]
    if alg is not None:
        if alg[0] != ffn_n:
            raise SystemExit("the pass log counts %d FFN launches, the counters %d" % (alg[0], ffn_n))
        ap = int(alg[1] / alg[0])
        lines += ["- `ffn_algorithmic_bytes_per_launch`: `%d`" % ap,
                  "- `ffn_traffic_ratio`: `%.4f`" % (per / ap)]
    lines += ["- `kernels_sha256`: `%s`" % kernel_sources_sha(), ""]
    with open(out, "w") as f:
        f.write("\n".join(lines))
    print("wrote %s: %d FFN dispatches, %.3f MB per launch" % (out, ffn_n, per / 1e6))


def mfma_pmc_summary(d, workload, out, cmd):
    """SQ_VALU_MFMA_BUSY_CYCLES and GRBM_GUI_ACTIVE per dispatch of a --pmc
    run of both counters, by kernel.  As rocprofv3 reports them on this GPU,
    GRBM_GUI_ACTIVE is summed over the 8 XCDs (per dispatch it is 8 x the
    kernel's cycles) and SQ_VALU_MFMA_BUSY_CYCLES over the 1024 SIMDs (16
    busy cycles per v_mfma_f32_16x16x32_bf16, the rate of the 2.5 PFLOP/s
    bf16 peak), so the matrix cores' busy fraction is
    busy / (GRBM_GUI_ACTIVE / 8 x 1024)."""
    by = {}
    for r in _read_rows(d, "counter_collection.csv"):
        e = by.setdefault(int(r["Dispatch_Id"]), {"name": r["Kernel_Name"]})
        e[r["Counter_Name"]] = e.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    kern = {}
    for e in by.values():
        short = e["name"].split("(")[0].replace("void ", "")
        k = kern.setdefault(short, [0, 0.0, 0.0])
        k[0] += 1
        k[1] += e.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0)
        k[2] += e.get("GRBM_GUI_ACTIVE", 0.0)
    lines = ["# Matrix-core busy cycles, %s workload, rocprofv3 counters" % workload, "",
             "Command (from the repository root, on one MI355X):", "", "    " + cmd, "",
             "GRBM_GUI_ACTIVE is summed over the 8 XCDs (8 x the kernel's cycles per dispatch) and "
             "SQ_VALU_MFMA_BUSY_CYCLES over the 1024 SIMDs (16 cycles per 16x16x32 bf16 MFMA), so the "
             "matrix cores are busy for busy / (GUI_ACTIVE / 8 x 1024) of the kernel's time.", "",
             "| kernel | dispatches | SQ_VALU_MFMA_BUSY_CYCLES / dispatch | GRBM_GUI_ACTIVE / dispatch | "
             "kernel cycles (GUI_ACTIVE / 8) | MFMA busy fraction |", "|---|---|---|---|---|---|"]
    for n, (c, busy, gui) in sorted(kern.items(), key=lambda x: -x[1][1]):
        lines.append("| `%s` | %d | %.4g | %.4g | %.4g | %.4f |" % (
            n, c, busy / c, gui / c, gui / c / 8.0, busy / max(gui / 8.0 * 1024.0, 1.0)))
    with open(out, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("wrote %s (%d kernels)" % (out, len(kern)))


def trace_summary(d, out, cmd):
    """Kernel statistics of a rocprofv3 --kernel-trace --stats run."""
    rows = _read_rows(d, "kernel_stats.csv")
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    lines = ["# Kernel time, rocprofv3 --kernel-trace --stats", "", "Command (from the repository root, on one MI355X):",
             "", "    " + cmd, "", "| kernel | calls | total ms | average us | min us | max us | share |",
             "|---|---|---|---|---|---|---|"]
    for r in rows:
        lines.append("| `%s` | %s | %.3f | %.2f | %.2f | %.2f | %.1f%% |" % (
            r["Name"].split("(")[0].replace("void ", ""), r["Calls"], float(r["TotalDurationNs"]) / 1e6,
            float(r["AverageNs"]) / 1e3, float(r["MinNs"]) / 1e3, float(r["MaxNs"]) / 1e3, float(r["Percentage"])))
    with open(out, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("wrote %s (%d kernels)" % (out, len(rows)))


def run_decoder(args):
    """A decoder loop: warm-up generation (LCP replacement fills the caches),
    then a fresh prompt (TTFT) and greedy decode steps (TPOT), then a few
    decode steps with events around each module (T_att, T_moe, T_head)."""
    import torch
    import synth
    from paper_2509_08342_amd import moesplit as ms
    from decoder import Decoder
    cfg = _decoders()[args.workload]
    shape, attn, P = cfg["shape"], cfg["attn"], cfg["prompt"]
    L, E = shape.n_layers, shape.n_experts
    n_warm, n_marks = 16, 4
    n_new = args.warmup + args.steps + 1
    max_ctx = P + max(n_warm, n_new + n_marks) + 8
    t_setup = time.perf_counter()
    log("generating %s weights (%d distinct sets over %d layers) and attention" % (shape.name, cfg["n_sets"], L))
    dec = Decoder(shape, attn, seed=0, n_sets=cfg["n_sets"], max_tokens=P, max_ctx=max_ctx,
                  budget_total=cfg["budget"], keep_f32=False)
    if args.copy_engine == "dma":
        ms.ms_set_copy_engine(dec.ctx, ms.MS_COPY_DMA)
    slots = dec.stack.configure(cfg["r"], cfg["budget"])
    log("setup %.1f s; warm-up generation (%d + %d tokens, LCP replacement)" % (time.perf_counter() - t_setup,
                                                                               P, n_warm))
    ms.ms_set_cache_policy(dec.ctx, ms.MS_CACHE_LCP)
    ms.ms_reset_plan_stats(dec.ctx)
    dec.generate(synth.prompt_tokens(attn, 0, P, tag=1), n_warm)
    ms.ms_sync(dec.ctx)
    stream = torch.cuda.current_stream()

    def module_times(n):
        """Per-token T_att, T_moe (summed over layers) and T_head in us."""
        x1 = torch.empty(1, shape.d_model, dtype=torch.bfloat16, device="cuda")
        acc = {"att": 0.0, "moe": 0.0, "head": 0.0}
        for _ in range(n):
            marks = []
            dec.embed_ids(dec.ids, 1, x1, stream)
            dec.step(x1, 1, stream=stream, marks=marks)
            stream.synchronize()
            for (name, e0), (_, e1) in zip(marks, marks[1:]):
                acc[name] += e0.elapsed_time(e1) * 1e3
        return {k: v / n for k, v in acc.items()}

    plan = None
    if args.configure:
        t = module_times(n_marks)
        hs_, ps_, phs_ = [], [], []
        for l in range(L):
            h_, p_, ph_, _ = ms.ms_plan_stats(dec.ctx, l, E)
            hs_.append(h_)
            ps_.append(p_)
            phs_.append(ph_)
        t_load = shape.expert_bytes / 55e3
        plan = ms.ms_plan_solve(L, E, shape.top_k, shape.expert_bytes, t["att"] / L, t["moe"] / L, t["head"],
                                t_load, np.array(hs_), np.array(ps_), np.array(phs_), cfg["budget"], args.zeta)
        ms.ms_cache_update(dec.ctx, plan["budgets"], plan["theta"].astype(np.float32))
        log("configurator (T_att %.0f us, T_moe %.0f us, T_head %.0f us): %d moves, theta %.3f..%.3f" % (
            t["att"] / L, t["moe"] / L, t["head"], plan["iters"], plan["theta"].min(), plan["theta"].max()))
    if args.policy == "static":
        ms.ms_set_cache_policy(dec.ctx, ms.MS_CACHE_STATIC)
    else:
        ms.ms_set_cache_policy(dec.ctx, {"lcp": ms.MS_CACHE_LCP, "lru": ms.MS_CACHE_LRU, "lfu": ms.MS_CACHE_LFU,
                                         "rnd": ms.MS_CACHE_RND}[args.policy])
    dec.reset()
    ms.ms_reset_stats(dec.ctx)
    prefill_st = []
    toks, ttft, tpot = dec.generate(synth.prompt_tokens(attn, 0, P, tag=2), n_new,
                                    after_prefill=lambda: prefill_st.extend(ms.ms_stats(dec.ctx, l) for l in range(L)))
    timed = tpot[args.warmup:]
    st = [ms.ms_stats(dec.ctx, l) for l in range(L)]
    # decode steps only: the counters after the prefill subtracted
    dst = [{k: x[k] - y[k] for k in x} for x, y in zip(st, prefill_st)]
    n_dec = max(len(tpot), 1)
    tm = module_times(n_marks)
    ms.ms_sync(dec.ctx)
    tpot_ms = float(np.mean(timed))
    sel = sum(x["experts_active"] for x in st)
    hits = sum(x["alpha"] + x["beta"] for x in st)
    out = {
        "metric": "decode time per output token (TPOT) of the decoder loop with split experts",
        "value": round(tpot_ms, 3), "unit": "ms/token", "higher_is_better": False,
        "data": "synthetic", "dtype": "bf16", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "config": {"workload": "%s: %s, %d layers, attention %d heads / %d kv heads x %d, vocab %d, V_e %.2f GiB, "
                               "r %s, prompt %d tokens, greedy decode, cache policy %s" % (
                                   args.workload, shape.name, L, attn.n_heads, attn.n_kv_heads, attn.head_dim,
                                   attn.vocab, cfg["budget"] / GIB,
                                   "from the configurator" if plan is not None else cfg["r"], P, args.policy)},
        "ttft_ms": round(ttft, 2),
        "tokens_per_s": round(1e3 / tpot_ms, 2),
        "tpot_ms": {q: round(float(np.percentile(timed, p)), 3) for q, p in (("p10", 10), ("p50", 50), ("p90", 90))},
        "module_us_per_token": {"attention_per_layer": round(tm["att"] / L, 1), "moe_per_layer": round(tm["moe"] / L, 1),
                                "head": round(tm["head"], 1)},
        "hit_rate": round(hits / max(sel, 1), 4),
        "h2d_bytes_per_decode_token": {k: sum(x["bytes_" + k] for x in dst) // n_dec
                                       for k in ("miss", "prefetch", "prefetch_used", "prefetch_dropped")},
        "h2d_bytes_prefill": {k: sum(x["bytes_" + k] for x in prefill_st) for k in ("miss", "prefetch")},
        "cache_inserts": sum(x["cache_inserts"] for x in st),
        "setup_s": round(time.perf_counter() - t_setup, 1),
    }
    if plan is not None:
        out["plan"] = {"moves": plan["iters"], "theta": [round(float(t), 4) for t in plan["theta"]],
                       "cache": [int(c) for c in plan["cache"]]}
    log("TTFT %.1f ms, TPOT %.2f ms" % (ttft, tpot_ms))
    dec.close()
    out["platform"] = platform_info()
    print(json.dumps(out), flush=True)


def measure_stack(name, steps, warmup, copy_engine="kernel", policy="static", configure=False, zeta=0.01,
                  instrument_steps=0):
    """A whole stack: warm-up statistics pick each layer's cached tops (or
    the configurator's plan), an optional prefill pass, then `steps` timed
    decode steps through every layer with cross-layer prediction and
    prefetch.  With instrument_steps > 0 the first that many timed tokens run
    again with the library's timeline on, which gives the copy / kernel
    overlap figures.  Returns the result dict."""
    import torch
    from paper_2509_08342_amd import moesplit as ms
    from stack import Stack, decode_inputs
    cfg = _stacks()[name]
    shape, T, P = cfg["shape"], cfg["T"], cfg["prefill"]
    L = shape.n_layers
    t_setup = time.perf_counter()
    log("generating %s weights (%d distinct sets over %d layers)" % (shape.name, cfg["n_sets"], L))
    st = Stack(shape, seed=0, n_sets=cfg["n_sets"], max_tokens=max(T, P), budget_total=cfg["budget"],
               keep_f32=False)
    if copy_engine == "dma":
        ms.ms_set_copy_engine(st.ctx, ms.MS_COPY_DMA)
    r = cfg["r"]
    rs = [(0.25, 0.5, 0.75)[l % 3] for l in range(L)] if r == "mixed" else [r] * L
    slots = st.configure(rs, cfg["budget"])
    n_warm, n_steps = 16, steps
    xs = decode_inputs(shape, 0, n_warm + warmup + n_steps, T)
    log("setup %.1f s; %d-step warm-up for the cache contents" % (time.perf_counter() - t_setup, n_warm))
    ms.ms_reset_plan_stats(st.ctx)
    counts = st.warmup_counts([x for x, _ in xs[:n_warm]], T)
    st.load_most_selected(counts)
    plan = None
    if configure:
        # Algorithm 1 on the warm-up statistics, then its cache update
        E = shape.n_experts
        hs_, ps_, phs_ = [], [], []
        for l in range(L):
            h_, p_, ph_, _ = ms.ms_plan_stats(st.ctx, l, E)
            hs_.append(h_)
            ps_.append(p_)
            phs_.append(ph_)
        t_load = shape.expert_bytes / 55e3   # us per whole expert at the kernel copy's 55 GB/s
        plan = ms.ms_plan_solve(L, E, shape.top_k, shape.expert_bytes, 0.0, cfg["t_moe_us"], 0.0, t_load,
                                np.array(hs_), np.array(ps_), np.array(phs_), cfg["budget"], zeta)
        ms.ms_cache_update(st.ctx, plan["budgets"], plan["theta"].astype(np.float32))
        slots = [int(sum(ms.ms_residency(st.ctx, l, E) > 0)) for l in range(L)]
        log("configurator: %d moves, theta %.3f..%.3f, C %d..%d" % (
            plan["iters"], plan["theta"].min(), plan["theta"].max(), min(slots), max(slots)))
    if policy != "static":
        ms.ms_set_cache_policy(st.ctx, {"lcp": ms.MS_CACHE_LCP, "lru": ms.MS_CACHE_LRU, "lfu": ms.MS_CACHE_LFU,
                                        "rnd": ms.MS_CACHE_RND}[policy])
    stream = torch.cuda.current_stream()
    n_slots = int(st.rig.sizes.buffer_bytes // st.rig.sizes.expert_bytes)
    out = {"metric": "MoE-stack decode µs/layer", "unit": "us/layer", "higher_is_better": False,
           "data": "synthetic", "dtype": "bf16", "n_gpus": 1,
           "config": {"workload": "%s: %s, %d layers, V_e %.0f GiB, r %s, C_i %s, %s decode batch %d, "
                                  "staging buffer %d whole-expert slots (K for the running layer's misses, "
                                  "K for the next layer's prefetch), cache policy %s" % (
               name, shape.name, L, cfg["budget"] / GIB,
               "from the configurator" if plan is not None else r, sorted(set(int(c) for c in slots)),
               ("prefill %d then" % P) if P else "", T, n_slots, policy)}}
    if plan is not None:
        out["plan"] = {"moves": plan["iters"], "theta": [round(float(t), 4) for t in plan["theta"]],
                       "cache": [int(c) for c in plan["cache"]],
                       "budget_mb": [round(int(b) / 1e6, 1) for b in plan["budgets"]],
                       "exposed_us_model": round(float(plan["exposed_us"].sum()), 1)}
    if P:
        h, _ = st.rig.hidden(P, tag=11)
        ms.ms_reset_stats(st.ctx)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        st.step(h, P)
        ms.ms_sync(st.ctx)
        torch.cuda.synchronize()
        out["prefill_ms"] = round((time.perf_counter() - t0) * 1e3, 2)
        out["prefill_tokens_per_s"] = round(P / (time.perf_counter() - t0), 1)
        log("prefill %d tokens: %.1f ms" % (P, out["prefill_ms"]))
    for x, _ in xs[n_warm:n_warm + warmup]:
        st.step(x, T)
    ms.ms_sync(st.ctx)
    torch.cuda.synchronize()
    ms.ms_reset_stats(st.ctx)
    step_ms = []
    t0 = time.perf_counter()
    for x, _ in xs[n_warm + warmup:]:
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        st.step(x, T)
        e1.record(stream)
        step_ms.append((e0, e1))
    ms.ms_sync(st.ctx)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per = [a.elapsed_time(b) for a, b in step_ms]
    stats = st.stats()
    tot = {k: sum(s_[k] for s_ in stats) for k in stats[0]}
    out.update({
        "value": round(wall / n_steps / L * 1e6, 1), "steps": n_steps, "warmup": warmup,
        "ms_per_step": round(wall / n_steps * 1e3, 3),
        "step_ms": {q: round(float(np.percentile(per, p_)), 3) for q, p_ in (("p10", 10), ("p50", 50), ("p90", 90))},
        "tokens_per_s": round(T * n_steps / wall, 2),
        "selected": tot["selected"], "alpha_beta_gamma": [tot["alpha"], tot["beta"], tot["gamma"]],
        "hit_rate": round((tot["alpha"] + tot["beta"]) / max(tot["experts_active"], 1), 4),
        "cache_inserts": tot["cache_inserts"],
        "buffer_hits": tot["buffer_hits"], "predicted_hits_per_layer_step": round(
            tot["predicted_hits"] / max(tot["predictions"], 1), 3),
        "h2d_bytes_per_step": {"miss": tot["bytes_miss"] // n_steps, "prefetch": tot["bytes_prefetch"] // n_steps,
                               "prefetch_used": tot["bytes_prefetch_used"] // n_steps,
                               "prefetch_dropped_before_issue": tot["bytes_prefetch_dropped"] // n_steps},
        "h2d_gbps_over_step": round((tot["bytes_miss"] + tot["bytes_prefetch"]) / wall / 1e9, 2),
    })
    if instrument_steps > 0:
        n_i = min(instrument_steps, n_steps)
        ms.ms_timeline_begin(st.ctx, stream, min(1 << 16, n_i * L * 64))
        torch.cuda.synchronize()
        ti = time.perf_counter()
        for x, _ in xs[n_warm + warmup:n_warm + warmup + n_i]:
            st.step(x, T)
        ms.ms_sync(st.ctx)
        torch.cuda.synchronize()
        wi = time.perf_counter() - ti
        tl = ms.ms_timeline_end(st.ctx)
        an = analyse(tl, n_i, wi * 1e3 / n_i, router_starts=False)
        out["overlap"] = {"steps": n_i, "h2d_hidden_frac": an["hidden_frac"],
                          "compute_hidden_frac": an["compute_hidden_frac"], "eta": an["overlap_eta"],
                          "copy_ms_per_step": round(an["copy_ms"] / n_i, 3),
                          "kernel_ms_per_step": round(an["kernel_ms"] / n_i, 3),
                          "h2d_gbps_during_copies": None if an["h2d_gbps"] is None else round(an["h2d_gbps"], 2)}
        out["copy_roofline"] = copy_roofline(tl)
        out["ffn_roofline"] = ffn_roofline(an)
    out["setup_s"] = round(time.perf_counter() - t_setup, 1)
    st.close()
    return out


def run_stack(args):
    out = measure_stack(args.workload, args.steps, args.warmup, args.copy_engine, args.policy, args.configure,
                        args.zeta, instrument_steps=min(args.steps, 32))
    out["platform"] = platform_info()
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=32)
    ap.add_argument("--warmup", type=int, default=4)
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-all-resident", action="store_true")
    ap.add_argument("--no-stack", action="store_true", help="skip the 32-layer stack of the default workload")
    ap.add_argument("--timeline-out", default=None)
    ap.add_argument("--workload", default="mixtral-decode",
                    help="mixtral-decode (default), deepseek-decode, deepseek-prefill, "
                         "qwen-decode16, qwen-prefill, mixtral-q2-decode; stacks: mixtral-stack, mixtral-stack-mixed, mixtral-q2-stack, "
                         "mixtral-decoder, mixtral-q2-decoder, "
                         "deepseek-stack, qwen-stack")
    ap.add_argument("--pmc-pass", action="store_true",
                    help="only the split pass, with the counter calibration copy before its timed steps "
                         "(run under rocprofv3 --pmc)")
    ap.add_argument("--pmc-summary", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="summarise two --pmc-pass runs (FETCH_SIZE, WRITE_SIZE) into --out")
    ap.add_argument("--pass-log", default=None, help="--pmc-summary: the JSON line a --pmc-pass run printed")
    ap.add_argument("--all-resident-pass", action="store_true",
                    help="--pmc-pass / --pmc-summary: the all-resident variant (r = 1, every expert cached)")
    ap.add_argument("--trace-summary", metavar="DIR", help="summarise a --kernel-trace --stats run into --out")
    ap.add_argument("--mfma-pmc-summary", metavar="DIR",
                    help="summarise a --pmc SQ_VALU_MFMA_BUSY_CYCLES GRBM_GUI_ACTIVE run into --out")
    ap.add_argument("--r", type=float, default=None,
                    help="split ratio instead of the workload's (the cache keeps the same number of tops)")
    ap.add_argument("--all-tops", action="store_true",
                    help="cache the top segment of every expert (the budget grows with it)")
    ap.add_argument("--policy", default="static", choices=["static", "lcp", "lru", "lfu", "rnd"],
                    help="stacks: online cache replacement on misses")
    ap.add_argument("--configure", action="store_true",
                    help="stacks: per-layer budgets and split ratios from the cache configurator")
    ap.add_argument("--zeta", type=float, default=0.01)
    ap.add_argument("--ffn-splits", type=int, default=0, help="work-groups per chunk (0: the library's choice)")
    ap.add_argument("--copy-engine", default="kernel", choices=["kernel", "dma"],
                    help="host-to-device copies: the copy kernel (default) or the DMA engines where possible")
    ap.add_argument("--out", default=None)
    ap.add_argument("--cmd", nargs="*", default=[], help="the profiling command(s), recorded in the summary")
    args = ap.parse_args()
    if args.pmc_summary:
        name = args.workload + ("-resident" if args.all_resident_pass else "")
        pmc_summary(args.pmc_summary[0], args.pmc_summary[1], name,
                    args.out or pmc_profile_path(name), *(args.cmd + ["", ""])[:2], pass_log=args.pass_log)
        return
    if args.trace_summary:
        trace_summary(args.trace_summary, args.out, " ".join(args.cmd))
        return
    if args.mfma_pmc_summary:
        mfma_pmc_summary(args.mfma_pmc_summary, args.workload, args.out, " ".join(args.cmd))
        return
    if args.gpus != 1:
        print("bench.py measures one GPU: the split-expert layer library has no "
              "multi-GPU path; run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    import synth
    from paper_2509_08342_amd import moesplit as ms
    from workload import SplitRig, to_device, top_bytes

    torch.cuda.set_device(0)
    if args.workload in _stacks():
        run_stack(args)
        return
    if args.workload in _decoders():
        run_decoder(args)
        return
    wl = _workloads()[args.workload]
    shape, T = wl["shape"], wl["T"]
    headline = args.workload == "mixtral-decode"
    t_setup = time.perf_counter()
    log("generating %s weights and filling the pinned store" % shape.name)
    rig = SplitRig(shape, seed=0, max_tokens=T, budget_bytes=shape.n_experts * shape.expert_bytes,
                   keep_f32=not args.no_cpu_baseline, threads=16, ffn_splits=args.ffn_splits,
                   n_buffer_slots=wl["slots"])
    if args.copy_engine == "dma":
        ms.ms_set_copy_engine(rig.ctx, ms.MS_COPY_DMA)
    n_tok = args.warmup + args.steps
    # independent N(0, 1) token batches, one per step
    seq = [synth.hidden(shape, 0, T, tag=1000 + i) for i in range(n_tok)]
    hs = [to_device(raw, shape.dtype) for raw, _ in seq]
    torch.cuda.synchronize()
    setup_s = time.perf_counter() - t_setup
    log("setup done in %.1f s; timing the split layer" % setup_s)
    # the split configuration: per-layer budget, split ratio, cached tops
    r = wl["r"] if args.r is None else args.r
    tops = [int(e) for e in wl["tops"](rig)]
    budget = wl["budget"](top_bytes(rig, r))
    if args.all_tops:
        tops = list(range(shape.n_experts))
        budget = shape.n_experts * top_bytes(rig, r)
    if args.all_resident_pass:
        r, tops, budget = 1.0, list(range(shape.n_experts)), shape.n_experts * shape.expert_bytes
    slots = rig.configure([budget], [r])
    rig.load_tops(0, tops[:int(slots[0])])
    ms.ms_sync(rig.ctx)
    flags = ms.MS_FWD_PREDICT_NEXT
    if args.pmc_pass:
        def calibrate():
            a = torch.empty(CALIB_BYTES, dtype=torch.uint8, device="cuda")
            b = torch.empty_like(a)
            b.copy_(a)
            torch.cuda.synchronize()
        # the timeline's events do not change the kernels; they give the
        # algorithmic bytes of the very dispatches the counters see
        ms_p, tl_p, _ = run_steps(rig, hs, args.steps, args.warmup, flags, timeline=True, cold=True, T=T,
                                  before_timed=calibrate)
        an_p = analyse(tl_p, args.steps, ms_p)
        ks = [an_p["kernels"][k] for k in ("ffn_resident", "ffn_streamed", "ffn_down")]
        rig.close()
        print(json.dumps({"pmc_pass": args.workload, "ms_per_step": round(ms_p, 4), "steps": args.steps,
                          "calib_bytes": CALIB_BYTES, "ffn_launches": sum(k["launches"] for k in ks),
                          "ffn_algorithmic_bytes": sum(k["bytes"] for k in ks)}), flush=True)
        return
    n_slots = int(rig.sizes.buffer_bytes // rig.sizes.expert_bytes)
    tb = top_bytes(rig, r)
    # the value: the layer's steady state in a deep stack -- the staging
    # buffer holds none of its segments when a token's routing arrives
    per = []
    ms_plain, _, st = run_steps(rig, hs, args.steps, args.warmup, flags, timeline=False, cold=True, T=T,
                                per_step=per)
    # the same steps with the library's timeline on: breakdown, overlap, roofline
    ms_step, tl, st_i = run_steps(rig, hs, args.steps, args.warmup, flags, timeline=True, cold=True, T=T)
    an = analyse(tl, args.steps, ms_step)
    roof = ffn_roofline(an)
    if roof is not None:
        tr = traffic_from_profile(args.workload)
        roof["traffic"] = None if tr is None else tr[0]
        roof["traffic_algorithmic_bytes"] = None if tr is None else tr[1]
        roof["traffic_ratio"] = None if tr is None else round(tr[0] / tr[1], 4)
        roof["by_launch"] = {k: ({"launches": v["launches"], "avg_us": round(v["total_ms"] / v["launches"] * 1e3, 2),
                                  "bytes_per_launch": int(v["bytes"] / v["launches"]),
                                  "gbps": round(v["bytes"] / (v["total_ms"] * 1e-3) / 1e9, 1)}
                                 if v["launches"] else None)
                             for k, v in an["kernels"].items() if k.startswith("ffn")}
    if args.timeline_out:
        with open(args.timeline_out, "w") as f:
            json.dump(dict(split=tl), f)
    sem = float(np.std(per, ddof=1) / np.sqrt(len(per))) if len(per) > 1 else None
    vram = {"top_segments_cached": int(slots[0]), "top_bytes_each": int(tb),
            "staging_slots": n_slots, "staging_bytes": int(rig.sizes.buffer_bytes)}
    out = {
        "metric": METRIC,
        # the pass without timeline events; the instrumented pass gives the breakdown
        "value": round(ms_plain * 1e3, 1),
        "unit": "us/layer",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_plain, 4),
        "ms_per_step_instrumented": round(ms_step, 4),
        "value_sem_us": None if sem is None else round(sem * 1e3, 1),
        "step_us": {q: round(float(np.percentile(per, p_)) * 1e3, 1) for q, p_ in (("p10", 10), ("p50", 50),
                                                                                   ("p90", 90))},
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "%s: %s-shaped MoE layer, %s batch of %d independent N(0,1) token(s) per step, "
                               "r=%.2f; in VRAM: the top segments of %d experts (%.1f MB each) and a staging "
                               "buffer of %d whole-expert slots that holds none of this layer's segments when a "
                               "step's routing arrives (a layer of a deep stack: the other layers' misses cycle "
                               "the buffer between two visits); the bottoms of the cached experts and the other "
                               "experts whole in pinned host RAM, copied after routing; next-layer prediction "
                               "and prefetch pass on" % (
                                   args.workload, shape.name, "prefill" if T > 16 else "decode", T, r,
                                   int(slots[0]), tb / 1e6, n_slots),
                   "d_model": shape.d_model, "d_ff": shape.d_ff, "n_experts": shape.n_experts,
                   "top_k": shape.top_k, "n_shared": shape.n_shared, "r": r, "tokens_per_step": T,
                   "n_buffer_slots": n_slots, "buffer_at_routing": "empty", "vram": vram,
                   "expert_bits": shape.expert_bits or None},
        "roofline": roof,
        # prefill: matrix-core utilisation of the FFN kernels (None at decode)
        "mfma": mfma_roofline(an, shape, T, args.steps),
        # the layer as a whole is bound by the link its missing segments cross
        "copy_roofline": copy_roofline(tl),
        "tokens_per_s": round(T * 1e3 / ms_plain, 2),
        "h2d_gbps": None if an["h2d_gbps"] is None else round(an["h2d_gbps"], 2),
        "overlap": {"h2d_hidden_frac": an["hidden_frac"], "compute_hidden_frac": an["compute_hidden_frac"],
                    "eta": an["overlap_eta"], "copy_ms_per_step": an["copy_ms"] / args.steps,
                    "kernel_ms_per_step": an["kernel_ms"] / args.steps},
        "h2d_bytes_per_step": {"miss": an["miss_bytes"] // args.steps,
                               "prefetch": an["prefetch_bytes"] // args.steps},
        "stats": st,
        "kernels": {k: {"launches": v["launches"], "avg_us": round(v["total_ms"] / v["launches"] * 1e3, 2)
                        if v["launches"] else None} for k, v in an["kernels"].items()},
        "setup_s": round(setup_s, 1),
    }
    out["h2d_link_peak_gbps"] = round(h2d_link_peak_gbps(), 2)
    log("split layer: %.3f ms/step (instrumented %.3f)" % (ms_plain, ms_step))

    # the hit path: every missing segment staged before routing
    hit, hit_experts = run_hit_path(rig, hs[args.warmup:], args.steps, T=T)
    if hit is None:
        out["hit_path"] = {"us_per_layer": None,
                           "what": "not defined here: a batch misses more experts than the staging buffer's "
                                   "%d slots hold" % n_slots}
        log("hit path: not defined (a batch misses more experts than the buffer holds)")
    else:
        out["hit_path"] = {"us_per_layer": round(float(np.mean(hit)) * 1e3, 1),
                           "step_us": {q: round(float(np.percentile(hit, p_)) * 1e3, 1)
                                       for q, p_ in (("p10", 10), ("p50", 50), ("p90", 90))},
                           "buffer_hits": int(hit_experts),
                           "what": "same tokens; each token's missing segments staged by an untimed forward just "
                                   "before, so the timed forward copies nothing (a right prediction whose "
                                   "prefetch landed in time)"}
        log("hit path: %.3f ms/step" % float(np.mean(hit)))
    if not args.no_all_resident:
        # all experts whole in VRAM (r = 1): the expert read is HBM-bound
        rig.configure([shape.n_experts * shape.expert_bytes], [1.0])
        rig.load_tops(0, range(shape.n_experts))
        ms.ms_sync(rig.ctx)
        ms_ar, tl_ar, _ = run_steps(rig, hs, args.steps, args.warmup, flags, T=T)
        ms_ar_plain, _, _ = run_steps(rig, hs, args.steps, args.warmup, flags, timeline=False, T=T)
        an_ar = analyse(tl_ar, args.steps, ms_ar)
        out["all_resident"] = {"us_per_layer": round(ms_ar_plain * 1e3, 1),
                               "us_per_layer_instrumented": round(ms_ar * 1e3, 1), "roofline": ffn_roofline(an_ar),
                               "mfma": mfma_roofline(an_ar, shape, T, args.steps),
                               "kernels": {k: {"launches": v["launches"],
                                               "avg_us": round(v["total_ms"] / v["launches"] * 1e3, 2)
                                               if v["launches"] else None}
                                           for k, v in an_ar["kernels"].items()}}
        tr = traffic_from_profile(args.workload + "-resident")
        if tr is not None and out["all_resident"]["roofline"] is not None:
            out["all_resident"]["roofline"].update(traffic=tr[0], traffic_algorithmic_bytes=tr[1],
                                                   traffic_ratio=round(tr[0] / tr[1], 4))
        log("all-resident variant: %.3f ms/step" % ms_ar_plain)
    if not args.no_cpu_baseline:
        log("timing the CPU oracle")
        out["cpu_baseline"] = cpu_baseline(rig, [f for _, f in seq], args.cpu_seconds)
    rig.close()
    if headline and not args.no_stack:
        # the Mixtral-shaped 32-layer stack at 12 GiB, r = .5: where
        # cross-layer prediction and prefetch move bytes
        log("Mixtral 32-layer stack")
        stk = measure_stack("mixtral-stack", args.steps, args.warmup, args.copy_engine,
                            instrument_steps=min(args.steps, 32))
        out["stack"] = {k: stk.get(k) for k in (
            "config", "value", "unit", "steps", "warmup", "ms_per_step", "step_ms", "tokens_per_s",
            "alpha_beta_gamma", "hit_rate", "buffer_hits", "predicted_hits_per_layer_step", "h2d_bytes_per_step",
            "h2d_gbps_over_step", "overlap", "copy_roofline", "ffn_roofline", "setup_s")}
    out["platform"] = platform_info()
    print(json.dumps(out), flush=True)

if __name__ == "__main__":
    main()
