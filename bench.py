#!/usr/bin/env python3
"""Decode-step throughput of the MiKV mixed-precision KV cache on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

A step is one pass of the whole decode hot path over the batch: append the
new token (quantize), attention over both precision pools with probability
emission, importance update (fused into attention by default; --fused 0
runs it as its own kernel), top-k re-rank with demotion/requantization.
Inputs are synthetic, seeded, drawn directly in device memory, and resident
before the timed region starts.  Prints ONE JSON line on stdout:

  value      effective GB/s = packed K/V bytes the steps read (codes + fp16
             scale/zero + fp16 values, both pools) / wall time of the K steps;
  roofline   the attention partial kernel (the dominant one): its algorithmic
             bytes per launch (the packed K/V bytes) / its mean duration from
             HIP events recorded on its stream, against 8 TB/s;
  cpu_baseline  the CPU oracle timed on a bounded sample of the same workload;
  secondary  the same fields for a second workload (default llama2_13b, the
             largest cache by bytes) timed in the same run;
  mall       untimed diagnostic: event-bracketed whole steps with warm caches,
             with the 256 MB last-level cache flushed before each step, and
             flushed with every row streamed (resident share 0: what a
             model whose layers share that cache would see);
  read_ceiling  the read bandwidth of a plain streaming kernel over 1 GiB
             (mikv_stream_read_probe, non-temporal loads): what HBM gives a
             plain kernel here; roofline.read_ceiling_same_bytes is the same
             probe over the step's own byte count, with the attention's
             split of plain (resident) and non-temporal (streamed) loads and
             passes alternating in direction as the steps do, and
             roofline.frac_of_read_ceiling the attention kernel's achieved /
             that (the practical ceiling).

Only one GPU is used; --gpus above 1 exits with an error.
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

HBM_PEAK_GBPS = 8000.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def track_counts(dec, n_hi, length):
    """Importance-pool size after one more step (append, then re-rank): the
    window is always high precision, eligible tokens beyond k_heavy demote."""
    L = length + 1
    n_attn = n_hi + 1
    elig = n_attn - min(dec.wl.window, L)
    n_new = n_attn - max(0, elig - dec.k_heavy(L))
    return L, n_attn, n_new


def cpu_baseline(wl, steps_inputs, budget_s: float):
    """The oracle, as it is, on a bounded sample: up to eight (sequence, KV
    head) pairs of batch element 0, decode steps from the end of prefill
    until the time budget is used -- once with the BLAS threads the process
    has, then, from a copy of the same prefilled cache, on one thread (half
    the budget).  Both legs start at the first decode step, so each times
    the same work per step; a leg that completes no step is an error."""
    import copy

    import numpy as np

    import oracle
    from paper_2402_18096_amd import workloads
    from threadpoolctl import threadpool_info, threadpool_limits

    q, kn, vn = steps_inputs
    heads = list(range(0, wl.kv_heads, max(1, wl.kv_heads // 8)))[:8]
    G, T = wl.group_size, wl.context
    k, v = workloads.prefill_kv(wl, q.device, batches=range(1))
    sc = workloads.initial_scores(wl, "cpu")[0].numpy()
    f16 = lambda t: t.detach().cpu().contiguous().numpy().view(np.float16)
    kk, vv = f16(k[0])[heads], f16(v[0])[heads]
    del k, v
    bal = None
    if wl.balanced:
        qp = f16(workloads.prefill_queries(wl, q.device, batches=range(1))[0])
        qp = qp.reshape(wl.kv_heads, G, T, 128)[heads]
        bal = oracle.balancer(qp, kk)
    n_steps = q.shape[0]
    orc0 = oracle.OracleCache(len(heads), G, T + n_steps, wl.hi_bits, wl.lo_bits, wl.group)
    orc0.prefill(kk, vv, sc[heads], oracle.heavy_budget(T, wl.ratio_num, wl.ratio_den, wl.window,
                                                        wl.window_in_ratio), wl.window, bal)
    qh = [h * G + i for h in heads for i in range(G)]
    tb = lambda bits: 0 if bits == 0 else 4 * 128 if bits == 16 else 2 * (128 * bits // 8 + 4 * (128 // wl.group))
    # decode inputs of the sampled heads, on the host before any timing
    qs = [f16(q[t, 0])[qh].reshape(len(heads), G, 128) for t in range(n_steps)]
    ks = [f16(kn[t, 0])[heads] for t in range(n_steps)]
    vs = [f16(vn[t, 0])[heads] for t in range(n_steps)]

    def run(orc, budget):
        done, nbytes, t0 = 0, 0, time.perf_counter()
        while done < n_steps and time.perf_counter() - t0 < budget:
            L = orc.length + 1
            n_hi = int(orc.is_hi[:, :L - 1].sum()) + len(heads)
            nbytes += n_hi * tb(wl.hi_bits) + (len(heads) * L - n_hi) * tb(wl.lo_bits)
            orc.step(qs[done], ks[done], vs[done], 1.0 / math.sqrt(128.0),
                     oracle.heavy_budget(L, wl.ratio_num, wl.ratio_den, wl.window, wl.window_in_ratio), wl.window,
                     bal)
            done += 1
        el = time.perf_counter() - t0
        if done == 0:
            raise RuntimeError(f"cpu baseline: no decode step completed within {budget:.1f} s")
        return done, nbytes, el

    orc1 = copy.deepcopy(orc0)
    done, nbytes, el = run(orc0, budget_s)
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    try:
        host_cpus = len(os.sched_getaffinity(0))
    except AttributeError:
        host_cpus = os.cpu_count() or 1
    with threadpool_limits(limits=1):
        done1, nbytes1, el1 = run(orc1, budget_s / 2)
    return {"value": round(nbytes / el / 1e9, 4), "unit": "GB/s", "cores": int(min(threads, host_cpus)),
            "kind": "oracle", "host_cpus": int(host_cpus), "host_cpu_count": os.cpu_count(),
            "sample": f"{len(heads)} of {wl.n_heads} (sequence, KV head) pairs x the first {done} decode steps "
                      f"({el:.1f} s); numpy oracle, BLAS threads = {threads}",
            "s_per_step_per_head": round(el / done / len(heads), 4),
            "single_thread": {"value": round(nbytes1 / el1 / 1e9, 4), "unit": "GB/s", "cores": 1,
                              "sample": f"the same pairs x the first {done1} decode steps ({el1:.1f} s), "
                                        "BLAS limited to one thread",
                              "s_per_step_per_head": round(el1 / done1 / len(heads), 4)}}


# The attention partial kernel's source files (its traffic record is keyed by them).
KERNEL_SOURCES = ("attention.hip", "mikv_internal.h", "append_device.h", "select_device.h")


def measured_traffic(workload: str):
    """HBM bytes per attention partial launch from the committed rocprofv3
    counter runs (FETCH_SIZE and WRITE_SIZE, each scaled by what the counter
    reads for a copy of known size), or None when there is no record for this
    workload or the kernel source has changed since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"attn_partial_{workload}_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2402_18096_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    if rec.get("source_sha256") != h.hexdigest():
        return None
    return rec


def copy_probe(mb: int):
    """Time a plain device-to-device copy of `mb` MB (read + write bytes):
    the reference for achievable HBM bandwidth and for scaling PMC counters."""
    import torch
    n = mb * (1 << 20)
    src = torch.empty(n, dtype=torch.uint8, device="cuda")
    src.fill_(1)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    reps = 20
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    x = src.view(torch.int32)
    for _ in range(3):
        x.sum(dtype=torch.int64)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(reps):
        x.sum(dtype=torch.int64)
    e1.record()
    torch.cuda.synchronize()
    ms_r = e0.elapsed_time(e1) / reps
    rec = {"copy_probe_MB": mb, "ms_per_copy": round(ms, 4), "copy_read_plus_write_GBps": round(2 * n / ms / 1e6, 1),
           "ms_per_sum": round(ms_r, 4), "sum_read_GBps": round(n / ms_r / 1e6, 1)}
    print(json.dumps(rec), flush=True)


def read_ceiling(mb: int, reps: int = 10, alternate: bool = False, resident: int = 0):
    """The library's streaming-read probe (16-byte loads, four in flight per
    thread, nothing else) over `mb` MiB, timed with HIP events on its stream:
    the read bandwidth a plain kernel reaches on this device, the practical
    ceiling of the HBM-bound kernels next to the 8 TB/s data-sheet peak.
    The leading `resident` bytes are read with plain loads, the rest
    non-temporally.  With `alternate` consecutive passes run in opposite
    directions, as the decode steps do."""
    import torch

    from paper_2402_18096_amd import mikv
    n = mb * (1 << 20)
    buf = torch.empty(n, dtype=torch.uint8, device="cuda")
    buf.fill_(1)
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    for i in range(3):
        mikv.mikv_stream_read_probe(buf, sink, resident, alternate and i % 2 == 1)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(reps):
        mikv.mikv_stream_read_probe(buf, sink, resident, alternate and i % 2 == 0)
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) / reps * 1e3
    del buf
    torch.cuda.empty_cache()
    return {"kernel": "stream_read_kernel (mikv_stream_read_probe)", "bytes": n, "launches": reps,
            "directions": "alternating" if alternate else "front to back", "resident_bytes": min(resident, n),
            "mean_launch_us": round(us, 2), "GBps": round(n / us / 1e3, 1)}


MFMA_FP16_PEAK_TFLOPS = 2500.0  # dense fp16 matrix-core peak of one MI355X


def prefill_importance_probe(workload: str, reps: int):
    """Time mikv_prefill_importance on the workload's prompt (its seeded fp16
    queries and keys): the H2O importance of every prompt token.  Algorithmic
    FLOPs are those of one causal Q K^T (2 * 128 per query-key pair with
    key <= query, every query head); the kernel computes the logits twice
    (statistics pass, then column-sum pass)."""
    import torch

    from paper_2402_18096_amd import mikv, workloads
    wl = workloads.WORKLOADS[workload]
    dev = torch.device("cuda:0")
    k, v = workloads.prefill_kv(wl, dev)
    del v
    q = workloads.prefill_queries(wl, dev)
    scores = torch.empty(wl.batch, wl.kv_heads, wl.context, dtype=torch.float32, device=dev)
    ws = torch.empty(mikv.lib().mikv_prefill_importance_workspace_size(wl.batch, wl.q_heads, wl.context),
                     dtype=torch.uint8, device=dev)
    scale = 1.0 / math.sqrt(wl.head_dim)
    mikv.mikv_prefill_importance(q, k, scores, scale, ws)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        mikv.mikv_prefill_importance(q, k, scores, scale, ws)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    T = wl.context
    flops = 2.0 * wl.head_dim * (T * (T + 1) / 2) * wl.batch * wl.q_heads
    tflops = flops / (ms * 1e-3) / 1e12
    mass = float(scores.double().sum()) / (wl.batch * wl.q_heads * T)
    rec = {"prefill_importance": {"workload": wl.name, "batch": wl.batch, "q_heads": wl.q_heads,
                                  "kv_heads": wl.kv_heads, "tokens": T, "ms": round(ms, 3),
                                  "algorithmic_tflop": round(flops / 1e12, 3), "achieved_tflops": round(tflops, 1),
                                  "peak_tflops": MFMA_FP16_PEAK_TFLOPS, "frac": round(tflops / MFMA_FP16_PEAK_TFLOPS, 4),
                                  "mass_per_query": round(mass, 6), "reps": reps,
                                  "note": "the kernel evaluates the logits twice (statistics, then column sums)"}}
    print(json.dumps(rec), flush=True)


def apply_overrides(wl, overrides):
    for ov in overrides:
        key, val = ov.split("=", 1)
        cur = getattr(wl, key)
        wl = wl.with_(**{key: type(cur)(val) if not isinstance(cur, bool) else val in ("1", "true", "True")})
    return wl


def run_workload(wl, args, steps: int, warmup: int, cpu_seconds: float, overridden: bool):
    """Prefill, warm up, time `steps` whole decode steps, then the untimed
    diagnostic passes and the CPU baseline.  Returns the record's fields."""
    import torch

    from paper_2402_18096_amd import mikv, workloads

    dev = torch.device("cuda:0")
    n_total = warmup + steps + args.phase_steps + 3 * args.mall_steps
    t_setup = time.perf_counter()
    dec = mikv.MikvDecoder(wl, max_len=wl.context + n_total, device=dev, fused=bool(args.fused))
    k, v = workloads.prefill_kv(wl, dev)
    sc = workloads.initial_scores(wl, dev)
    qp = workloads.prefill_queries(wl, dev) if wl.balanced else None
    steps_inputs = workloads.decode_inputs(wl, n_total, dev)
    q, kn, vn = steps_inputs
    dec.prefill(k, v, sc, qp)
    del k, v, qp
    torch.cuda.synchronize()
    log(f"[bench] {wl.name}: prefill of {wl.context} tokens x {wl.n_heads} heads done "
        f"({time.perf_counter() - t_setup:.1f} s); warmup {warmup}, timed {steps}")

    for t in range(warmup):
        dec.step_native(q[t], kn[t], vn[t])
    torch.cuda.synchronize()

    n_hi = int(dec.cache.n_hi[0].item())
    length = dec.length
    step_bytes = []
    for _ in range(steps):
        length, n_attn, n_hi = track_counts(dec, n_hi, length)
        step_bytes.append(dec.cache.packed_bytes(length, n_attn))

    def fresh_events(n):
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(n)]
        for e in evs:
            e.record()
        return evs

    # Timed steps: two events per step around the attention partial kernel
    # (recorded on the stream it runs on), nothing else.
    every = max(1, args.event_every)
    sampled = [i for i in range(steps) if i % every == 0] if args.events == "partial" else []
    part_ev = {i: fresh_events(2) for i in sampled}
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        t = warmup + i
        ev = [None, part_ev[i][0], part_ev[i][1], None, None, None] if i in part_ev else None
        dec.step_native(q[t], kn[t], vn[t], phase_events=ev)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0

    nh_dev = dec.cache.n_hi.cpu()
    status = int(dec.cache.status.item())
    if status != 0 or not bool((nh_dev == n_hi).all()):
        log(f"[bench] ERROR: device status {status}, n_hi {nh_dev[:4].tolist()} vs tracked {n_hi}")
        sys.exit(1)

    # Diagnostics, untimed: an event at every phase boundary (each event adds
    # a little time of its own to the phase it closes).
    phases = ["append", "attn_partial", "attn_finalize", "importance", "select"]
    ph_ev = [fresh_events(6) for _ in range(args.phase_steps)]
    torch.cuda.synchronize()
    for i in range(args.phase_steps):
        t = warmup + steps + i
        dec.step_native(q[t], kn[t], vn[t], phase_events=ph_ev[i])
    torch.cuda.synchronize()
    mean = lambda xs: sum(xs) / len(xs) if xs else float("nan")
    dur = {p: [ph_ev[i][j].elapsed_time(ph_ev[i][j + 1]) for i in range(args.phase_steps)]
           for j, p in enumerate(phases)}

    # Diagnostics, untimed: whole steps bracketed by events, warm, then cold
    # (the last-level cache and L2 flushed by reading 1 GiB before each
    # step, outside the bracket; a read leaves no dirty lines behind), then
    # cold with nothing read plainly (mikv_set_resident_bytes(0): every row
    # streamed, the setting for a model whose layers share that cache).
    mall = None
    if args.mall_steps > 0:
        flush = torch.zeros(1 << 28, dtype=torch.float32, device=dev)
        mb, ln, nh = [], dec.length, int(dec.cache.n_hi[0].item())
        for _ in range(3 * args.mall_steps):
            ln, n_attn, nh = track_counts(dec, nh, ln)
            mb.append(dec.cache.packed_bytes(ln, n_attn))
        res = {}
        base = warmup + steps + args.phase_steps
        resident = mikv.mikv_resident_bytes()
        for j, kind in enumerate(("warm", "cold", "cold_streamed")):
            evs = [fresh_events(2) for _ in range(args.mall_steps)]
            if kind == "cold_streamed":
                mikv.mikv_set_resident_bytes(0)
            torch.cuda.synchronize()
            for i in range(args.mall_steps):
                t = base + j * args.mall_steps + i
                if kind != "warm":
                    flush.sum()  # reads only: no dirty lines left to write back
                evs[i][0].record()
                dec.step_native(q[t], kn[t], vn[t])
                evs[i][1].record()
            torch.cuda.synchronize()
            mikv.mikv_set_resident_bytes(resident)
            us = sorted(e[0].elapsed_time(e[1]) * 1e3 for e in evs)
            nb = mb[j * args.mall_steps:(j + 1) * args.mall_steps]
            res[kind] = {"step_us_median": round(us[len(us) // 2], 2), "step_us_mean": round(sum(us) / len(us), 2),
                         "effective_GBps_median": round(sum(nb) / len(nb) / (us[len(us) // 2] * 1e-6) / 1e9, 1)}
        del flush
        mall = {**res, "steps_each": args.mall_steps, "flush": "1 GiB fp32 read (sum) before each cold step",
                "cold_streamed": res["cold_streamed"] | {"resident_bytes": 0},
                "note": "each step bracketed by two events on the stream (adds about empty_event_bracket_us)"}
        log(f"[bench] {wl.name} whole step (event-bracketed): warm median {res['warm']['step_us_median']} us, "
            f"cold median {res['cold']['step_us_median']} us, cold with every row streamed "
            f"{res['cold_streamed']['step_us_median']} us")

    total_bytes = sum(step_bytes)
    value = total_bytes / elapsed / 1e9
    ms = elapsed / steps * 1e3
    mean_bytes = total_bytes / steps
    roofline = None
    if part_ev:
        part_ms = [part_ev[i][0].elapsed_time(part_ev[i][1]) for i in sampled]
        # per-launch algorithmic bytes / per-launch duration over the sampled
        # launches (each counts with its own step's bytes)
        achieved = sum(step_bytes[i] for i in sampled) / (sum(part_ms) * 1e-3) / 1e9
        # An empty event bracket (the kernel-free "importance" phase of the
        # fused step, measured in the diagnostic pass) shows the time the two
        # events add to a bracketed launch.
        overhead_ms = mean(dur["importance"]) if args.fused else float("nan")
        tr = measured_traffic(wl.name) if not overridden else None
        roofline = {"kernel": "attn_partial_kernel", "bound": "hbm", "achieved": round(achieved, 2),
                    "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                    "traffic": tr["read_bytes"] + tr["write_bytes"] if tr else None,
                    "traffic_unit": "HBM bytes per launch (read + write, rocprofv3 FETCH_SIZE/WRITE_SIZE, "
                                    "copy-calibrated)",
                    "mean_launch_us": round(mean(part_ms) * 1e3, 2),
                    "launches_timed": len(part_ms), "launch_timing": f"HIP events on every {every}-th timed step",
                    "empty_event_bracket_us": round(overhead_ms * 1e3, 2) if overhead_ms == overhead_ms else None,
                    "algorithmic_bytes_per_launch": int(mean_bytes)}
        if tr:
            roofline["traffic_read_bytes"] = tr["read_bytes"]
            roofline["traffic_write_bytes"] = tr["write_bytes"]
    log(f"[bench] {wl.name}: {steps} steps in {elapsed * 1e3:.2f} ms: {ms * 1e3:.1f} us/step, "
        f"{value:.1f} GB/s effective ({100 * value / HBM_PEAK_GBPS:.1f} % of peak)")
    if roofline:
        log(f"[bench] {wl.name} attn_partial: {roofline['mean_launch_us']} us/launch, {roofline['achieved']} GB/s")
    log(f"[bench] {wl.name} phase means (us, diagnostic pass): " +
        ", ".join(f"{p} {mean(dur[p]) * 1e3:.1f}" for p in phases))
    del dec
    torch.cuda.empty_cache()
    if roofline and args.read_probe_mb > 0:
        # the probe over as many bytes as the step reads, re-read the same
        # way: back to back, in alternating directions, the attention's
        # resident share with plain loads and the rest non-temporally (so the
        # last-level cache serves the same share of them)
        from paper_2402_18096_amd import mikv
        ceil_w = read_ceiling(max(1, math.ceil(mean_bytes / (1 << 20))), alternate=True,
                              resident=mikv.mikv_resident_bytes())
        roofline["read_ceiling_same_bytes"] = ceil_w
        roofline["frac_of_read_ceiling"] = round(roofline["achieved"] / ceil_w["GBps"], 4)
        log(f"[bench] {wl.name} streaming-read probe over the same bytes: {ceil_w['GBps']} GB/s; attn_partial at "
            f"{100 * roofline['frac_of_read_ceiling']:.1f} % of it")

    cpu = None
    if cpu_seconds > 0:
        cpu = cpu_baseline(wl, (q, kn, vn), cpu_seconds)
        log(f"[bench] {wl.name} cpu oracle: {cpu['value']} GB/s ({cpu['sample']}); one thread "
            f"{cpu['single_thread']['value']} GB/s ({cpu['single_thread']['sample']})")
    del q, kn, vn, steps_inputs
    torch.cuda.empty_cache()
    return {
        "value": round(value, 2),
        "ms_per_step": round(ms, 5),
        "config": {"workload": wl.name, "batch": wl.batch, "q_heads": wl.q_heads, "kv_heads": wl.kv_heads,
                   "head_dim": wl.head_dim, "context": wl.context, "hi_bits": wl.hi_bits, "lo_bits": wl.lo_bits,
                   "group": wl.group, "ratio": f"{wl.ratio_num}/{wl.ratio_den}", "window": wl.window,
                   "balanced": wl.balanced, "importance_fused": bool(args.fused),
                   "parallelism": "single GPU"},
        "pct_of_hbm_peak": round(100 * value / HBM_PEAK_GBPS, 2),
        "steps_per_s": round(1e3 / ms, 1),
        "packed_bytes_per_step": int(mean_bytes),
        "phase_us": {p: round(mean(dur[p]) * 1e3, 2) for p in phases} if args.phase_steps > 0 else None,
        "roofline": roofline,
        "mall": mall,
        "cpu_baseline": cpu,
    }


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=256)
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--workload", default="long_context")
    ap.add_argument("--secondary", default="llama2_13b",
                    help="a second workload timed in the same run and reported under `secondary` ('none' for none); "
                         "it runs min(--steps, its own step count) timed steps")
    ap.add_argument("--fused", type=int, default=1, help="fuse the importance update into attention (default 1)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="time budget of the CPU oracle baseline (all threads; one thread gets half)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--override", action="append", default=[], metavar="FIELD=VALUE",
                    help="change a workload field, e.g. ratio_num=0 (experiments; reported in config)")
    ap.add_argument("--phase-steps", type=int, default=16,
                    help="untimed steps after the timed ones that record an event at every phase boundary")
    ap.add_argument("--events", choices=["partial", "none"], default="partial",
                    help="events inside the timed steps: around the attention partial kernel (default; gives "
                         "the roofline), or none (wall time only)")
    ap.add_argument("--event-every", type=int, default=7, metavar="K",
                    help="bracket the attention partial kernel with events on every K-th timed step (each event "
                         "costs a few microseconds of GPU time; default 7: odd, so the sampled steps alternate "
                         "between the two grid orders that consecutive steps use)")
    ap.add_argument("--mall-steps", type=int, default=16,
                    help="untimed steps after the phase pass, each bracketed by two events: this many with the "
                         "caches as the previous step left them (warm), then this many each preceded by a "
                         "1 GiB read that evicts the 256 MB last-level cache (cold)")
    ap.add_argument("--prefill-importance", action="store_true",
                    help="instead of the bench: time the prompt-importance kernel on the workload's prompt")
    ap.add_argument("--read-probe-mb", type=int, default=1024, metavar="MB",
                    help="size of the streaming-read probe run before the workloads (the measured read "
                         "ceiling reported next to the data-sheet peak; 0 skips it)")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MB",
                    help="instead of the bench: time a plain device-to-device copy of MB megabytes")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py runs on exactly one GPU (asked for --gpus {args.gpus}, WORLD_SIZE {world}); "
              "this build measures one GPU's share and has no multi-GPU path.", file=sys.stderr)
        sys.exit(2)

    from paper_2402_18096_amd import workloads

    if args.copy_probe:
        return copy_probe(args.copy_probe)
    if args.prefill_importance:
        return prefill_importance_probe(args.workload, max(1, args.steps if args.steps < 256 else 3))
    wl = apply_overrides(workloads.WORKLOADS[args.workload], args.override)
    cpu_s = 0.0 if args.no_cpu_baseline else args.cpu_seconds
    ceiling = read_ceiling(args.read_probe_mb) if args.read_probe_mb > 0 else None
    if ceiling:
        log(f"[bench] streaming-read probe: {ceiling['GBps']} GB/s over {args.read_probe_mb} MiB "
            f"({ceiling['mean_launch_us']} us/launch)")
    head = run_workload(wl, args, args.steps, args.warmup, cpu_s, bool(args.override))
    secondary = None
    if args.secondary and args.secondary not in ("none", args.workload):
        wl2 = apply_overrides(workloads.WORKLOADS[args.secondary], args.override)
        secondary = run_workload(wl2, args, min(args.steps, wl2.steps), args.warmup, cpu_s * 2 / 3,
                                 bool(args.override))
        secondary["steps"] = min(args.steps, wl2.steps)
        secondary["warmup"] = args.warmup
    rec = {
        "metric": "mixed-KV decode attention effective GB/s (% of HBM peak) + decode steps/s",
        "value": head["value"],
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        **{k: v for k, v in head.items() if k not in ("value", "ms_per_step")},
        "read_ceiling": ceiling,
        "secondary": secondary,
    }
    if args.override:
        rec["config"]["overrides"] = args.override
        if secondary:
            secondary["config"]["overrides"] = args.override
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
