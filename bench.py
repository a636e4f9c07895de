"""Benchmark: prefix-cached paged attention on one MI355X.

A step is one pass of the whole hot path over one batch of the workload:
prefix-hit lookup and block allocation for the batch (host C++), metadata and
launch plan (host C++), their asynchronous upload, the K/V append of the new
tokens and the attention launch (HIP), then the batch's release/rollback.
Default workload: suffix prefill of 64 requests against a cached 2048-token
prefix at the Llama-3-8B attention shape (the TFLOP/s headline).  Other
workloads: --workload decode|verify|mixed|tiny.

Prints one JSON line.  ``value`` is the step throughput (prefill and mixed:
attention TFLOP/s; decode and verify: algorithmic HBM GB/s of the step);
``roofline`` is the attention launch alone, timed with HIP events on the
stream it runs on; ``cpu_baseline`` is the float64 oracle on a bounded sample
of the same launch, on this host's cores.  A default (prefill) run then
measures the other configurations the same way, each with its own warm-up,
timed steps and short oracle sample, under ``workloads`` (decode and verify
against HBM bandwidth, mixed against bf16 MFMA, tiny float32 against the
vector ALU).
"""
from __future__ import annotations

import argparse
import gc
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "prefix-cached paged attn: prefill TFLOP/s, decode HBM GB/s, % of peak"
DESCRIPTIONS = {
    "prefill": "suffix prefill: 64 requests sharing one cached 2048-token prefix, suffix "
               "U[256,1024], causal within the suffix; 32 q / 8 kv heads, head_dim 128, "
               "block 16, bf16 (Llama-3-8B attention shape)",
    "decode": "decode: 256 sequences, context 2048 shared + U[256,1024] + U[1,128], 1 query "
              "each; 32/8 heads, d128, bf16",
    "mixed": "mixed launch: 512 requests over 4 cached prefixes 1k/2k/4k/8k (Zipf 1.1), "
             "64 x 512-token prefill chunks + 448 decode tokens; 28/4 heads, d128, bf16",
    "verify": "speculative verify: 32 requests, 16384 shared prefix + 4096 cached suffix, "
              "5 causal query tokens; 64/8 heads, d128, bf16 (Llama-3-70B attention shape)",
    "tiny": "tiny fp32: 4 requests, 128-token shared prefix, suffix U[32,64]; 8/2 heads, d64",
}


# HBM traffic of one attention call (attention kernel + split merge), from
# rocprofv3 FETCH_SIZE / WRITE_SIZE counter runs scaled by the factors a plain
# copy of known size gives; valid only for the kernel sources it was taken on.
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic.json")
KERNEL_SOURCES = ["attn_bf16.hip", "attn_f32.hip", "device_common.h", "plan.cpp",
                  "plan_format.h", "api.hip"]


def kernel_fingerprint() -> str:
    """sha256 of the kernel and planner sources without comments and blank
    lines (a comment edit does not change the kernels)."""
    import re
    h = hashlib.sha256()
    for s in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2605_11232_amd", "csrc", s)) as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        text = re.sub(r"//[^\n]*", "", text)
        h.update("\n".join(ln.rstrip() for ln in text.splitlines() if ln.strip()).encode())
    return h.hexdigest()


def cpu_model() -> str:
    """The host CPU's model name (as /proc/cpuinfo gives it)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown CPU"


def measured_traffic(name: str):
    """Counter-measured HBM bytes per call for this workload, or None when no
    record exists or the kernels changed since it was taken."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("kernel_sources_sha256") != kernel_fingerprint():
        return None
    w = rec.get("workloads", {}).get(name)
    return None if w is None else float(w["traffic_bytes"])


def cpu_baseline(wl, launch, budget_s: float = 12.0):
    """Time the float64 oracle on the first requests of the launch until the
    budget is spent; report its throughput in the metric's unit."""
    from oracle.run import OracleReplay
    from oracle.attention import gather_sequence, sequence_attention
    from paper_2605_11232_amd import perf
    orc = OracleReplay(wl).setup()
    res = orc.launch(launch, attend=False)
    md = res["meta"]
    q = launch.q.get()
    cu, L = md["cu_seqlens_q"], md["seq_lens"]
    cfg = wl.cfg
    scale = cfg.head_dim ** -0.5
    t0 = time.perf_counter()
    done = 0
    flops = 0.0
    for r in range(len(L)):
        a, b = int(cu[r]), int(cu[r + 1])
        if a == b:
            continue
        K, V = gather_sequence(orc.k_cache, orc.v_cache, md["block_table"][r], int(L[r]))
        sequence_attention(q[a:b].astype(np.float64), K, V, scale)
        flops += perf.attention_flops([L[r]], [0, b - a], cfg.num_q_heads, cfg.head_dim)
        done += 1
        if time.perf_counter() - t0 > budget_s:
            break
    dt = time.perf_counter() - t0
    sub = {"block_table": md["block_table"][:done], "seq_lens": md["seq_lens"][:done],
           "cu_seqlens_q": md["cu_seqlens_q"][:done + 1]}
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = len(os.sched_getaffinity(0))
    return dt, done, flops, threads, sub


def run_workload(name, W, K, C, cpu_budget, profile=False, settle_ms=0.0):
    """Settle the device clock (untimed steps for settle_ms of device load),
    warm up W steps, time K steps (HIP events around every attention call),
    then C cold-cache steps; returns the figures of one workload."""
    import torch
    from paper_2605_11232_amd import binding as B, perf, synth
    from paper_2605_11232_amd.runtime import DeviceReplay, Staging, plan_words_bound, marshal_launch

    wl = synth.workload(name, steps=W + K + C + 2)
    cfg = wl.cfg
    dev = DeviceReplay(wl).setup()
    # one launch more than the steps: the host side of the step after the
    # timed ones runs inside the timed region (see there)
    launches = [wl.step(s) if wl.step else wl.launches[0] for s in range(W + K + C + 1)]
    # pack each step's token batches (input marshalling) before timing
    for ln in launches:
        marshal_launch(ln)
    L0 = launches[0]
    T = L0.total_q
    tdt = dev.tdtype
    q = torch.from_numpy(L0.q.get()).to("cuda", tdt)
    k_new = torch.from_numpy(L0.k_new.get()).to("cuda", tdt)
    v_new = torch.from_numpy(L0.v_new.get()).to("cuda", tdt)
    out = torch.empty((T, cfg.num_q_heads, cfg.head_dim), dtype=tdt, device="cuda")
    lse = torch.empty((T, cfg.num_q_heads), dtype=torch.float32, device="cuda")
    n = len(L0.seq_ids)
    plan_words = plan_words_bound(cfg, n, T, wl.max_blocks_per_seq)
    stagings = [Staging("cuda", n, wl.max_blocks_per_seq, T, plan_words) for _ in range(2)]
    stream = torch.cuda.current_stream()

    kv_memory = {}
    state = {"scrub": None}
    scrub_sink = []

    def host(s, record=None):
        # the host side of step s: pool operations, metadata and plan into
        # its pinned staging buffer
        share = record is not None and state["scrub"] is None
        return dev.prepare_staged(launches[s], stagings[s % 2], q, k_new, v_new, out, lse,
                                  guard=record[0] if share else None, upload=False)

    def step(s, record=None, p=None):
        # A timed step's attention call carries its start and stop events on
        # its first and last kernel dispatches (no event packets between the
        # kernels); in a warm-cache step the start event also releases the
        # staging buffer, so the step records no event of its own.  p: its
        # host side, when that already ran.
        if p is None:
            p = host(s, record)
        dev.upload(p)
        if s == 0 and record is None:
            # KV memory of the live batch: blocks versus contiguous reservations
            # of the block-table capacity (outside the timed steps)
            kv_memory.update(dev.pool.kv_waste(wl.max_blocks_per_seq * cfg.block_size))
        dev.append(p, record_guard=False)
        if state["scrub"] is not None:
            # read 1 GiB: L2 and MALL then hold none of the inputs (a read leaves
            # no dirty lines whose write-back would compete with the call)
            scrub_sink.append(state["scrub"].sum())
        dev.attend(p, events=record)
        dev.finish(launches[s], batched=True)
        return p

    events = [(B.StreamEvent(timing=True), B.StreamEvent(timing=True)) for _ in range(K)]
    # no garbage-collector pass inside the timed steps: a full collection of
    # the interpreter's objects takes milliseconds, several steps' worth.
    # Collect before the warm-up, not between it and the timed steps: after
    # an idle pause of that length the device's power management repeats its
    # start-up transient (a fast call, then 10-20 calls 5-30 % slower), so
    # the timed steps would not start from the state the warm-up reached.
    gc.collect()
    gc.freeze()
    gc.disable()
    # The device has idled through the host-side setup (and, for the later
    # configurations of a full run, through the previous one's oracle timing).
    # Under load after idle its power management runs a transient (a fast
    # call, then 10-20 calls 5-30 % slower) before the clock settles, so a
    # short warm-up would leave the timed steps inside it.  One step, then its
    # attention call again and again (same inputs, output overwritten; paced
    # by events so at most 2 * SETTLE_BATCH calls are queued and the host
    # mostly waits) keep the device loaded for settle_ms first (at least
    # SETTLE_MIN_CALLS calls); the W warm-up and K timed steps follow without
    # a pause, whatever W is.
    n_settle = 0
    settle_s = 0.0
    if settle_ms > 0:
        p0 = step(0)
        t_s = time.perf_counter()
        pace = []
        while n_settle < SETTLE_MIN_CALLS or settle_s * 1e3 < settle_ms:
            for _ in range(SETTLE_BATCH):
                dev.attend(p0)
            n_settle += SETTLE_BATCH
            ev = B.StreamEvent()
            ev.record(stream)
            pace.append(ev)
            if len(pace) > 2:
                pace.pop(0).synchronize()
            settle_s = time.perf_counter() - t_s
    for s in range(W):
        p = step(s)
    # The host side of each step overlaps the device work of the step before
    # (the pinned staging buffers alternate).  The barrier before the timed
    # steps drains that pipeline, so the first timed step's host side runs
    # before it, as it would have during the step before, and the host side
    # of the step after the timed ones runs inside the timed region, as it
    # would during the last one (its pool operations are rolled back after
    # the region): the region holds exactly K steps of host work and K of
    # device work, as a K-step stretch of the running pipeline does.
    p = host(W, events[0]) if K else None
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(K):
        p = step(W + i, events[i], p)
        p_next = host(W + i + 1, events[i + 1] if i + 1 < K else None)
        if i + 1 < K:
            p = p_next
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    if K:
        dev.finish(launches[W + K], batched=True)  # the prepared, never-run step
    gc.enable()
    gc.unfreeze()
    meta = {k: np.array(v, copy=True) for k, v in p.meta.items()}
    per_ms = [a.elapsed_time(b) for a, b in events]
    attn_ms = float(np.mean(per_ms))
    cold_ms = None
    if C:
        # cold caches: the same call after a 1 GiB read, outside the timed steps
        state["scrub"] = torch.ones(1 << 28, dtype=torch.int32, device="cuda")
        cev = [(B.StreamEvent(timing=True), B.StreamEvent(timing=True)) for _ in range(C)]
        for i in range(C):
            step(W + K + i, cev[i])
        torch.cuda.synchronize()
        cold_ms = float(np.mean([a.elapsed_time(b) for a, b in cev]))
        state["scrub"] = None

    flops = perf.attention_flops(meta["seq_lens"], meta["cu_seqlens_q"], cfg.num_q_heads,
                                 cfg.head_dim)
    attn_bytes = perf.attention_bytes(meta, cfg, unique=True)
    logical_bytes = perf.attention_bytes(meta, cfg, unique=False)
    app_bytes = perf.append_bytes(T, cfg)
    ms = wall / K * 1e3
    compute_bound = name in ("prefill", "mixed")
    if cfg.dtype == "f32":
        peak, unit, bound = perf.MI355X_PEAKS["fp32_vector_tflops"], "TFLOP/s", "alu"
        work, scale_u = flops, 1e12
        value = flops / (ms * 1e-3) / 1e12
    elif compute_bound:
        peak, unit, bound = perf.MI355X_PEAKS["bf16_tflops"], "TFLOP/s", "mfma"
        work, scale_u = flops, 1e12
        value = flops / (ms * 1e-3) / 1e12
    else:
        peak, unit, bound = perf.MI355X_PEAKS["hbm_gbs"], "GB/s", "hbm"
        work, scale_u = attn_bytes, 1e9
        value = (attn_bytes + app_bytes) / (ms * 1e-3) / 1e9
    achieved = work / (attn_ms * 1e-3) / scale_u
    # the timed calls as three consecutive runs: each run's mean call time,
    # and the median and range of the three (the paper's protocol reports
    # the median and range of three runs)
    runs = [float(np.mean(c)) for c in np.array_split(np.asarray(per_ms), 3) if len(c)]
    res = {
        "name": name, "cfg": cfg, "requests": len(L0.seq_ids), "query_tokens": T,
        "flops": flops, "attn_bytes": attn_bytes, "logical_bytes": logical_bytes,
        "app_bytes": app_bytes, "ms": ms, "value": value, "unit": unit, "bound": bound,
        "peak": peak, "achieved": achieved, "attn_ms": attn_ms, "per_ms": per_ms, "runs": runs,
        "run_achieved": [work / (r * 1e-3) / scale_u for r in runs], "kv_memory": kv_memory,
        "W": W, "K": K,
        "settle": {"attention_calls": n_settle, "ms": round(settle_s * 1e3, 1)},
    }
    if cold_ms is not None:
        cold_ach = work / (cold_ms * 1e-3) / scale_u
        res["cold"] = {"steps": C, "avg_launch_ms": round(cold_ms, 4),
                       "achieved": round(cold_ach, 2), "unit": unit,
                       "frac": round(cold_ach / peak, 4),
                       "note": "attention call after a 1 GiB device read (L2 and MALL "
                               "flushed); not part of value or roofline"}
    del dev, stagings, q, k_new, v_new, out, lse
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    if cpu_budget > 0 and not profile:
        dt, done, cflops, threads, sub = cpu_baseline(synth.workload(name, steps=2), L0,
                                                      budget_s=cpu_budget)
        if compute_bound or cfg.dtype == "f32":
            cval, cunit = cflops / dt / 1e12, "TFLOP/s"
        else:
            cval = perf.attention_bytes(sub, cfg, unique=True) / dt / 1e9
            cunit = "GB/s"
        res["cpu_baseline"] = {"value": cval, "unit": cunit, "cores": threads, "kind": "oracle",
                               "sample": f"float64 oracle attention of the first {done} of "
                                         f"{len(L0.seq_ids)} requests of the same launch "
                                         f"(all heads), {dt:.1f} s on {cpu_model()}"}
    return res


def measured_ceilings():
    """What the device's own libraries reach in this process, as context for
    the roofline fractions: a bf16 GEMM (torch.matmul, 16384^3), a read of 1 GiB
    (float32 row sums of a [65536, 4096] array, the fastest of torch's
    reductions on this device) and a 1 GiB device-to-device copy (bytes read +
    written), each timed with HIP events after a warm-up."""
    import torch
    from paper_2605_11232_amd import binding as B

    def timed(fn, reps):
        fn()
        torch.cuda.synchronize()
        a, b = B.StreamEvent(timing=True), B.StreamEvent(timing=True)
        stream = torch.cuda.current_stream()
        a.record(stream)
        for _ in range(reps):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e-3 / reps

    n = 16384
    g = torch.Generator(device="cuda").manual_seed(0)
    x = torch.randn(n, n, device="cuda", generator=g).to(torch.bfloat16)
    y = torch.randn(n, n, device="cuda", generator=g).to(torch.bfloat16)
    gemm_s = timed(lambda: torch.matmul(x, y), 5)
    del x, y
    src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")  # 1 GiB
    dst = torch.empty_like(src)
    rows = src.view(1 << 16, -1)
    read_s = timed(lambda: rows.sum(dim=1), 5)
    copy_s = timed(lambda: dst.copy_(src), 5)
    nbytes = src.numel() * 4
    del src, dst, rows
    torch.cuda.empty_cache()
    return {"bf16_gemm_tflops": round(2 * n ** 3 / gemm_s / 1e12, 1),
            "hbm_read_gbs": round(nbytes / read_s / 1e9, 1),
            "hbm_copy_gbs": round(2 * nbytes / copy_s / 1e9, 1),
            "note": "torch.matmul bf16 16384^3, float32 row sums over 1 GiB, 1 GiB device "
                    "copy (read + write bytes), timed in this run; context for the roofline "
                    "fractions, which use the published peaks"}


def add_measured_fraction(summary, ceilings):
    """The roofline object's achieved figure against the measured ceiling of
    its bound (bf16 GEMM for MFMA-bound calls, the 1 GiB read for HBM-bound)."""
    key = {"mfma": "bf16_gemm_tflops", "hbm": "hbm_read_gbs"}.get(summary["bound"])
    if key:
        summary["frac_of_measured_ceiling"] = round(summary["achieved"] / ceilings[key], 4)
        summary["measured_ceiling"] = key


def call_summary(res):
    """Attention-call figures of one workload (the roofline object's body)."""
    per = np.asarray(res["per_ms"])
    runs = res["runs"]
    ra = res["run_achieved"]
    return {"bound": res["bound"], "achieved": round(res["achieved"], 2), "peak": res["peak"],
            "unit": res["unit"], "frac": round(res["achieved"] / res["peak"], 4),
            "traffic": measured_traffic(res["name"]),
            "traffic_unit": "HBM bytes per call (counters)",
            "kernel": "pa_attn_" + ("prefill" if res["name"] in ("prefill", "mixed", "tiny")
                                    else res["name"]),
            "avg_launch_ms": round(res["attn_ms"], 4),
            "launch_ms_median": round(float(np.median(per)), 4),
            "launch_ms_min": round(float(np.min(per)), 4),
            "launch_ms_max": round(float(np.max(per)), 4),
            "runs_ms": [round(r, 4) for r in runs],
            "runs_achieved_median": round(float(np.median(ra)), 2),
            "runs_achieved_range": [round(float(min(ra)), 2), round(float(max(ra)), 2)],
            "effective_logical_gbs": round(res["logical_bytes"] / (res["attn_ms"] * 1e-3) / 1e9, 1)}


# The other configurations, measured in the same run after the headline.
SECONDARY = ["decode", "verify", "mixed", "tiny"]
SETTLE_MIN_CALLS = 24
SETTLE_BATCH = 8


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=30,
                    help="untimed steps first; the device clock settles over ~20 calls")
    ap.add_argument("--workload", default="prefill", choices=list(DESCRIPTIONS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-secondary", action="store_true",
                    help="measure only --workload (by default a prefill run also measures "
                         "the decode, verify, mixed and tiny configurations)")
    ap.add_argument("--secondary-steps", type=int, default=40,
                    help="timed steps of each secondary configuration")
    ap.add_argument("--secondary-warmup", type=int, default=25)
    ap.add_argument("--secondary-cpu-budget", type=float, default=3.0,
                    help="seconds of float64 oracle per secondary configuration")
    ap.add_argument("--profile-steps", type=int, default=0,
                    help="run only this many steps without the CPU baseline (profiling)")
    ap.add_argument("--settle-ms", type=float, default=200.0,
                    help="before the warm-up, one step and then its attention call repeated "
                         "until the device has been under load this long (at least 24 calls), "
                         "so the timed steps start in the clock's steady state after the idle "
                         "setup; 0 skips it")
    ap.add_argument("--cold-steps", type=int, default=5,
                    help="extra steps, after the timed ones, whose attention call runs after a "
                         "1 GiB device read has flushed the caches (0 skips them)")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="only run a plain device-to-device copy of this many MiB, 5 times "
                         "(calibrates the HBM byte counters against a known transfer)")
    ap.add_argument("--matmul-n", type=int, default=0,
                    help="only run a bf16 [n, n] x [n, n] torch.matmul 5 times (calibrates the "
                         "MFMA operation counters against a known FLOP count)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the hot path here is a single-GPU kernel "
              f"library; --gpus {args.gpus} is not supported (see DESIGN.md for how the "
              f"path would shard).", file=sys.stderr)
        sys.exit(2)

    import torch
    if args.copy_mib:
        n = args.copy_mib << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": n, "launches": 5}), flush=True)
        return
    if args.matmul_n:
        n = args.matmul_n
        g = torch.Generator(device="cuda").manual_seed(0)
        x = torch.randn(n, n, device="cuda", generator=g).to(torch.bfloat16).contiguous()
        y = torch.randn(n, n, device="cuda", generator=g).to(torch.bfloat16).contiguous()
        for _ in range(5):
            z = torch.matmul(x, y)
        torch.cuda.synchronize()
        print(json.dumps({"matmul_n": n, "flop_per_launch": 2 * n ** 3, "launches": 5,
                          "checksum": float(z.float().abs().mean())}), flush=True)
        return

    torch.cuda.set_device(0)
    name = args.workload
    W, K = args.warmup, args.steps
    C = 0 if args.profile_steps else max(0, args.cold_steps)
    if args.profile_steps:
        W, K = 1, args.profile_steps
    profile = bool(args.profile_steps)
    budget = 0.0 if args.no_cpu_baseline else 10.0
    settle = 0.0 if profile else max(0.0, args.settle_ms)
    res = run_workload(name, W, K, C, budget, profile, settle)
    cfg = res["cfg"]
    rec = {
        "metric": METRIC,
        "value": round(res["value"], 3),
        "unit": res["unit"],
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "settle": res["settle"],
        "ms_per_step": round(res["ms"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {"workload": DESCRIPTIONS[name], "name": name,
                   "requests": res["requests"], "query_tokens": res["query_tokens"],
                   "attn_flops": res["flops"], "attn_unique_bytes": res["attn_bytes"],
                   "attn_logical_bytes": res["logical_bytes"], "append_bytes": res["app_bytes"],
                   "parallelism": "single GPU"},
        "kv_memory": {k: (round(v, 4) if isinstance(v, float) else v)
                      for k, v in res["kv_memory"].items()},
        "roofline": call_summary(res),
    }
    if "cold" in res:
        rec["cold_caches"] = res["cold"]
    if "cpu_baseline" in res:
        rec["cpu_baseline"] = res["cpu_baseline"]
    if name == "prefill" and not args.no_secondary and not profile:
        # every other configuration, each its own warm-up and timed steps;
        # its figures are per attention call, like the roofline object
        wls = {}
        for other in SECONDARY:
            print(f"[bench] {other}", file=sys.stderr, flush=True)
            r2 = run_workload(other, args.secondary_warmup, args.secondary_steps, 0,
                              0.0 if args.no_cpu_baseline else args.secondary_cpu_budget,
                              settle_ms=settle)
            w = {"workload": DESCRIPTIONS[other], "dtype": r2["cfg"].dtype,
                 "requests": r2["requests"], "query_tokens": r2["query_tokens"],
                 "attn_flops": r2["flops"], "attn_unique_bytes": r2["attn_bytes"],
                 "steps": r2["K"], "warmup": r2["W"], "settle": r2["settle"],
                 "ms_per_step": round(r2["ms"], 4),
                 "step_value": round(r2["value"], 3), "step_unit": r2["unit"],
                 "roofline": call_summary(r2)}
            if "cpu_baseline" in r2:
                w["cpu_baseline"] = r2["cpu_baseline"]
            wls[other] = w
        rec["workloads"] = wls
    if name == "prefill" and not args.no_secondary and not profile:
        # the full run only (profiling runs keep their traces to the hot path),
        # after every timed step, so the extra work cannot disturb them
        ceil = measured_ceilings()
        rec["measured_ceilings"] = ceil
        add_measured_fraction(rec["roofline"], ceil)
        for w in rec.get("workloads", {}).values():
            add_measured_fraction(w["roofline"], ceil)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
