#!/usr/bin/env python3
"""Benchmark of the EDiT outer synchronization step on one MI355X.

One step = one outer round over every sync unit of the workload (default:
Llama-1B-shaped, 24 units x 51,384,320 parameters, K = 8 bf16 replicas, fp32
theta and momentum), issued in forward order over HIP streams.  Between
steps (untimed) the seeded generator rewrites every replica as
cast(theta_t + s_j * N(0, 1e-3)), i.e. what K workers would hold after their
inner steps; the timed region is the outer step alone, with all inputs
resident in HBM.

Prints ONE JSON line: the metric, value (GB/s of algorithmic bytes), ms per step,
the dominant kernel's roofline and the oracle's CPU baseline.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0  # MI355X HBM3E, published
PEAK_HOST_LINK_GBPS = 64.0  # PCIe 5.0 x16 host interface, per direction, published
METRIC = "outer-sync ms/step and achieved HBM GB/s (% of peak), 1B model K=8"
DEFAULT_WORKLOAD = "llama1b-k8-bf16"  # 24 units x 51,384,320 elements, K = 8, bf16 replicas
WORKLOAD_NAMES = ("linear1m-k4", "llama350m-k8-f32", "llama1b-k8-bf16", "llama7b-half-k8-bf16",
                  "aedit1b-k16-bf16", "paper1b-k8-bf16")
CSRC = os.path.join(ROOT, "paper_2412_07210_amd", "csrc")
COUNTERS_FILE = os.path.join(ROOT, "profiles", "hbm_traffic_counters.json")


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_code_hash(text: str) -> str:
    """Hash of kernel source with comments and whitespace removed: the identity
    of the code the HBM counters were taken on (a comment edit keeps it)."""
    import re
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    text = " ".join(text.split())
    return hashlib.sha256(text.encode()).hexdigest()[:16]


def kernel_source_hash() -> str:
    """The kernels file and the code fragments it includes."""
    text = ""
    for name in ["edit_outer_kernels.hip"] + sorted(f for f in os.listdir(CSRC) if f.endswith(".inc")):
        with open(os.path.join(CSRC, name)) as f:
            text += f.read()
    return kernel_code_hash(text)


def unit_bytes(n: int, K: int, R: int, active: int, rolled_back: bool, one_pass: bool = False) -> tuple:
    """Algorithmic HBM bytes of one unit's step: (pass 1, pass 2).

    pass 1 reads theta (4 B) and the K replicas; pass 2 reads theta, b and the
    replicas of contributing workers, writes theta, b and all K replicas.  On
    a rollback pass 2 reads theta and writes the K replicas only.  The
    one-pass mean step reads theta, b and the K replicas and writes them all
    (reported as its first element, the second being 0).
    """
    if one_pass:
        return n * (16 + 2 * K * R), 0
    p1 = n * (4 + K * R)
    if rolled_back:
        p2 = n * (4 + K * R)
    else:
        p2 = n * (8 + active * R + 8 + K * R)
    return p1, p2


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch of `kernel` (pass2, fused) from committed rocprofv3
    counters, if they were taken on this workload and on the current kernel
    code; else None."""
    try:
        with open(COUNTERS_FILE) as f:
            data = json.load(f)
    except (OSError, ValueError):
        return None
    if data.get("kernel_source_sha256_16") != kernel_source_hash() or data.get("workload") != workload:
        return None
    try:
        return float(data[f"{kernel}_bytes_per_launch"])
    except (KeyError, TypeError, ValueError):
        return None


def _on_traffic(traffic, avg_ms):
    """GB/s of the counter-measured HBM bytes per launch over the event average."""
    return None if traffic is None else round(traffic / (avg_ms * 1e-3) / 1e9, 2)


def copy_probe_gbps(torch, outer, nbytes: int = 2 << 30, reps: int = 5) -> float:
    src = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    src.fill_(1.0)
    outer.copy_probe(dst, src)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        outer.copy_probe(dst, src)
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / reps
    del src, dst
    return 2 * nbytes / (ms * 1e-3) / 1e9


def host_link_probe_gbps(torch, nbytes: int = 1 << 30, reps: int = 3) -> dict:
    """Pinned host <-> device copy rates (GB/s) of plain torch copies, one
    direction at a time and both at once on two streams: the practical
    ceiling of the host-state round."""
    h = torch.empty(nbytes // 4, dtype=torch.float32, pin_memory=True)
    h2 = torch.empty_like(h, pin_memory=True)
    d = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda")
    d2 = torch.empty_like(d)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    out = {}
    for name, both in (("h2d", False), ("d2h", False), ("both_each_way", True)):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(reps):
            if name == "h2d" or both:
                with torch.cuda.stream(s1):
                    d.copy_(h, non_blocking=True)
            if name == "d2h" or both:
                with torch.cuda.stream(s2):
                    h2.copy_(d2, non_blocking=True)
        torch.cuda.synchronize()
        out[name] = round(nbytes * reps / (time.perf_counter() - t0) / 1e9, 2)
    del h, h2, d, d2
    return out


def update_probe(torch, lib, units, wl, reps: int, roofline: dict) -> dict:
    """Each unit's update-pass traffic with no arithmetic
    (edit_outer_update_probe: the update pass's grid and 16-byte loads and
    stores of theta, b and all K replicas, values written back unchanged),
    each launch timed with HIP events on the current stream, against the
    update pass's own sampled launches of the timed rounds."""
    K, R = wl.num_workers, wl.replica_bytes
    ve = 16 // R
    ms, nbytes = [], []
    for _ in range(reps):
        for u, (th, b, rp) in enumerate(units):
            a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            lib.update_probe(u, th, b, rp)
            z.record()
            torch.cuda.synchronize()
            ms.append(a.elapsed_time(z))
            nbytes.append((th.numel() // ve) * ve * (16 + 2 * K * R))
    avg = sum(ms) / len(ms)
    gbps = sum(nbytes) / len(nbytes) / (avg * 1e-3) / 1e9
    return {
        "kernel": "update_pattern_probe_kernel (the update pass's loads and stores, no arithmetic)",
        "avg_launch_ms": round(avg, 5), "gbps": round(gbps, 2), "frac": round(gbps / PEAK_HBM_GBPS, 4),
        "bytes_per_launch": int(sum(nbytes) / len(nbytes)), "launches": len(ms),
        "update_pass_avg_launch_ms": roofline["avg_launch_ms"],
        "update_pass_over_probe_time": round(roofline["avg_launch_ms"] / avg, 4),
    }


def host_cpu() -> dict:
    """The host's CPU model (as lscpu reports it) and the cores this process
    may run on."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"model": model, "affinity_cores": len(os.sched_getaffinity(0))}


def oracle_threads() -> int:
    """Threads for the CPU baseline: every core in the affinity mask, capped
    by OMP_NUM_THREADS when the environment sets it (the host's share)."""
    n = len(os.sched_getaffinity(0))
    cap = os.environ.get("OMP_NUM_THREADS", "")
    return max(1, min(n, int(cap))) if cap.isdigit() and int(cap) > 0 else max(1, n)


def cpu_baseline(samples, wl, one_pass: bool = False):
    """Time the CPU oracle (as it stands: one thread per unit step) on every
    unit of one captured round.  First one unit alone on one thread, then all
    units at once, one per thread on every core of the host's share (the
    units are independent; each unit's step is unchanged).  For the one-pass
    mode, the oracle with every penalty component off."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np
    from oracle import OracleConfig, OracleUnit

    K, R = wl.num_workers, wl.replica_bytes
    cfg = OracleConfig(**wl.hyper(), **({"flags": 0} if one_pass else {}))
    per_elt = (2 * K * R + 16) if one_pass else (3 * K * R + 20)
    total_bytes = sum(th.size for (_, th, _, _) in samples) * per_elt
    # one unit, one thread (on a copy: the all-core run below steps every unit in place)
    u0, th0, b0, reps0 = samples[0]
    t0 = time.perf_counter()
    OracleUnit(K, cfg).step(th0.copy(), b0.copy(), [r.copy() for r in reps0])
    one_s = time.perf_counter() - t0
    log(f"cpu oracle, one thread: unit {u0} in {one_s:.2f} s")
    threads = oracle_threads()

    def step(sample):
        _, th, b, reps = sample
        OracleUnit(K, cfg).step(th, b, reps)

    t0 = time.perf_counter()
    with ThreadPoolExecutor(threads) as pool:
        list(pool.map(step, samples))
    all_s = time.perf_counter() - t0
    log(f"cpu oracle, {threads} threads: {len(samples)} units in {all_s:.2f} s")
    n0 = samples[0][1].size
    return {
        "value": round(total_bytes / all_s / 1e9, 4),
        "unit": "GB/s",
        "cores": threads,
        "kind": "oracle",
        "ms_per_step": round(all_s * 1e3, 1),
        "one_thread_ms_per_unit": round(one_s * 1e3, 1),
        "one_thread_ms_per_step": round(one_s * 1e3 * len(samples), 1),
        "host_cpu": host_cpu(),
        "sample": f"all {len(samples)} units of one round ({n0:,} elements each, K={K}) stepped by the "
                  f"C oracle (fp64) one unit per thread on {threads} threads: ms_per_step and value are "
                  f"that run's wall time; one_thread_* is one unit alone on one thread (times "
                  f"{len(samples)} for a step)",
    }


# The other single-GPU workloads, measured after the headline in the same run
# (the 1024x1024 layer fits the Infinity Cache and is latency-bound: a parity
# case, not a bandwidth line).
SECONDARY = ("llama350m-k8-f32", "llama7b-half-k8-bf16", "aedit1b-k16-bf16")


def measure_secondary(torch, np, name: str, steps: int, warmup: int, seed: int, dev, profile_every: int = 12):
    """One workload's rounds through edit_outer_step_round, as the headline
    (fresh handle and inputs, cache settle before each round, HIP events on
    every `profile_every`-th unit): ms/step percentiles, GB/s of the design
    bytes and the sampled kernels' rooflines.  Frees everything it made."""
    from paper_2412_07210_amd import EditOuter, OuterConfig, outer, synth

    wl = synth.get(name)
    K, R = wl.num_workers, wl.replica_bytes
    hyper = wl.hyper()
    warm = hyper.pop("warmup_rounds")
    lib = EditOuter(OuterConfig(num_workers=K, layer_numel=wl.layer_numel, replica_dtype=wl.replica_dtype,
                                ema_warmup_rounds=warm, **hyper), dev)
    units = []
    for u in range(wl.num_units):
        th = wl.init_theta(u, dev, seed)
        units.append((th, torch.zeros_like(th), [torch.empty(th.numel(), dtype=wl.torch_dtype, device=dev)
                                                 for _ in range(K)]))
    plan = lib.prepare_round(units)
    lib.set_profiling(profile_every)
    settle_src = torch.zeros(256 << 20, dtype=torch.float32, device=dev)
    settle_dst = torch.empty_like(settle_src)
    step_ms, p1, p2 = [], [], []  # p1/p2: (ms, algorithmic bytes) of sampled launches
    step_bytes = min_bytes = 0
    masked = rollbacks = 0
    for t in range(warmup + steps):
        std = wl.worker_std(t, seed)
        for u, (th, _, reps) in enumerate(units):
            wl.fill_replicas(th, reps, u, t, seed, std=std)
        outer.copy_probe(settle_dst, settle_src)
        torch.cuda.synchronize()
        a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        plan.run()
        z.record()
        torch.cuda.synchronize()
        if t < warmup:
            continue
        step_ms.append(a.elapsed_time(z))
        for u, (th, _, _) in enumerate(units):
            st = lib.state_get(u)
            active = int(np.count_nonzero(st.weight > 0)) if st.clip_coef > 0 else 0
            b1, b2 = unit_bytes(th.numel(), K, R, active, st.rolled_back)
            step_bytes += b1 + b2
            min_bytes += th.numel() * (2 * K * R + 16)
            masked += int(st.anomalous.sum())
            rollbacks += int(st.rolled_back)
            if u % profile_every == 0:
                k1, k2 = lib.kernel_times(u)
                p1.append((k1, b1))
                p2.append((k2, b2))
    lib.close()
    del units, plan, settle_src, settle_dst
    torch.cuda.empty_cache()
    total_ms = sum(step_ms)
    q = np.percentile(step_ms, [10, 50, 90])
    value = step_bytes / (total_ms * 1e-3) / 1e9

    def roof(samples, kernel):
        ms = sum(m for m, _ in samples) / len(samples)
        achieved = sum(b for _, b in samples) / len(samples) / (ms * 1e-3) / 1e9
        return {"kernel": kernel, "bound": "hbm", "achieved": round(achieved, 2), "peak": PEAK_HBM_GBPS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBPS, 4), "avg_launch_ms": round(ms, 5),
                "sampled_launches": len(samples)}

    pass1_name = "pass1_gram_mfma_kernel" if K > 8 else "pass1_gram_kernel"
    out = {
        "workload": f"{wl.name}: {wl.description}", "units": wl.num_units, "num_workers": K,
        "replica_dtype": wl.replica_dtype, "steps": steps, "warmup": warmup,
        "ms_per_step": round(total_ms / len(step_ms), 4), "ms_p10": round(float(q[0]), 4),
        "ms_p50": round(float(q[1]), 4), "ms_p90": round(float(q[2]), 4),
        "value": round(value, 2), "unit": "GB/s", "pct_peak_hbm": round(100 * value / PEAK_HBM_GBPS, 2),
        "gbps_on_min_bytes": round(min_bytes / (total_ms * 1e-3) / 1e9, 2),
        "masked_workers_total": masked, "rollbacks_total": rollbacks,
        "pass1": roof(p1, pass1_name + " (its unit's Gram pass; in a round up to K = 8 it also "
                          "carries earlier units' decisions)"),
        "pass2": roof(p2, "pass2_update_kernel"),
    }
    # the dominant kernel by time: the update pass (twice pass 1's bytes)
    out["dominant"] = "pass2" if sum(m for m, _ in p2) >= sum(m for m, _ in p1) else "pass1"
    return out


# ----------------------------------------------------------------------------
# Summaries of rocprofv3 output (CPU only): --summarize-profiles
# ----------------------------------------------------------------------------

def _profile_cmds(variant: str) -> dict:
    """The rocprofv3 commands whose output summarize_profiles reads."""
    tag, flag = ("llama1b_onepass", " --one-pass") if variant == "one-pass" else ("llama1b", "")
    sfx = "_op" if variant == "one-pass" else ""
    return {
        "tag": tag, "suffix": sfx,
        "trace": f"rocprofv3 --kernel-trace --stats -f csv -d <out>/prof_trace{sfx} -o {tag} -- "
                 f"python bench.py{flag}",
        "fetch": f"rocprofv3 --pmc FETCH_SIZE -f csv -d <out>/prof_fetch{sfx} -o {tag} -- "
                 f"python bench.py --steps 2 --warmup 1 --no-cpu-baseline --profile-every 0 --secondary 0 "
                 f"--update-probe 0{flag}",
        "write": f"rocprofv3 --pmc WRITE_SIZE -f csv -d <out>/prof_write{sfx} -o {tag} -- "
                 f"python bench.py --steps 2 --warmup 1 --no-cpu-baseline --profile-every 0 --secondary 0 "
                 f"--update-probe 0{flag}",
    }


# The two-unit Gram launch and the one-unit launch that takes two earlier
# units' decisions are one kernel template (its last argument is the unit
# count); they are told apart here.
PAIR2, PAIR1 = "pass1_gram_pair_kernel<..., 2>", "pass1_gram_pair_kernel<..., 1>"
PASS1_KINDS = ("pass1_gram_kernel", "pass1_gram_mfma_kernel", PAIR2, PAIR1)
UNITS_PER_LAUNCH = {PAIR2: 2}

SHORT = {"pass1_gram_kernel": "pass1", PAIR2: "pass1_pair", PAIR1: "pass1_pair1", "decide_kernel": "decide",
         "pass2_update_kernel": "pass2", "fused_mean_kernel": "fused", "fused_finish_kernel": "finish",
         "update_pattern_probe_kernel": "probe"}


def _kernel_kind(name: str) -> str:
    m = re.search(r"pass1_gram_pair_kernel<[^>]*, (\d+)>", name)
    if m:
        return PAIR2 if m.group(1) == "2" else PAIR1
    for kind in ("pass1_gram_kernel", "pass1_gram_mfma_kernel", "decide_kernel", "pass2_update_kernel",
                 "round_small_kernel", "fused_mean_kernel", "fused_finish_kernel", "update_pattern_probe_kernel",
                 "copy_kernel"):
        if kind in name:
            return kind
    return ""


def summarize_trace_by_grid(out_dir: str, name: str) -> str:
    """Group a rocprofv3 kernel trace (`<out>/prof_trace_<name>/<name>_kernel_trace.csv`) by
    kernel and grid size, so units of different sizes in one workload get rows of their own.
    Streams the CSV (it is large); returns the markdown table written to profiles/."""
    import csv
    from paper_2412_07210_amd import synth

    wl = synth.get(name)
    tag = name.replace("-", "_")  # file-name form of the workload name
    K, R = wl.num_workers, wl.replica_bytes
    sizes = sorted(set(wl.layer_numel))
    groups, regs = {}, {}
    spans = []  # (start, end, kind) of every dispatch, for the gaps between kernels
    with open(os.path.join(out_dir, f"prof_trace_{tag}", f"{tag}_kernel_trace.csv")) as f:
        for row in csv.DictReader(f):
            kind = _kernel_kind(row["Kernel_Name"])
            spans.append((int(row["Start_Timestamp"]), int(row["End_Timestamp"]), kind))
            if not kind or kind == "copy_kernel":
                continue
            grid = int(row.get("Grid_Size") or row.get("Grid_Size_X"))
            dur = int(row["End_Timestamp"]) - int(row["Start_Timestamp"])
            groups.setdefault((kind, grid), []).append(dur)
            regs[kind] = (row.get("VGPR_Count", "?"), row.get("Accum_VGPR_Count", "?"),
                          row.get("LDS_Block_Size", "?"))

    ve = 8 if wl.replica_dtype == "bf16" else 4  # elements per 16-byte replica vector

    def unit_of(kind, grid):
        for n in sizes:
            nvec = -(-n // ve)
            if kind in ("pass2_update_kernel", "update_pattern_probe_kernel") and -(-nvec // 64) * 64 == grid:
                return n
            tpb = 768 if kind == "pass1_gram_mfma_kernel" else 256  # threads per Gram-pass block
            if kind in PASS1_KINDS and -(-nvec // 256) >= grid // tpb - 1:
                return n
        return None

    # a two-unit launch counts two units of the size its grid matches (the
    # workloads that pair units have units of one size)
    def algo(kind, n):
        if kind in PASS1_KINDS:
            return UNITS_PER_LAUNCH.get(kind, 1) * n * (4 + K * R)
        if kind == "update_pattern_probe_kernel":  # every replica, whole vectors only
            return (n // (16 // R)) * (16 // R) * (16 + 2 * K * R)
        return n * (16 + 2 * K * R) if kind == "pass2_update_kernel" else None
    lines = [f"# Kernel durations by unit size: {wl.description}", "",
             "Command (from the repository root; `<out>` = the directory the profiler wrote to):", "",
             f"    rocprofv3 --kernel-trace --stats -f csv -d <out>/prof_trace_{tag} -o {tag} -- "
             f"python bench.py --config {name} --steps 10 --warmup 5 --no-cpu-baseline --secondary 0", "",
             f"Summarised with `python bench.py --summarize-trace <out> {name}` (groups the trace's "
             "dispatches by kernel and grid size).", "",
             "| kernel | grid work-items | unit elements | calls | avg us | min us | max us | "
             "algorithmic bytes | GB/s at avg |", "|---|---|---|---|---|---|---|---|---|"]
    for (kind, grid) in sorted(groups, key=lambda kg: (kg[0], -kg[1])):
        d = groups[(kind, grid)]
        avg = sum(d) / len(d)
        n = unit_of(kind, grid)
        b = algo(kind, n) if n else None
        gbps = f"{b / (avg * 1e-9) / 1e9:.1f}" if b else "-"
        lines.append(f"| {kind} | {grid} | {n if n else '-'} | {len(d)} | {avg / 1e3:.1f} | "
                     f"{min(d) / 1e3:.1f} | {max(d) / 1e3:.1f} | {b if b else '-'} | {gbps} |")
    # idle time between consecutive dispatches that are both steps of the
    # method (the stream's dependency latency; torch and copy kernels excluded)
    spans.sort()
    ours = {*PASS1_KINDS, "decide_kernel", "pass2_update_kernel", "round_small_kernel", "fused_mean_kernel",
            "fused_finish_kernel"}
    pairs = [(a[2], b[2], b[0] - a[1]) for a, b in zip(spans, spans[1:]) if a[2] in ours and b[2] in ours]
    gaps = sorted(g for _, _, g in pairs)
    if gaps:
        med = gaps[len(gaps) // 2]
        lines += ["", f"Gap between consecutive dispatches of the method's kernels (end of one to start "
                  f"of the next, same stream): median {med / 1e3:.2f} us, 10th percentile "
                  f"{gaps[len(gaps) // 10] / 1e3:.2f} us, 90th {gaps[9 * len(gaps) // 10] / 1e3:.2f} us "
                  f"over {len(gaps)} pairs.", "", "| from | to | pairs | median gap us | 90th us |",
                  "|---|---|---|---|---|"]
        for a, b in sorted({(a, b) for a, b, _ in pairs}):
            g = sorted(x for pa, pb, x in pairs if (pa, pb) == (a, b))
            lines.append(f"| {a} | {b} | {len(g)} | {g[len(g) // 2] / 1e3:.2f} | {g[9 * len(g) // 10] / 1e3:.2f} |")
    lines += ["", "The trace's VGPR_Count, Accum_VGPR_Count and LDS bytes per block (VGPR_Count reads "
              "half the compiler's per-lane VGPR figure on this ROCm, e.g. 60 for a 119-VGPR kernel):", ""]
    for kind, (v, a, l) in sorted(regs.items()):
        lines.append(f"- {kind}: VGPR_Count {v}, Accum_VGPR_Count {a}, {l} B LDS")
    text = "\n".join(lines) + "\n"
    os.makedirs(os.path.join(ROOT, "profiles"), exist_ok=True)
    with open(os.path.join(ROOT, "profiles", f"{tag}_kernel_trace_by_unit.md"), "w") as f:
        f.write(text)
    return text


def summarize_profiles(out_dir: str, bench_json: str, variant: str = "two-pass") -> None:
    """Turn rocprofv3 CSVs of the 1B K=8 workload (two-pass step, or the
    one-pass mean step) into profiles/*.md and the counters file bench.py
    reads for the roofline's `traffic`."""
    import csv
    from paper_2412_07210_amd import synth

    cmds = _profile_cmds(variant)
    tag, sfx = cmds["tag"], cmds["suffix"]
    one = variant == "one-pass"
    kinds = ("fused_mean_kernel", "fused_finish_kernel") if one else \
        ("pass1_gram_kernel", PAIR2, PAIR1, "decide_kernel", "pass2_update_kernel", "update_pattern_probe_kernel")
    dominant = "fused_mean_kernel" if one else "pass2_update_kernel"
    wl = synth.get(DEFAULT_WORKLOAD)
    n, K, R = wl.layer_numel[0], wl.num_workers, wl.replica_bytes
    algo = {"pass1_gram_kernel": n * (4 + K * R), PAIR2: 2 * n * (4 + K * R), PAIR1: n * (4 + K * R),
            "pass2_update_kernel": n * (8 + K * R + 8 + K * R),
            "update_pattern_probe_kernel": n * (8 + K * R + 8 + K * R),
            "fused_mean_kernel": n * (8 + K * R + 8 + K * R)}
    title = "one-pass mean step (no penalty components)" if one else "outer step"
    prof_dir = os.path.join(ROOT, "profiles")
    os.makedirs(prof_dir, exist_ok=True)
    name = "llama1b_k8_one_pass" if one else "llama1b_k8"
    with open(bench_json) as f:
        bench = json.load(f)

    # kernel durations of the headline workload: the default run also steps
    # the secondary workloads afterwards, the first of them with fp32
    # replicas, so the headline's dispatches are those before the first
    # method kernel built for fp32 replicas (template argument false)
    disp = []
    with open(os.path.join(out_dir, f"prof_trace{sfx}", f"{tag}_kernel_trace.csv")) as f:
        for row in csv.DictReader(f):
            kind = _kernel_kind(row["Kernel_Name"])
            if kind and kind != "copy_kernel":
                disp.append((int(row["Start_Timestamp"]), int(row["End_Timestamp"]), kind,
                             bool(re.search(r"<\d+, false|ILi\d+ELb0E", row["Kernel_Name"]))))
    disp.sort()
    cutoff = next((t0 for t0, _, _, f32 in disp if f32), None)
    durs = {}
    for t0, t1, kind, _ in disp:
        if cutoff is None or t0 < cutoff:
            durs.setdefault(kind, []).append(t1 - t0)
    stats = {k: {"Calls": len(v), "AverageNs": sum(v) / len(v), "MinNs": min(v), "MaxNs": max(v)}
             for k, v in durs.items()}
    lines = [f"# Kernel durations: 1B K=8 {title} (24 units x 51,384,320, bf16 replicas)", "",
             "Command (from the repository root; `<out>` = the directory the profiler wrote to):", "",
             "    " + cmds["trace"], "",
             "Dispatches of the headline workload only (those before the secondary workloads' first "
             "kernel); summarised with `python bench.py --summarize-profiles <out> <bench json>`.", "",
             "| kernel | calls | avg us | min us | max us | algorithmic bytes | GB/s at avg |",
             "|---|---|---|---|---|---|---|"]
    for kind in kinds:
        st = stats.get(kind)
        if not st:
            continue
        b = algo.get(kind)
        gbps = f"{b / (st['AverageNs'] * 1e-9) / 1e9:.1f}" if b else "-"
        lines.append(f"| {kind} | {int(st['Calls'])} | {st['AverageNs'] / 1e3:.1f} | "
                     f"{st['MinNs'] / 1e3:.1f} | {st['MaxNs'] / 1e3:.1f} | {b if b else '-'} | {gbps} |")
    rl = bench.get("roofline") or {}
    if dominant in stats and rl:
        ours = rl["avg_launch_ms"] * 1e3
        prof = stats[dominant]["AverageNs"] / 1e3
        lines += ["", f"bench.py's own HIP-event average for {dominant} in the traced run "
                  f"(sampled units, its JSON line's roofline.avg_launch_ms): {ours:.1f} us; "
                  f"rocprofv3 over all launches of the same run: {prof:.1f} us "
                  f"({100 * (ours - prof) / prof:+.1f}%)."]
    with open(os.path.join(prof_dir, f"{name}_kernel_trace_stats.md"), "w") as f:
        f.write("\n".join(lines) + "\n")

    # HBM counters, calibrated on the 2 GiB copy probe of the same run
    def counters(which):
        per = {}
        with open(os.path.join(out_dir, f"prof_{which}{sfx}", f"{tag}_counter_collection.csv")) as f:
            for row in csv.DictReader(f):
                kind = _kernel_kind(row["Kernel_Name"])
                if kind:
                    per.setdefault((kind, int(row["Grid_Size"])), []).append(float(row["Counter_Value"]))
        return per

    fetch, write = counters("fetch"), counters("write")
    copy_bytes = 2 << 30
    copy_fetch = max(v for (k, g), vals in fetch.items() if k == "copy_kernel" for v in vals)
    copy_write = max(v for (k, g), vals in write.items() if k == "copy_kernel" for v in vals)
    fetch_scale = copy_bytes / (copy_fetch * 1024)
    write_scale = copy_bytes / (copy_write * 1024)
    try:  # keep the other variant's entries when they were taken on this source
        with open(COUNTERS_FILE) as f:
            out = json.load(f)
        if out.get("kernel_source_sha256_16") != kernel_source_hash():
            out = {}
    except (OSError, ValueError):
        out = {}
    out.update({"workload": DEFAULT_WORKLOAD, "kernel_source_sha256_16": kernel_source_hash(),
                f"{variant}_fetch_scale": round(fetch_scale, 4),
                f"{variant}_write_scale": round(write_scale, 4),
                f"{variant}_commands": [cmds["fetch"], cmds["write"]]})
    lines = [f"# HBM traffic counters: 1B K=8 {title}", "",
             "Commands (from the repository root; `<out>` = the directory the profiler wrote to):", "",
             "    " + cmds["fetch"], "    " + cmds["write"], "",
             f"Calibration on the plain 2 GiB copy kernel in the same runs: FETCH_SIZE reads "
             f"{copy_fetch:.0f} KiB and WRITE_SIZE {copy_write:.0f} KiB for 2,097,152 KiB moved each "
             f"way, so FETCH_SIZE is scaled by {fetch_scale:.4f} and WRITE_SIZE by {write_scale:.4f}.", "",
             "| kernel | dispatches | FETCH_SIZE KiB | WRITE_SIZE KiB | scaled bytes/launch | "
             "algorithmic bytes | ratio | GB/s on measured bytes at trace avg |",
             "|---|---|---|---|---|---|---|---|"]
    for kind in kinds:
        fv = [v for (k, g), vals in fetch.items() if k == kind for v in vals]
        wv = [v for (k, g), vals in write.items() if k == kind for v in vals]
        if not fv or not wv:
            continue
        f_kib, w_kib = sum(fv) / len(fv), sum(wv) / len(wv)
        traffic = f_kib * 1024 * fetch_scale + w_kib * 1024 * write_scale
        b = algo.get(kind)
        ratio = f"{traffic / b:.4f}" if b else "-"
        st = stats.get(kind)
        gbps = f"{traffic / (st['AverageNs'] * 1e-9) / 1e9:.1f}" if st else "-"
        lines.append(f"| {kind} | {len(fv)} | {f_kib:.1f} | {w_kib:.1f} | {traffic:.4e} | "
                     f"{b if b else '-'} | {ratio} | {gbps} |")
        short = SHORT[kind]
        out[f"{short}_bytes_per_launch"] = round(traffic)
        out[f"{short}_fetch_kib"] = round(f_kib, 1)
        out[f"{short}_write_kib"] = round(w_kib, 1)
        if b:
            out[f"{short}_algorithmic_bytes"] = b
    with open(os.path.join(prof_dir, f"{name}_hbm_counters.md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    with open(COUNTERS_FILE, "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")
    print(json.dumps(out))

def run_sync_group(args, torch, np, wl, dev) -> int:
    """One worker's share of a sync group whose K replicas sit on K GPUs
    (rank `--sync-group-rank`): per unit, edit_group_norm (norm pass and the
    worker's own z-test), edit_group_weights (the group decision) and
    edit_group_apply (Delta_bar norm, clip, Nesterov, the own replica).  The
    two collectives between them are not this GPU's kernels and are stood in
    for on the device: the all-gather by a copy of the rank's own {G, flag}
    pair into all K slots (so every worker counts as unflagged), the
    all-reduce by nothing (the rank's own export serves as Delta_bar).  The
    timed step is the rank's kernels for every unit; its bytes per element
    are (4 + R + 4) for the norm pass, 4 for the Delta_bar pass and
    12 + 8 + R for the update."""
    from paper_2412_07210_amd import OuterConfig, SyncGroupWorker

    K, R = wl.num_workers, wl.replica_bytes
    rank = args.sync_group_rank
    if not 0 <= rank < K:
        print(json.dumps({"error": f"--sync-group-rank must be in 0..{K - 1}"}), flush=True)
        return 2
    hyper = wl.hyper()
    warm = hyper.pop("warmup_rounds")
    w = SyncGroupWorker(OuterConfig(num_workers=K, layer_numel=wl.layer_numel, replica_dtype=wl.replica_dtype,
                                    ema_warmup_rounds=warm, **hyper), rank, dev)
    log(f"sync-group worker {rank} of {K}: {wl.num_units} units of {wl.name}")
    units = []
    for u in range(wl.num_units):
        th = wl.init_theta(u, dev, args.seed)
        units.append(dict(th=th, b=torch.zeros_like(th), rep=torch.empty(th.numel(), dtype=wl.torch_dtype, device=dev),
                          delta=torch.empty_like(th), pair=torch.empty(2, dtype=torch.float64, device=dev),
                          gathered=torch.empty(K, 2, dtype=torch.float64, device=dev),
                          w=torch.empty(1, dtype=torch.float64, device=dev)))

    def step(u, d, ev=None):
        if ev is not None:
            ev[0].record()
        w.norm(u, d["th"], d["rep"], d["delta"], d["pair"])
        if ev is not None:
            ev[1].record()
        d["gathered"].copy_(d["pair"].expand(K, 2))  # stands in for the all-gather
        w.weights(u, d["gathered"].view(-1), d["delta"], d["w"])
        if ev is not None:
            ev[2].record()
        w.apply(u, d["delta"], d["th"], d["b"], d["rep"])  # the own export stands in for Delta_bar
        if ev is not None:
            ev[3].record()

    every = max(1, args.profile_every) if args.profile_every > 0 else 0
    step_ms, norm_ms, apply_ms = [], [], []
    for t in range(args.warmup + args.steps):
        for u, d in enumerate(units):
            wl.fill_replicas(d["th"], [d["rep"]], u, t, args.seed)
        torch.cuda.synchronize()
        if t == 1:  # leave the warm-up: an EMA state that every later norm passes
            for u, d in enumerate(units):
                G = float(d["pair"][0])
                w.state_set(u, G, 10.0 * G, warm)
        a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        evs = {u: [torch.cuda.Event(enable_timing=True) for _ in range(4)]
               for u in range(wl.num_units) if every and u % every == 0}
        a.record()
        for u, d in enumerate(units):
            step(u, d, evs.get(u))
        z.record()
        torch.cuda.synchronize()
        if t < args.warmup:
            continue
        step_ms.append(a.elapsed_time(z))
        for u, ev in evs.items():
            norm_ms.append(ev[0].elapsed_time(ev[1]))
            apply_ms.append(ev[2].elapsed_time(ev[3]))
    states = [w.state_get(u) for u in range(wl.num_units)]
    w.close()
    n_tot = sum(wl.layer_numel)
    step_bytes = n_tot * (8 + R + 4 + 20 + R)
    ms = sum(step_ms) / len(step_ms)
    value = step_bytes / (ms * 1e-3) / 1e9
    q = np.percentile(step_ms, [10, 50, 90])
    n0 = wl.layer_numel[0]
    result = {
        "metric": "sync-group worker: one rank's outer-step kernels per round, GB/s of its own HBM bytes",
        "value": round(value, 2), "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f64", "data": "synthetic",
        "config": {
            "workload": f"{wl.name}: {wl.description}", "units": wl.num_units, "unit_numel": n0,
            "group_size": K, "rank": rank, "replica_dtype": wl.replica_dtype, "master_dtype": "f32",
            "entry_point": "edit_group_norm + edit_group_weights + edit_group_apply per unit",
            "collectives": "not this GPU's work; stood in for on the device: the all-gather by a copy of "
                           "the rank's own pair into all K slots, the all-reduce by nothing (the rank's "
                           "own fp32 export serves as Delta_bar)",
            "bytes_per_element": 32 + 2 * R,
            "parallelism": "one worker of a sync group with one replica per GPU",
        },
        "ms_p10": round(float(q[0]), 4), "ms_p50": round(float(q[1]), 4), "ms_p90": round(float(q[2]), 4),
        "pct_peak_hbm": round(100 * value / PEAK_HBM_GBPS, 2),
        "rollbacks_total": sum(int(st.rolled_back) for st in states),
    }
    if apply_ms:
        per_launch = n0 * (4 + 20 + R)
        avg = sum(apply_ms) / len(apply_ms)
        achieved = per_launch / (avg * 1e-3) / 1e9
        result["roofline"] = {
            "kernel": "edit_group_apply (group_dbar + group_clip + group_update)", "bound": "hbm",
            "achieved": round(achieved, 2), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
            "frac": round(achieved / PEAK_HBM_GBPS, 4), "traffic": None,
            "bytes_per_launch": per_launch, "avg_launch_ms": round(avg, 5), "sampled_launches": len(apply_ms),
        }
        norm_avg = sum(norm_ms) / len(norm_ms)
        result["kernels_ms_avg"] = {
            "norm_call": round(norm_avg, 5), "apply_call": round(avg, 5),
            "norm_call_gbps": round(n0 * (8 + R) / (norm_avg * 1e-3) / 1e9, 2),
        }
    else:
        result["roofline"] = None
    print(json.dumps(result), flush=True)
    return 0


def summarize_group_trace(out_dir: str, bench_json: str) -> str:
    """profiles/ table of a rocprofv3 --kernel-trace --stats run of
    `bench.py --sync-group-rank 0` (`<out>/prof_group/group_kernel_stats.csv`)."""
    import csv

    with open(bench_json) as f:
        bench = json.load(f)
    n, R = bench["config"]["unit_numel"], 2 if bench["config"]["replica_dtype"] == "bf16" else 4
    algo = {"group_norm_kernel": n * (8 + R), "group_dbar_kernel": n * 4, "group_update_kernel": n * (20 + R)}
    rows = []
    with open(os.path.join(out_dir, "prof_group", "group_kernel_stats.csv")) as f:
        for row in csv.DictReader(f):
            name = row["Name"]
            kind = next((k for k in ("group_norm_kernel", "group_self_kernel", "group_weights_kernel",
                                     "group_clear_kernel", "group_dbar_kernel", "group_clip_kernel",
                                     "group_update_kernel") if k in name), None)
            if kind:
                rows.append((kind, int(float(row["Calls"])), float(row["AverageNs"]) / 1e3,
                             float(row["MinNs"]) / 1e3, float(row["MaxNs"]) / 1e3))
    order = ["group_norm_kernel", "group_self_kernel", "group_weights_kernel", "group_clear_kernel",
             "group_dbar_kernel", "group_clip_kernel", "group_update_kernel"]
    rows.sort(key=lambda r: order.index(r[0]))
    lines = [f"# Kernel durations: one sync-group worker (rank 0 of {bench['config']['group_size']}), "
             f"{bench['config']['units']} units x {n:,} elements, {bench['config']['replica_dtype']} replica", "",
             "Command (from the repository root; `<out>` = the directory the profiler wrote to):", "",
             "    rocprofv3 --kernel-trace --stats -f csv -d <out>/prof_group -o group -- "
             "python bench.py --sync-group-rank 0", "",
             "The collectives between the calls are stood in for on the device (see the bench's config).", "",
             "| kernel | calls | avg us | min us | max us | algorithmic bytes | GB/s at avg |",
             "|---|---|---|---|---|---|---|"]
    for kind, calls, avg, mn, mx in rows:
        b = algo.get(kind)
        gbps = f"{b / (avg * 1e-6) / 1e9:.1f}" if b else "-"
        lines.append(f"| {kind} | {calls} | {avg:.1f} | {mn:.1f} | {mx:.1f} | {b if b else '-'} | {gbps} |")
    lines += ["", f"The traced run's own line: {bench['ms_per_step']} ms per step, {bench['value']} GB/s "
              f"({bench['pct_peak_hbm']}% of 8 TB/s) on the rank's bytes."]
    text = "\n".join(lines) + "\n"
    with open(os.path.join(ROOT, "profiles", "sync_group_worker_1b_kernel_trace_stats.md"), "w") as f:
        f.write(text)
    return text


# SQ counters of the matrix-core Gram pass, two rocprofv3 --pmc runs (at most
# eight SQ counters each) of a short K = 16 run.
SQ_PASSES = {
    "a": ["SQ_INSTS_VALU", "SQ_INSTS_MFMA", "SQ_VALU_MFMA_BUSY_CYCLES", "SQ_BUSY_CYCLES", "SQ_WAIT_INST_ANY",
          "SQ_WAVE_CYCLES", "SQ_ACTIVE_INST_VALU", "SQ_INSTS_VALU_CVT", "GRBM_GUI_ACTIVE"],
    "b": ["SQ_INSTS_VALU_ADD_F64", "SQ_INSTS_VALU_MFMA_F64", "SQ_INSTS_VALU_MFMA_MOPS_F64", "SQ_INSTS_VALU_INT32",
          "SQ_INSTS_VALU_FMA_F64", "SQ_WAIT_ANY", "SQ_INSTS_SALU", "SQ_ACTIVE_INST_ANY"],
}
SQ_WORKLOAD_ARGS = ("--config aedit1b-k16-bf16 --units 3 --steps 2 --warmup 1 --no-cpu-baseline --profile-every 0 "
                    "--secondary 0 --update-probe 0 --no-copy-probe --no-settle")


def sq_commands() -> dict:
    return {k: f"rocprofv3 --pmc {' '.join(v)} -f csv -d <out>/prof_sq_{k} -o sq -- python bench.py "
               f"{SQ_WORKLOAD_ARGS}" for k, v in SQ_PASSES.items()}


def summarize_sq_counters(out_dir: str) -> str:
    """profiles/ table of the Gram pass's SQ counters (K = 16, one
    51,380,224-element unit per dispatch): per-dispatch averages and what
    they say about the pass's bound."""
    import csv

    vals = {}
    for k in SQ_PASSES:
        with open(os.path.join(out_dir, f"prof_sq_{k}", "sq_counter_collection.csv")) as f:
            for row in csv.DictReader(f):
                if "pass1_gram_mfma_kernel" not in row["Kernel_Name"] or int(row["Grid_Size"]) < 100_000:
                    continue  # the unit's launches, not the gains' single blocks
                vals.setdefault(row["Counter_Name"], []).append(float(row["Counter_Value"]))
    avg = {c: sum(v) / len(v) for c, v in vals.items()}
    n = 51_380_224
    lines = ["# SQ counters of the matrix-core Gram pass: K = 16, bf16, 51,380,224-element unit", "",
             "Commands (from the repository root; `<out>` = the directory the profiler wrote to):", ""]
    lines += ["    " + c for c in sq_commands().values()]
    lines += ["", f"Summarised with `python bench.py --summarize-sq-counters <out>`; per-dispatch averages over "
              f"{min(len(v) for v in vals.values())} dispatches of pass1_gram_mfma_kernel on the unit.", "",
              "| counter | per dispatch | per element |", "|---|---|---|"]
    for c in SQ_PASSES["a"] + SQ_PASSES["b"]:
        if c in avg:
            lines.append(f"| {c} | {avg[c]:.4g} | {avg[c] / n:.4g} |")
    text = "\n".join(lines) + "\n"
    with open(os.path.join(ROOT, "profiles", "aedit1b_k16_gram_pass_sq_counters.md"), "w") as f:
        f.write(text)
    return text


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[1])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=90)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default=DEFAULT_WORKLOAD,
                    help="workload: " + ", ".join(WORKLOAD_NAMES))
    ap.add_argument("--streams", type=int, default=1, help="HIP streams for the unit pipeline")
    ap.add_argument("--per-unit", action="store_true",
                    help="one edit_outer_step_layer call per unit instead of edit_outer_step_round")
    ap.add_argument("--units", type=int, default=0, help="use only the first N units (0 = all)")
    ap.add_argument("--one-pass", action="store_true",
                    help="the DiLoCo outer step (no penalty components) as one fused pass "
                         "(flag EDIT_ONE_PASS)")
    ap.add_argument("--host-state", action="store_true",
                    help="theta and momentum in pinned host memory, stepped through "
                         "edit_outer_step_round_host (the outer optimizer state off the GPU)")
    ap.add_argument("--shards", type=int, default=1,
                    help="split every unit into S shards that share one decision through "
                         "edit_outer_gram_layer / edit_outer_apply_layer (the module-norm path)")
    ap.add_argument("--sync-group-rank", type=int, default=None, metavar="R",
                    help="time rank R's share of a sync group whose K replicas sit on K GPUs "
                         "(edit_group_*; the collectives stood in for on the device)")
    ap.add_argument("--update-probe", type=int, default=3, metavar="REPS",
                    help="after the timed rounds, time REPS launches per unit of the update pass's access "
                         "pattern with no arithmetic (edit_outer_update_probe); 0: skip")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--profile-every", type=int, default=12,
                    help="record per-kernel HIP events on every k-th unit (0: none, roofline then null)")
    ap.add_argument("--records", metavar="PATH",
                    help="write every unit's decision of every timed round as JSON lines "
                         "(G, mask, weights, Gbar, beta, EMA state)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--secondary", type=int, default=1,
                    help="1: after the default workload, also measure " + ", ".join(SECONDARY) + " (0: skip)")
    ap.add_argument("--secondary-steps", type=int, default=10, help="timed rounds of each secondary workload")
    ap.add_argument("--no-copy-probe", action="store_true")
    ap.add_argument("--no-settle", action="store_true",
                    help="skip the untimed cache settle between input generation and the step")
    ap.add_argument("--summarize-profiles", nargs=2, metavar=("OUT_DIR", "BENCH_JSON"),
                    help="write profiles/ summaries from rocprofv3 CSVs under OUT_DIR (no GPU)")
    ap.add_argument("--profile-variant", default="two-pass", choices=("two-pass", "one-pass"),
                    help="which step --summarize-profiles reads (default: the two-pass step)")
    ap.add_argument("--summarize-group-trace", nargs=2, metavar=("OUT_DIR", "BENCH_JSON"),
                    help="write the profiles/ table of a traced --sync-group-rank run (no GPU)")
    ap.add_argument("--summarize-sq-counters", metavar="OUT_DIR",
                    help="write the profiles/ table of the K = 16 Gram pass's SQ counters (no GPU)")
    ap.add_argument("--summarize-trace", nargs=2, metavar=("OUT_DIR", "WORKLOAD"),
                    help="write a per-unit-size kernel table from a rocprofv3 kernel trace (no GPU)")
    args = ap.parse_args(argv)
    if args.summarize_profiles:
        summarize_profiles(*args.summarize_profiles, variant=args.profile_variant)
        return 0
    if args.summarize_sq_counters:
        print(summarize_sq_counters(args.summarize_sq_counters))
        return 0
    if args.summarize_trace:
        print(summarize_trace_by_grid(*args.summarize_trace))
        return 0
    if args.summarize_group_trace:
        print(summarize_group_trace(*args.summarize_group_trace))
        return 0

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "this benchmark runs on exactly one GPU: the outer step reduces "
                                   "all K replicas in one GPU's HBM; --gpus must be 1"}), flush=True)
        return 2

    import numpy as np
    import torch

    from paper_2412_07210_amd import ONE_PASS, EditOuter, OuterConfig, outer, synth

    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}), flush=True)
        return 3
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    wl = synth.get(args.config)
    if args.units:
        wl = wl.with_units(range(args.units))
    if args.sync_group_rank is not None:
        return run_sync_group(args, torch, np, wl, dev)
    K, R = wl.num_workers, wl.replica_bytes
    hyper = wl.hyper()
    warm_rounds = hyper.pop("warmup_rounds")
    S = max(1, args.shards)
    if S > 1 and (args.per_unit or args.streams > 1):
        print(json.dumps({"error": "--shards runs its own issue order; drop --per-unit/--streams"}))
        return 2
    if S > 1 and args.one_pass:
        print(json.dumps({"error": "the one-pass step has no Gram to share between shards"}))
        return 2
    if args.one_pass:
        hyper["flags"] = ONE_PASS
    if args.host_state and (S > 1 or args.per_unit or args.streams > 1):
        print(json.dumps({"error": "--host-state runs whole rounds; drop --shards/--per-unit/--streams"}))
        return 2

    def shard_cuts(n):
        # contiguous shards whose starts are multiples of 8 elements (16-byte aligned views)
        step = -(-n // (8 * S)) * 8
        return [min(n, i * step) for i in range(S)] + [n]

    handle_numel = wl.layer_numel if S == 1 else \
        [b - a for n in wl.layer_numel for a, b in zip(shard_cuts(n)[:-1], shard_cuts(n)[1:])]
    lib = EditOuter(OuterConfig(num_workers=K, layer_numel=handle_numel, replica_dtype=wl.replica_dtype,
                                ema_warmup_rounds=warm_rounds, **hyper), dev)
    log(f"workload {wl.name}: {wl.num_units} units, {wl.total_numel:,} params, K={K}, {wl.replica_dtype}")

    units = []
    for u in range(wl.num_units):
        th = wl.init_theta(u, dev, args.seed)
        reps = [torch.empty(th.numel(), dtype=wl.torch_dtype, device=dev) for _ in range(K)]
        if args.host_state:  # the outer optimizer state lives in pinned host memory
            th_h = torch.empty(th.numel(), dtype=torch.float32, pin_memory=True)
            th_h.copy_(th)
            b_h = torch.zeros(th.numel(), dtype=torch.float32, pin_memory=True)
            del th
            units.append((th_h, b_h, reps))
        else:
            units.append((th, torch.zeros_like(th), reps))
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(device=dev) for _ in range(args.streams)] if args.streams > 1 else None
    # validated once; each step is one C call
    plan = lib.prepare_round(units, host=args.host_state) if S == 1 else None
    shard_views = []  # per unit: [(handle layer, theta, momentum, replicas)] and its Gram buffers
    for u, (th, b, reps) in enumerate(units):
        cuts = shard_cuts(th.numel())
        views = [(u * S + s, th[a:z], b[a:z], [r[a:z] for r in reps])
                 for s, (a, z) in enumerate(zip(cuts[:-1], cuts[1:]))] if S > 1 else []
        shard_views.append((views, torch.empty(S, lib.num_pairs, dtype=torch.float64, device=dev),
                            torch.empty(lib.num_pairs, dtype=torch.float64, device=dev)))

    def sharded_round():
        for views, grams, total in shard_views:
            for s, (layer, th, b, reps) in enumerate(views):
                lib.gram_layer(layer, th, reps, gram=grams[s])
            torch.sum(grams, dim=0, out=total)  # stands in for the shard group's all-reduce
            for layer, th, b, reps in views:
                lib.apply_layer(layer, total, th, b, reps)

    events = args.profile_every > 0 and S == 1
    lib.set_profiling(args.profile_every if events else 0)

    # Input generation leaves dirty lines of the freshly written replicas in
    # L2 and the 256 MB Infinity Cache.  Streaming 1 GiB through the copy
    # kernel (untimed) writes them back, so the timed step starts with its
    # inputs resident in HBM and pays for no one else's write-backs.
    settle_src = settle_dst = None
    if not args.no_settle:
        settle_src = torch.zeros(256 << 20, dtype=torch.float32, device=dev)
        settle_dst = torch.empty_like(settle_src)

    step_ms, p1_ms, p2_ms = [], [], []
    p1_bytes = p2_bytes = step_bytes = nominal_bytes = 0
    p1_sample_bytes = p2_sample_bytes = 0
    p1_launches = p2_launches = 0
    masked_total = rollbacks = 0
    samples = []
    total_rounds = args.warmup + args.steps
    records = open(args.records, "w") if args.records else None
    t_start = time.time()
    for t in range(total_rounds):
        std = wl.worker_std(t, args.seed)
        for u, (th, b, reps) in enumerate(units):
            wl.fill_replicas(th.to(dev) if args.host_state else th, reps, u, t, args.seed, std=std)
        timed = t >= args.warmup
        if timed and t == args.warmup and not args.no_cpu_baseline:
            for u in range(wl.num_units):  # every unit of the first timed round
                th, b, reps = units[u]
                hb = [r.view(torch.int16).cpu().numpy().view(np.uint16) if r.dtype == torch.bfloat16
                      else r.cpu().numpy() for r in reps]
                samples.append((u, th.cpu().numpy().copy(), b.cpu().numpy().copy(), hb))
        if settle_src is not None:
            outer.copy_probe(settle_dst, settle_src)
        torch.cuda.synchronize()
        a = torch.cuda.Event(enable_timing=True)
        z = torch.cuda.Event(enable_timing=True)
        a.record()
        if S > 1:
            sharded_round()
        elif args.per_unit and streams is None:
            for u, (th, b, reps) in enumerate(units):
                lib.step_layer(u, th, b, reps)
        elif streams is None:
            plan.run()
        else:
            lib.step_round(units, streams=streams)
        z.record()
        torch.cuda.synchronize()
        if not timed:
            continue
        step_ms.append(a.elapsed_time(z))
        for u, (th, b, reps) in enumerate(units):
            st = lib.state_get(u * S)  # every shard of a module holds the same decision
            active = int(np.count_nonzero(st.weight > 0)) if st.clip_coef > 0 else 0
            b1, b2 = unit_bytes(th.numel(), K, R, active, st.rolled_back, args.one_pass)
            p1_bytes += b1
            p2_bytes += b2
            step_bytes += b1 + b2
            nominal_bytes += th.numel() * ((2 * K * R + 16) if args.one_pass else (3 * K * R + 20))
            masked_total += int(st.anomalous.sum())
            rollbacks += int(st.rolled_back)
            if records:
                records.write(json.dumps({
                    "round": t, "unit": u, "G": st.norm.tolist(), "mask": st.anomalous.tolist(),
                    "w": st.weight.tolist(), "gbar": st.synced_norm, "beta": st.clip_coef,
                    "rolled_back": bool(st.rolled_back), "z_tested": bool(st.z_tested),
                    "mu": st.ema_mean.tolist(), "sigma": st.ema_std.tolist()}) + "\n")
            if events and u % args.profile_every == 0:
                k1, k2 = lib.kernel_times(u)
                p1_ms.append(k1)
                p2_ms.append(k2)
                p1_sample_bytes += b1
                p2_sample_bytes += b2
            p1_launches += 1
            p2_launches += 1
        if (t - args.warmup) % 10 == 0:
            log(f"round {t}: {step_ms[-1]:.3f} ms")
    wall = time.time() - t_start
    if records:
        records.close()
    del settle_src, settle_dst

    total_ms = sum(step_ms)
    ms_per_step = total_ms / len(step_ms)
    value = step_bytes / (total_ms * 1e-3) / 1e9
    min_bytes = sum(th.numel() * (2 * K * R + 16) for th, _, _ in units) * len(step_ms)
    q = np.percentile(step_ms, [10, 50, 90])
    result = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",  # the arithmetic type; theta and b are stored fp32, replicas per config
        "data": "synthetic",
        "config": {
            "workload": f"{wl.name}: {wl.description}",
            "units": wl.num_units,
            "unit_numel": wl.layer_numel[0],
            "total_params": wl.total_numel,
            "num_workers": K,
            "replica_dtype": wl.replica_dtype,
            "master_dtype": "f32",
            "streams": args.streams,
            "entry_point": ("edit_outer_gram_layer + sum + edit_outer_apply_layer per shard" if S > 1 else
                            "edit_outer_step_layer per unit" if args.per_unit else
                            "edit_outer_step_round" if args.streams <= 1 else "edit_outer_step_layer, streams"),
            "shards_per_unit": S,
            "entry_point_host_state": "edit_outer_step_round_host" if args.host_state else None,
            "penalty": "none: DiLoCo outer step in one pass (EDIT_ONE_PASS)" if args.one_pass else
                       "anomaly elimination + weighted averaging + clip (Sec. 3.2)",
            "cache_settle_before_step": not args.no_settle,
            "parallelism": "single GPU, K replicas reduced in HBM",
        },
        "ms_p10": round(float(q[0]), 4),
        "ms_p50": round(float(q[1]), 4),
        "ms_p90": round(float(q[2]), 4),
        "pct_peak_hbm": round(100 * value / PEAK_HBM_GBPS, 2),
        "gbps_on_min_bytes": round(min_bytes / (total_ms * 1e-3) / 1e9, 2),
        "gbps_on_nominal_design_bytes": round(nominal_bytes / (total_ms * 1e-3) / 1e9, 2),
        "masked_workers_total": masked_total,
        "rollbacks_total": rollbacks,
        "wall_s": round(wall, 1),
    }
    if events and args.one_pass and p1_ms:
        per_launch = p1_sample_bytes / len(p1_ms)
        avg_ms = sum(p1_ms) / len(p1_ms)
        achieved = per_launch / (avg_ms * 1e-3) / 1e9
        result["roofline"] = {
            "kernel": "fused_mean_kernel (one pass: mean + Nesterov + write-back + norms)",
            "bound": "hbm",
            "achieved": round(achieved, 2),
            "peak": PEAK_HBM_GBPS,
            "unit": "GB/s",
            "frac": round(achieved / PEAK_HBM_GBPS, 4),
            "traffic": measured_traffic("fused", wl.name),
            "achieved_on_traffic": _on_traffic(measured_traffic("fused", wl.name), avg_ms),
            "bytes_per_launch": int(per_launch),
            "avg_launch_ms": round(avg_ms, 5),
            "sampled_launches": len(p1_ms),
        }
        result["kernels_ms_avg"] = {"fused_mean": round(avg_ms, 5)}
    elif events and p2_ms:
        # average over the sampled launches (units 0, k, 2k, ... of every timed step)
        per_launch = p2_sample_bytes / len(p2_ms)
        avg_ms = sum(p2_ms) / len(p2_ms)
        achieved = per_launch / (avg_ms * 1e-3) / 1e9
        traffic = measured_traffic("pass2", wl.name)
        result["roofline"] = {
            "kernel": "pass2_update_kernel (fused average + clip + Nesterov + write-back)",
            "bound": "hbm",
            "achieved": round(achieved, 2),
            "peak": PEAK_HBM_GBPS,
            "unit": "GB/s",
            "frac": round(achieved / PEAK_HBM_GBPS, 4),
            "traffic": traffic,
            "achieved_on_traffic": _on_traffic(traffic, avg_ms),
            "bytes_per_launch": int(per_launch),
            "avg_launch_ms": round(avg_ms, 5),
            "sampled_launches": len(p2_ms),
        }
        result["kernels_ms_avg"] = {
            "pass1_gram_decide": round(sum(p1_ms) / len(p1_ms), 5),
            "pass2_update": round(avg_ms, 5),
            "pass1_gbps": round((p1_sample_bytes / len(p1_ms)) / (sum(p1_ms) / len(p1_ms) * 1e-3) / 1e9, 2),
        }
    else:
        result["roofline"] = None
    if args.host_state:
        # Bound by the host link: theta and b cross it once each way per step.
        each_way = sum(th.numel() for th, _, _ in units) * 8
        achieved = each_way / (ms_per_step * 1e-3) / 1e9
        result["config"]["state_placement"] = "theta, momentum in pinned host memory; replicas in HBM"
        result["hbm_kernels_roofline"] = result["roofline"]
        result["roofline"] = {
            "kernel": "staging copies of theta and b (hipMemcpyAsync on two copy streams)",
            "bound": "host-link",
            "achieved": round(achieved, 2),
            "peak": PEAK_HOST_LINK_GBPS,
            "unit": "GB/s each way",
            "frac": round(achieved / PEAK_HOST_LINK_GBPS, 4),
            "traffic": None,
            "bytes_per_step_each_way": each_way,
        }
        result["host_link_probe_gbps"] = host_link_probe_gbps(torch)
    if not args.no_copy_probe:
        result["copy_probe_gbps"] = round(copy_probe_gbps(torch, outer), 1)
    if args.update_probe > 0 and S == 1 and not (args.one_pass or args.host_state) and result.get("roofline"):
        result["update_probe"] = update_probe(torch, lib, units, wl, args.update_probe, result["roofline"])
    lib.close()
    del units, plan, shard_views
    torch.cuda.empty_cache()
    if args.secondary and args.config == DEFAULT_WORKLOAD and S == 1 and not (
            args.one_pass or args.host_state or args.per_unit or args.units):
        result["secondary"] = {}
        for name in SECONDARY:
            t0 = time.time()
            result["secondary"][name] = measure_secondary(torch, np, name, args.secondary_steps, 10, args.seed,
                                                          dev)
            log(f"secondary {name}: {result['secondary'][name]['ms_per_step']} ms/step "
                f"({time.time() - t0:.1f} s)")
    if samples:
        result["cpu_baseline"] = cpu_baseline(samples, wl, args.one_pass)
        samples.clear()
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
