#!/usr/bin/env python3
"""Benchmark of one DeDLOC averaging step on one MI355X.

A step is one pass of the whole path over one batch of synthetic input:
shard bounds on the host, the local peer's encode of its own fp32 gradient
(the sender side), and the round: every shard averaged from the N peer
messages, the average re-encoded and gathered, and one LAMB step with
per-tensor trust ratios over the whole parameter vector.  The local
peer's gradient is handed to the round (dedloc_local_peer): the fp16 round
encodes it inside its averaging pass, the int8 round in a launch of its own;
with --separate-encode the caller encodes it before the round.

Default workload: ALBERT-large-shaped (17.7M parameters in 25 tensors,
16 peers, fp16 wire).  Prints ONE JSON line.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E


def _parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="albert_large")
    ap.add_argument("--mode", default="round", choices=["round", "group", "balance", "accumulate"],
                    help="round: the averaging round (default); group: the group (Moshpit) "
                         "all-reduce of the workload's peer messages; balance: host solve time of "
                         "the load-balancing LP for 4..128 peers; accumulate: the local peer's "
                         "gradient accumulation and its overlap with the round")
    ap.add_argument("--group-size", type=int, default=8)
    ap.add_argument("--micro", type=int, default=8,
                    help="accumulate mode: micro-batches accumulated per round")
    ap.add_argument("--graph", action="store_true",
                    help="capture one step (encode + round) in a HIP graph and time its replays")
    ap.add_argument("--optimizer", default="lamb", choices=["lamb", "lars"],
                    help="optimizer after the gather: LAMB (ALBERT runs) or LARS (SwAV runs)")
    ap.add_argument("--separate-encode", action="store_true",
                    help="encode the local peer's gradient in its own launch before the round")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-reps", type=int, default=5)
    ap.add_argument("--copy-probe", type=int, default=0, metavar="BYTES",
                    help="only run a plain device-to-device copy of BYTES, 10 times "
                         "(calibrates HBM byte counters), then exit")
    ap.add_argument("--summarize-trace", metavar="DIR", default=None,
                    help="only turn the rocprofv3 --kernel-trace --stats run under DIR "
                         "(run_kernel_stats.csv) into profiles/kernel_stats_<workload>.json, then exit")
    ap.add_argument("--summarize-counters", metavar="DIR", default=None,
                    help="only turn the rocprofv3 counter runs under DIR (pmc_FETCH_SIZE, "
                         "pmc_WRITE_SIZE, pmc_copy_FETCH_SIZE, pmc_copy_WRITE_SIZE) into "
                         "profiles/traffic_<kernel>_<workload>.json, then exit")
    return ap.parse_args()


# rocprofv3 kernel names -> the library's kernel kinds
KERNEL_KINDS = {
    "dedloc::encode_fp16_kernel": "encode_fp16",
    "dedloc::encode_i8_kernel": "encode_i8",
    "dedloc::decode_fp16_kernel": "decode_fp16",
    "dedloc::decode_i8_kernel": "decode_i8",
    "void dedloc::reduce_fp16_kernel<4>": "reduce_fp16",
    "void dedloc::reduce_fp16_kernel<16>": "reduce_fp16",
    "void dedloc::reduce_i8_kernel<4>": "reduce_i8",
    "void dedloc::reduce_i8_kernel<16>": "reduce_i8",
    "void dedloc::opt_a_kernel<0, 0>": "lamb_a_f32",
    "void dedloc::opt_a_kernel<1, 0>": "lamb_a_fp16",
    "void dedloc::opt_a_kernel<2, 0>": "lamb_a_i8",
    "void dedloc::opt_a_kernel<3, 0>": "lamb_a_fused_fp16",
    "void dedloc::opt_a_kernel<4, 0>": "lamb_a_fused_fp16",
    "void dedloc::opt_a_kernel<5, 0>": "lamb_a_fused_fp16",
    "void dedloc::opt_b_kernel<0, 0>": "lamb_b",
    "void dedloc::opt_a_kernel<0, 1>": "lars_a_f32",
    "void dedloc::opt_a_kernel<1, 1>": "lars_a_fp16",
    "void dedloc::opt_a_kernel<2, 1>": "lars_a_i8",
    "void dedloc::opt_a_kernel<3, 1>": "lars_a_fused_fp16",
    "void dedloc::opt_a_kernel<4, 1>": "lars_a_fused_fp16",
    "void dedloc::opt_a_kernel<5, 1>": "lars_a_fused_fp16",
    "void dedloc::opt_b_kernel<0, 1>": "lars_b",
    "void dedloc::opt_b_kernel<1, 1>": "lars_b",
    "void dedloc::opt_b_kernel<2, 1>": "lars_b",
    "void dedloc::accumulate_kernel<false>": "accumulate",
    "void dedloc::accumulate_kernel<true>": "accumulate_fp16",
    "dedloc::finalize_fp16_kernel": "finalize_fp16",
    "dedloc::finalize_i8_kernel": "finalize_i8",
}
# kernels whose counters come from the accumulate mode (the other kinds from the round)
ACCUMULATE_KINDS = ("accumulate", "accumulate_fp16", "finalize_fp16", "finalize_i8")

COUNTER_COMMANDS = (
    "timeout -s KILL 120 rocprofv3 --pmc {c} --output-format csv -d DIR/pmc_{c} -o run -- "
    "python3 bench.py --mode {m} --workload {w} --steps 5 --warmup 1 --no-cpu-baseline",
    "timeout -s KILL 60 rocprofv3 --pmc {c} --output-format csv -d DIR/pmc_copy_{c} -o run -- "
    "python3 bench.py --copy-probe 268435456",
)


def summarize_counters(root_dir, workload, mode="round"):
    """Per-kernel HBM bytes per launch from FETCH_SIZE and WRITE_SIZE (KiB per
    dispatch), each scaled by the ratio of known bytes to the counter's
    reading for a plain 256 MiB device copy.  Counters taken in `mode` give
    the records of that mode's own kernels only."""
    import csv
    import hashlib
    from collections import defaultdict

    def per_kernel(d):
        acc = defaultdict(list)
        for r in csv.DictReader(open(os.path.join(root_dir, d, "run_counter_collection.csv"))):
            acc[r["Kernel_Name"].split("(")[0]].append(float(r["Counter_Value"]))
        return {k: sum(v) / len(v) for k, v in acc.items()}

    copy_bytes = 268435456
    scale = {}
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        cp = per_kernel(f"pmc_copy_{c}")
        copy_kib = max(cp.values())  # the copy kernel
        scale[c] = copy_bytes / (copy_kib * 1024.0)
    fetch, write = per_kernel("pmc_FETCH_SIZE"), per_kernel("pmc_WRITE_SIZE")
    root = os.path.dirname(os.path.abspath(__file__))
    digest = hashlib.sha256(open(os.path.join(root, "paper_2106_10207_amd", "csrc", "kernels.hip"),
                                 "rb").read()).hexdigest()
    written = []
    for name, kind in KERNEL_KINDS.items():
        if name not in fetch or name not in write or (kind in ACCUMULATE_KINDS) != (mode == "accumulate"):
            continue
        fb = fetch[name] * 1024.0 * scale["FETCH_SIZE"]
        wb = write[name] * 1024.0 * scale["WRITE_SIZE"]
        rec = {
            "kernel": kind, "workload": workload,
            "fetch_kib_per_launch_raw": fetch[name], "write_kib_per_launch_raw": write[name],
            "copy_calibration": {"bytes": copy_bytes, "fetch_scale": scale["FETCH_SIZE"],
                                 "write_scale": scale["WRITE_SIZE"]},
            "hbm_bytes_per_launch": fb + wb, "read_bytes_per_launch": fb, "write_bytes_per_launch": wb,
            "bytes_kind": "L2 <-> fabric (FETCH_SIZE / WRITE_SIZE count L2 misses and write-backs; "
                          "Infinity Cache hits are included, so these are not DRAM bytes)",
            "commands": [c.format(c=k, w=workload, m=mode) for c in COUNTER_COMMANDS
                         for k in ("FETCH_SIZE", "WRITE_SIZE")],
            "kernels_hip_sha256": digest,
        }
        out = os.path.join(root, "profiles", f"traffic_{kind}_{workload}.json")
        json.dump(rec, open(out, "w"), indent=1)
        written.append(out)
    return written


TRACE_COMMAND = ("rocprofv3 --kernel-trace --stats --output-format csv -d DIR -o run -- "
                 "python3 bench.py --workload {w} {extra}--no-cpu-baseline")


def _kernel_source_digest():
    import hashlib
    root = os.path.dirname(os.path.abspath(__file__))
    return hashlib.sha256(open(os.path.join(root, "paper_2106_10207_amd", "csrc", "kernels.hip"),
                               "rb").read()).hexdigest()


def summarize_trace(root_dir, workload, extra=""):
    """Average, minimum and maximum duration and call count of every library
    kernel instance from a rocprofv3 --kernel-trace --stats run, with the
    hash of the kernel source it was taken with; with the run's per-dispatch
    trace beside it, also the median duration (the run also times the cold
    steps, a third of the launches, which the median leaves out)."""
    import csv
    rows = {}
    for r in csv.DictReader(open(os.path.join(root_dir, "run_kernel_stats.csv"))):
        name = r["Name"].split("(")[0]
        if "dedloc::" not in name:
            continue
        rows[name] = {"calls": int(r["Calls"]), "avg_us": float(r["AverageNs"]) / 1e3,
                      "min_us": float(r["MinNs"]) / 1e3, "max_us": float(r["MaxNs"]) / 1e3,
                      "kind": KERNEL_KINDS.get(name)}
    trace = os.path.join(root_dir, "run_kernel_trace.csv")
    if os.path.exists(trace):
        durs = {}
        for r in csv.DictReader(open(trace)):
            name = r["Kernel_Name"].split("(")[0]
            if name in rows:
                durs.setdefault(name, []).append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
        for name, d in durs.items():
            if len(d) == rows[name]["calls"]:
                rows[name]["median_us"] = float(np.median(d))
    root = os.path.dirname(os.path.abspath(__file__))
    rec = {"workload": workload, "command": TRACE_COMMAND.format(w=workload, extra=extra),
           "kernels": rows, "kernels_hip_sha256": _kernel_source_digest()}
    out = os.path.join(root, "profiles", f"kernel_stats_{workload}.json")
    json.dump(rec, open(out, "w"), indent=1)
    return out


def _instance(kind, dr):
    """rocprofv3's name of the kernel instance a step of `dr` launches for `kind`."""
    src = 5 if dr.local_in_kernel else (4 if int(np.count_nonzero(dr.counts)) > 64 else 3)
    names = {"lamb_a_fused_fp16": f"void dedloc::opt_a_kernel<{src}, 0>",
             "lars_a_fused_fp16": f"void dedloc::opt_a_kernel<{src}, 1>",
             "reduce_i8": "void dedloc::reduce_i8_kernel<16>",
             "lamb_b": "void dedloc::opt_b_kernel<0, 0>",
             "lamb_a_i8": "void dedloc::opt_a_kernel<2, 0>"}
    return names.get(kind)


def rocprof_durations_us(kind, dr):
    """The committed rocprofv3 average and median durations of the step's
    `kind` kernel for this workload (median None when not recorded), or
    (None, None, why) when there is no summary or the kernel source changed
    since."""
    root = os.path.dirname(os.path.abspath(__file__))
    path = os.path.join(root, "profiles", f"kernel_stats_{dr.wl.name}.json")
    if not os.path.exists(path):
        return None, None, None
    rec = json.load(open(path))
    rel = os.path.relpath(path, root)
    if rec.get("kernels_hip_sha256") != _kernel_source_digest():
        return None, None, rel + " (stale: kernel source changed)"
    k = rec["kernels"].get(_instance(kind, dr))
    return (k["avg_us"], k.get("median_us"), rel) if k else (None, None, rel)


def kernel_roofline(dr, prof, steps):
    """Achieved algorithmic HBM bandwidth of the kernel that dominates the
    step.  Algorithmic bytes per launch (b = wire bytes per element,
    N = active peers, P elements):
      lamb_a_fused_fp16: N*b*P peer reads + b*P code writes + 12P reads of
                         x, m, v + 8P writes of m', v'
      (with the local peer's encode inside the averaging pass, the
      lamb_a_fused_fp16 and lars_a_fused_fp16 launches read its 4P fp32
      gradient and write its b*P message instead of reading that message:
      +4P)
      reduce_i8:         N*b*P peer reads + b*P code/scale writes
      lamb_a_i8:         b*P code reads + 20P (x, m, v reads; m', v' writes)
      lamb_b:            12P reads (x, m', v') + 4P writes
      lars_a_fused_fp16: N*b*P peer reads + b*P code writes + 4P reads of x
      lars_a_i8:         b*P code reads + 4P reads of x
      lars_b:            b*P code reads + 8P reads (x, v) + 8P writes (x', v')
      encode_fp16 / encode_i8: 4P reads + b*P writes"""
    wl = dr.wl
    P = wl.P
    b = wl.wire_bytes_per_elem
    n_act = int(np.count_nonzero(dr.counts))
    loc = 4.0 if dr.local_in_kernel else 0.0
    per_launch = {
        "lamb_a_fused_fp16": (n_act * b + b + 20.0 + loc) * P,
        "reduce_i8": (n_act * b + b) * P,
        "lamb_a_i8": (b + 20.0) * P,
        "lamb_a_fp16": (b + 20.0) * P,
        "lamb_b": 16.0 * P,
        "lars_a_fused_fp16": (n_act * b + b + 4.0 + loc) * P,
        "lars_a_i8": (b + 4.0) * P,
        "lars_a_fp16": (b + 4.0) * P,
        "lars_b": (b + 16.0) * P,
        "encode_fp16": (4.0 + b) * P,
        "encode_i8": (4.0 + b) * P,
    }
    name = max(prof, key=lambda k: prof[k][0])
    total_ms, launches = prof[name]
    per_step = launches / steps
    avg_ms = total_ms / launches
    # chunked kernels launch several times per step; bytes per launch scale
    nbytes = per_launch.get(name, 0.0) / per_step
    achieved = nbytes / (avg_ms * 1e-3) / 1e9
    roof = {
        "bound": "hbm",
        "kernel": name,
        "achieved": round(achieved, 1),
        "peak": HBM_PEAK_GBPS,
        "unit": "GB/s",
        "frac": round(achieved / HBM_PEAK_GBPS, 4),
        "traffic": None,
        "avg_launch_us": round(avg_ms * 1e3, 2),
        "algorithmic_bytes_per_launch": nbytes,
    }
    if name.endswith("_fused_fp16") and loc:
        # the local peer's 4P gradient read is its encode's (a sender-side
        # step), not the round's: the pass's share of the round's own bytes
        strict = nbytes - loc * P / per_step
        roof["round_bytes_per_launch"] = strict
        roof["frac_round_bytes"] = round(strict / (avg_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4)
    rp_avg, rp_med, rp_src = rocprof_durations_us(name, dr)
    roof["rocprof_avg_launch_us"] = None if rp_avg is None else round(rp_avg, 2)
    roof["rocprof_median_launch_us"] = None if rp_med is None else round(rp_med, 2)
    # the trace also times the cold-cache steps; with one launch per step its
    # median is the warm launch the events above time (launch chunks of
    # unequal size, several per step, compare by the average)
    rp_us = rp_med if rp_med is not None and per_step == 1 else rp_avg
    roof["frac_rocprof"] = None if rp_us is None else round(nbytes / (rp_us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4)
    roof["rocprof_source"] = rp_src
    return name, roof, {k: _kernel_entry(v, steps, per_launch.get(k)) for k, v in prof.items()}


def _kernel_entry(v, steps, step_bytes):
    """ms per step and launches of one kernel kind; with its algorithmic
    bytes per step (summed over its launches), the achieved GB/s."""
    total_ms, launches = v
    e = {"ms_per_step": round(total_ms / steps, 4), "launches_per_step": launches / steps}
    if step_bytes:
        e["algorithmic_GBps"] = round(step_bytes / (total_ms / steps * 1e-3) / 1e9, 1)
    return e


def measured_traffic(kernel, workload):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter
    summary (FETCH_SIZE + WRITE_SIZE, calibrated on a plain copy), or None
    when there is none or the kernel source changed since it was taken."""
    import hashlib
    root = os.path.dirname(os.path.abspath(__file__))
    path = os.path.join(root, "profiles", f"traffic_{kernel}_{workload}.json")
    src = os.path.join(root, "paper_2106_10207_amd", "csrc", "kernels.hip")
    if not os.path.exists(path):
        return None, None
    rec = json.load(open(path))
    digest = hashlib.sha256(open(src, "rb").read()).hexdigest()
    if rec.get("kernels_hip_sha256") != digest:
        return None, os.path.relpath(path, root) + " (stale: kernel source changed)"
    return rec["hbm_bytes_per_launch"], os.path.relpath(path, root)


def bench_balance():
    """Host time of dedloc_balance (the library's interior point; median of 5
    solves after one warm-up) and of the oracle (HiGHS: the literal n^3
    program up to 32 peers, its O(n^2) reformulation above) on random
    collaborations: compute 1..200 samples/s, bandwidths 10..1000 Mbit/s,
    ALBERT-large P."""
    from oracle import lp
    from paper_2106_10207_amd import dedloc as D
    rows = []
    for n in (4, 8, 16, 24, 32, 48, 64, 96, 128):
        rng = np.random.default_rng(n)
        s = rng.uniform(1, 200, n)
        d = rng.uniform(10, 1000, n) * 1e5 / 4
        u = rng.uniform(10, 1000, n) * 1e5 / 4
        B, P = 4096.0, 17_683_968.0
        r = D.dedloc_balance(s, d, u, B, P)
        times = []
        for _ in range(5):
            t0 = time.perf_counter()
            r = D.dedloc_balance(s, d, u, B, P)
            times.append(time.perf_counter() - t0)
        reduced = n > 32
        t1 = time.perf_counter()
        o = lp.solve(s, d, u, B, P, reduced=reduced)
        t2 = time.perf_counter()
        rows.append({"peers": n, "lib_ms": round(float(np.median(times)) * 1e3, 2),
                     "oracle_ms": round((t2 - t1) * 1e3, 1), "oracle_program": "reduced" if reduced else "literal",
                     "xi": r["xi"], "xi_oracle": o["xi"]})
        print(json.dumps(rows[-1]), file=sys.stderr, flush=True)
    return {"metric": "load-balancing LP solve time (host)", "unit": "ms", "higher_is_better": False,
            "cores": 1, "cpu_model": _cpu_model(), "rows": rows}


def bench_group(args, wl):
    """Group (Moshpit) all-reduce of the workload's peer messages in groups
    of --group-size: ceil(log_m n) iterations, one launch each.  Algorithmic
    bytes per iteration: every member's message read once (N_k * P * b) and
    every group message written once (G_k * P * b)."""
    import torch
    from paper_2106_10207_amd import dedloc as D
    from paper_2106_10207_amd import harness as H
    from paper_2106_10207_amd import workloads as W
    dr = H.DeviceRound(wl, "cuda")
    m = args.group_size
    ga = D.GroupAllreduce(dr.codes, dr.counts, m, wl.P, dr.codec,
                          dr.scales if dr.codec == D.DEDLOC_CODEC_I8 else None)
    # member and group counts per iteration from the same grid rule as the library
    n = wl.n_peers
    d = D.group_iterations(n, m)
    cnt = list(dr.counts) + [0] * (m ** d - n)
    reads = writes = 0
    lo = 1
    for k in range(d):
        new = cnt[:]
        for g in range(m ** d // m):
            base = (g // lo) * lo * m + (g % lo)
            members = [base + j * lo for j in range(m)]
            tot = sum(cnt[s] for s in members)
            reads += sum(1 for s in members if cnt[s] > 0)
            writes += 1 if tot > 0 else 0
            for s in members:
                new[s] = tot
        cnt = new
        lo *= m
    alg = (reads + writes) * wl.P * wl.wire_bytes_per_elem
    for _ in range(args.warmup):
        ga()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.steps):
        ga()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    D.dedloc_profile_begin(64 * args.steps + 64)
    for _ in range(args.steps):
        ga()
    prof = D.dedloc_profile_end()
    kname = max(prof, key=lambda k: prof[k][0])
    kms = prof[kname][0] / args.steps
    peer_bytes = dr.bytes_peer_input()
    return {
        "metric": "group all-reduce GB/s of peer input",
        "value": round(peer_bytes / (ms * 1e-3) / 1e9, 2),
        "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms, 5), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": wl.name, "mode": "group", "group_size": m, "iterations": d,
                   "peers": n, "wire": wl.codec},
        "roofline": {"bound": "hbm", "kernel": kname, "achieved": round(alg / (kms * 1e-3) / 1e9, 1),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(alg / (kms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4), "traffic": None,
                     "algorithmic_bytes_per_step": alg, "launches_per_step": prof[kname][1] / args.steps},
    }


def _event_ms(fn, reps, stream=None):
    """Average ms of fn() over reps back-to-back calls, timed with HIP events
    on `stream` (torch's current stream by default)."""
    import torch
    s = stream or torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(s)
    for _ in range(reps):
        fn()
    e1.record(s)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def bench_accumulate(args, wl):
    """Local accumulation (Section 3.1: a peer accumulates micro-batch
    gradients until the collaboration reaches its target batch).  A step adds
    --micro micro-batches of 32 samples into the fp32 accumulator
    (dedloc_accumulate), then turns it into the peer's message
    (dedloc_finalize, which also zeroes the accumulator).  Algorithmic bytes
    per element: accumulate 12 (fp32 gradient: acc read and written, gradient
    read) or 10 (fp16 codes); finalize 8 + b (acc read and zeroed, message
    written).  The overlap case runs the workload's round on the current
    stream while the next step's accumulation runs on a second stream
    (Section 3.2's delayed update), against the two one after the other."""
    import torch
    from paper_2106_10207_amd import dedloc as D
    from paper_2106_10207_amd import harness as H
    dr = H.DeviceRound(wl, "cuda", keep_local_grad=True, fused_local=True)
    P = wl.P
    k = args.micro
    acc = torch.zeros(P, dtype=torch.float32, device="cuda")
    g32 = dr.local_grad
    g16 = D.dedloc_encode(g32, D.DEDLOC_CODEC_FP16)[0]
    msg, msg_scales = D.dedloc_finalize(acc, 1, dr.codec, reset=False)

    def acc32():
        D.dedloc_accumulate(acc, g32, 32.0)

    def acc16():
        D.dedloc_accumulate(acc, g16, 32.0)

    def fin():
        D.dedloc_finalize(acc, 32 * k, dr.codec, codes=msg, scales=msg_scales, reset=True)

    def accumulate_step(stream=None):
        with torch.cuda.stream(stream or torch.cuda.current_stream()):
            for _ in range(k):
                acc32()
            fin()

    reps = max(args.steps, 1)
    for fn in (acc32, acc16, fin, accumulate_step, dr.run):
        for _ in range(args.warmup):
            fn()
    t_acc32 = _event_ms(acc32, reps * k)
    t_acc16 = _event_ms(acc16, reps * k)
    t_fin = _event_ms(fin, reps)
    t_step = _event_ms(accumulate_step, reps)
    t_round = _event_ms(dr.run, reps)

    side = torch.cuda.Stream()  # default priority

    def serial():
        dr.run()
        accumulate_step()

    def overlapped():
        main = torch.cuda.current_stream()
        side.wait_stream(main)
        accumulate_step(side)
        dr.run()
        main.wait_stream(side)

    for _ in range(args.warmup):
        serial()
        overlapped()
    t_serial = _event_ms(serial, reps)
    t_overlap = _event_ms(overlapped, reps)

    # per-launch events of the library's own profiler for the roofline
    D.dedloc_profile_begin(4 * reps * (k + 1) + 64)
    for _ in range(reps):
        for _ in range(k):
            acc32()
        fin()
    prof = D.dedloc_profile_end()
    b = wl.wire_bytes_per_elem
    acc_ms = prof["accumulate"][0] / prof["accumulate"][1]
    fin_kind = "finalize_fp16" if dr.codec == D.DEDLOC_CODEC_FP16 else "finalize_i8"
    fin_ms = prof[fin_kind][0] / prof[fin_kind][1]

    def gbps(nbytes, ms):
        return round(nbytes / (ms * 1e-3) / 1e9, 1)

    acc_bytes = 12.0 * P
    traffic, traffic_source = measured_traffic("accumulate", wl.name)
    return {
        "metric": "local gradient accumulation, algorithmic GB/s of the accumulate kernel",
        "value": gbps(acc_bytes, t_acc32), "unit": "GB/s", "n_gpus": 1, "steps": reps,
        "warmup": args.warmup, "ms_per_step": round(t_step, 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": wl.name, "mode": "accumulate", "params": P, "micro_batches": k,
                   "wire": wl.codec},
        "accumulate_fp32": {"ms": round(t_acc32, 5), "GBps": gbps(acc_bytes, t_acc32)},
        "accumulate_fp16": {"ms": round(t_acc16, 5), "GBps": gbps(10.0 * P, t_acc16)},
        "finalize": {"ms": round(t_fin, 5), "GBps": gbps((8.0 + b) * P, t_fin)},
        "overlap": {"round_ms": round(t_round, 5), "accumulate_step_ms": round(t_step, 5),
                    "serial_ms": round(t_serial, 5), "overlapped_ms": round(t_overlap, 5)},
        "roofline": {"bound": "hbm", "kernel": "accumulate", "achieved": gbps(acc_bytes, acc_ms),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(acc_bytes / (acc_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
                     "traffic": traffic, "traffic_source": traffic_source,
                     "avg_launch_us": round(acc_ms * 1e3, 2), "algorithmic_bytes_per_launch": acc_bytes,
                     "finalize_avg_launch_us": round(fin_ms * 1e3, 2),
                     "finalize_GBps": gbps((8.0 + b) * P, fin_ms)},
    }


def cpu_baseline(wl, dr, reps):
    """The oracle (plain C, no contraction) on the same workload: one local
    encode plus one round, on the host, timed after its inputs are prepared.
    Built for this host's CPU (-O3 -march=native) with its element loops
    split statically over OpenMP threads; timed on one thread and on every
    thread this process may use, and the two runs' outputs are compared bit
    for bit."""
    import oracle
    from paper_2106_10207_amd import workloads as W
    oracle.use_library(oracle.build_fast())
    codec = 1 if wl.codec == "fp16" else 2
    codes, scales = [], []
    local_grad = None
    for p in range(wl.n_peers):
        g = W.peer_gradient(wl, p, "cuda").cpu().numpy()
        if codec == 1:
            codes.append(oracle.encode_fp16(g))
        else:
            c, s = oracle.encode_i8(g, 1024)
            codes.append(c)
            scales.append(s)
        if p == dr.local:
            local_grad = g
        del g
    state = [t.cpu().numpy() for t in W.optimizer_state(wl, "cuda")]
    if dr.optimizer == "lamb":
        cfg = oracle.lamb_cfg(wl.lr, wl.beta1, wl.beta2, wl.eps, wl.weight_decay, step=wl.step)
    else:
        cfg = oracle.lars_cfg(wl.lars_lr, wl.lars_momentum, wl.lars_trust_coef, wl.lars_weight_decay)
    bw = W.bandwidth_weights(wl)

    def step():
        x, m, v = state  # the oracle's round copies its state arguments
        bounds = oracle.partition(wl.P, wl.n_shards, bw, wl.shard_align)
        if codec == 1:
            oracle.encode_fp16(local_grad)
        else:
            oracle.encode_i8(local_grad, 1024)
        if dr.optimizer == "lamb":
            return oracle.round_(codes, dr.counts, bounds, codec, x, m, v, wl.offsets(), wl.flags(), cfg,
                                 scales or None, 1024)
        return oracle.round_lars(codes, dr.counts, bounds, codec, x, m, wl.offsets(), wl.flags(), cfg,
                                 scales or None, 1024)

    def timed(threads, n):
        oracle.threads(threads)
        times, out = [], None
        for _ in range(n):
            t0 = time.perf_counter()
            out = step()
            times.append(time.perf_counter() - t0)
        return float(np.median(times)), out

    all_threads = int(os.environ.get("OMP_NUM_THREADS") or 0) or len(os.sched_getaffinity(0))
    all_threads = min(all_threads, len(os.sched_getaffinity(0)))
    t1, r1 = timed(1, max(1, min(reps, 3)))
    tn, rn = timed(all_threads, reps)
    same = all(np.array_equal(np.asarray(r1[k]).view(np.uint8), np.asarray(rn[k]).view(np.uint8))
               for k in r1 if r1[k] is not None)
    peer = dr.bytes_peer_input()
    return {
        "value": round(peer / tn / 1e9, 4),
        "unit": "GB/s",
        "cores": oracle.threads(0),
        "kind": "oracle",
        "sample": f"the full {wl.name} step (partition + local encode + round over all "
                  f"{wl.P} elements), median of {reps} runs on {all_threads} threads; "
                  f"single thread: median of {max(1, min(reps, 3))}",
        "s_per_step": round(tn, 3),
        "single_thread": {"value": round(peer / t1 / 1e9, 4), "s_per_step": round(t1, 3)},
        "threads_bit_identical": bool(same),
        "build": "gcc -O3 -march=native -fopenmp -ffp-contract=off (static partition over elements)",
        "cpu_model": _cpu_model(),
        "nproc": os.cpu_count(),
        "host_threads_available": len(os.sched_getaffinity(0)),
    }


def _cpu_model():
    """Model name of the host CPU with its family/model/stepping numbers."""
    info = {}
    try:
        for line in open("/proc/cpuinfo"):
            if ":" in line:
                k, v = (a.strip() for a in line.split(":", 1))
                if k in ("model name", "cpu family", "model", "stepping", "cache size") and k not in info:
                    info[k] = v
            elif info:
                break
    except OSError:
        return None
    if "model name" not in info:
        return None
    return (f"{info['model name']} (family {info.get('cpu family')}, model {info.get('model')}, "
            f"stepping {info.get('stepping')}, cache {info.get('cache size')})")


def main():
    args = _parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: this build has no multi-GPU path (asked for --gpus {args.gpus}).",
              file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2106_10207_amd import dedloc as D
    from paper_2106_10207_amd import harness as H
    from paper_2106_10207_amd import workloads as W

    if args.mode == "balance":
        print(json.dumps(bench_balance()), flush=True)
        return

    if args.summarize_trace:
        print(summarize_trace(args.summarize_trace, args.workload))
        return

    if args.summarize_counters:
        for f in summarize_counters(args.summarize_counters, args.workload, args.mode):
            print(f)
        return

    if args.copy_probe:
        a = torch.ones(args.copy_probe // 4, device="cuda")
        b = torch.empty_like(a)
        for _ in range(10):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": args.copy_probe, "launches": 10}))
        return

    wl = W.WORKLOADS[args.workload]
    torch.cuda.set_device(0)
    D.load()
    if args.mode == "group":
        print(json.dumps(bench_group(args, wl)), flush=True)
        return
    if args.mode == "accumulate":
        print(json.dumps(bench_accumulate(args, wl)), flush=True)
        return
    dr = H.DeviceRound(wl, "cuda", keep_local_grad=True, optimizer=args.optimizer,
                       fused_local=not args.separate_encode)
    bw = W.bandwidth_weights(wl)

    def eager_step():
        D.dedloc_partition(wl.P, wl.n_shards, bw, wl.shard_align)
        if args.separate_encode:
            dr.encode_local()
        dr.run()

    step = eager_step
    if args.graph:
        # the partition is host-only integer work, outside the graph
        side = torch.cuda.Stream()
        graph = torch.cuda.CUDAGraph()
        eager_step()
        torch.cuda.synchronize()
        with torch.cuda.graph(graph, stream=side):
            if args.separate_encode:
                dr.encode_local()
            dr.call(stream=side)

        def step():
            D.dedloc_partition(wl.P, wl.n_shards, bw, wl.shard_align)
            graph.replay()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # timed region: K steps bracketed by device synchronisation, HIP events
    # on the stream every kernel is launched on
    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    ms_per_step = ev0.elapsed_time(ev1) / args.steps

    # same K steps again with per-kernel events (roofline of the dominant kernel)
    D.dedloc_profile_begin(64 * args.steps + 64)
    for _ in range(args.steps):
        eager_step()
    prof = D.dedloc_profile_end()
    kname, roof, per_kernel = kernel_roofline(dr, prof, args.steps)
    roof["traffic"], roof["traffic_source"] = measured_traffic(kname, wl.name)
    roof["traffic_kind"] = ("FETCH_SIZE + WRITE_SIZE: bytes between the L2 caches and the fabric "
                            "(Infinity Cache hits included, so not DRAM bytes), calibrated on a plain copy")
    if kname.endswith("fused_fp16") and not dr.local_in_kernel and roof["traffic"] is not None:
        # the committed counters were taken with the local peer's encode
        # inside this pass, which moves 4P more bytes
        roof["traffic"], roof["traffic_source"] = None, roof["traffic_source"] + " (other launch: local encode inside)"

    # Back-to-back steps let the 256 MB Infinity Cache keep part of one
    # step's data for the next.  The same steps, each timed alone after
    # reading a 1 GiB buffer (which evicts it with clean lines), give the
    # cold-cache figure.
    flush = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
    sink = torch.empty((), device="cuda")
    evs = []
    for _ in range(args.steps):
        torch.sum(flush, dim=0, out=sink)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        step()
        b.record(stream)
        evs.append((a, b))
    torch.cuda.synchronize()
    cold_ms = sum(a.elapsed_time(b) for a, b in evs) / args.steps
    del flush

    # the round alone (every message, the local one included, encoded
    # beforehand): the time the round's compulsory bytes are quoted against
    for _ in range(2):
        dr.call_round_only()
    torch.cuda.synchronize()
    ev0.record(stream)
    for _ in range(args.steps):
        dr.call_round_only()
    ev1.record(stream)
    torch.cuda.synchronize()
    round_ms = ev0.elapsed_time(ev1) / args.steps

    # the round alone, each call timed after the cache flush
    flush = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
    evs = []
    for _ in range(args.steps):
        torch.sum(flush, dim=0, out=sink)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        dr.call_round_only()
        b.record(stream)
        evs.append((a, b))
    torch.cuda.synchronize()
    round_cold_ms = sum(a.elapsed_time(b) for a, b in evs) / args.steps
    del flush

    # the round's own compulsory bytes over the round alone, warm and cold:
    # the figures the 70% target is about (the kernel figure above is the
    # dominant pass's)
    roof["round"] = {
        "compulsory_bytes": dr.bytes_round(),
        "frac_warm": round(dr.bytes_round() / (round_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
        "frac_cold": round(dr.bytes_round() / (round_cold_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
    }

    t = ms_per_step * 1e-3
    peer_bytes = dr.bytes_peer_input()
    alg_bytes = dr.bytes_step()
    out = {
        "metric": "reduce+LAMB round GB/s of peer input (fraction of HBM peak); params/s",
        "value": round(peer_bytes / t / 1e9, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": wl.name,
            "params": wl.P,
            "tensors": wl.n_tensors,
            "peers": wl.n_peers,
            "active_peers": int(np.count_nonzero(dr.counts)),
            "wire": wl.codec,
            "shards": wl.n_shards,
            "optimizer": args.optimizer,
            "graph": bool(args.graph),
            "local_encode": "separate" if args.separate_encode else "fused",
            "parallelism": "single GPU; peers are HBM regions",
        },
        "params_per_s": round(wl.P / t, 1),
        "cold_cache": {"ms_per_step": round(cold_ms, 5),
                       "value": round(peer_bytes / (cold_ms * 1e-3) / 1e9, 2),
                       "algorithmic_frac_of_peak": round(alg_bytes / (cold_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4)},
        "round_only": {"ms": round(round_ms, 5), "compulsory_bytes": dr.bytes_round(),
                       "algorithmic_frac_of_peak": round(dr.bytes_round() / (round_ms * 1e-3) / 1e9
                                                         / HBM_PEAK_GBPS, 4)},
        "round_only_cold": {"ms": round(round_cold_ms, 5),
                            "algorithmic_frac_of_peak": round(dr.bytes_round() / (round_cold_ms * 1e-3) / 1e9
                                                              / HBM_PEAK_GBPS, 4)},
        "algorithmic_GBps": round(alg_bytes / t / 1e9, 2),
        "algorithmic_frac_of_peak": round(alg_bytes / t / 1e9 / HBM_PEAK_GBPS, 4),
        "roofline": roof,
        "kernels": per_kernel,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, dr, args.cpu_reps)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
