#!/usr/bin/env python3
"""Benchmark of region attribution over marker traces on one MI355X.

Workload: the large skewed trace -- 2^28 records of 16 B (4 GiB), 2048 blocks
x 16 warps = 32768 contexts with Zipf(1.2) record counts, 1024 regions, depth
<= 8, 1% malformed markers, 40-bit timestamps, 4 region classes over 2048
groups -- generated with a fixed seed, resident in HBM before timing.

One step = one call of the whole path (argus_attr_run): validate, sort,
match, exclusive times, per-region statistics, ambiguity counts and the
class-overlap sweep, with instance and exclusive-time outputs written.
`value` = records attributed per second over the timed steps.

Also reported: the roofline of the dominant kernel (algorithmic bytes per
launch / its average launch time vs 8 TB/s HBM; the launch times come from HIP
events recorded on the run's stream around that kernel only, during the timed
steps), a per-launch breakdown from instrumented steps before the timed ones
(an event after every launch), the whole pipeline's algorithmic bytes per
record and GB/s, practical HBM ceilings (copy, fill, read) measured in the same
process, and the CPU oracle timed on the same trace (1 core).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
METRIC = "marker records attributed/sec (sort+match+aggregate) + achieved HBM GB/s"
WORKLOADS = {
    5: "large skewed trace: 2^28 x 16 B records, 2048x16 warps (32768 contexts, Zipf 1.2), "
       "1024 regions, depth<=8, 1% malformed, 4 classes x 2048 groups",
    4: "compute/comm overlap trace: 2^25 records, 256x8 warps, 2 classes x 256 groups",
    3: "decode-megakernel trace: 2^26 records less 0.1% dropped ENDs, 256x16 warps, 177 regions",
    2: "persistent-GEMM trace: 2^24 records, 256x8 warps, 12 regions",
    1: "tiny well-formed trace: 2^16 records, 8x4 warps",
}


def err(*a):
    print(*a, file=sys.stderr, flush=True)


def byte_model(name: str, c: dict, plan: dict, R: int, K: int, G: int, flags: int) -> float:
    """Algorithmic bytes moved by one launch (element data read and written;
    look-back status and histogram traffic excluded)."""
    n, nv, nb, nev = c["n"], c["nv"], c["nb"], plan["n_ev"]
    wide = plan["rec_wide"]
    if name == "ingest":
        # records in; runs of one context out (one word per run, a count per chunk)
        return 16.0 * n + 8.0 * plan.get("n_runs", 0) + 4.0 * (-(-n // 256))
    if name.startswith("radix_") or name.startswith("ev_radix_"):
        ev = name.startswith("ev_")
        slots = plan["ev_slots"] if ev else plan["rec_slots"]
        idx = {"ctx0": 0, "ctx1": 1, "ctx2": 2, "ctx3": 3, "ts0": 4, "ts1": 5, "ts2": 6, "ts3": 7,
               "ts4": 8, "ts5": 9, "ts6": 10, "ts7": 11, "ctx0b": 12, "ctx1b": 13, "ctx2b": 14,
               "ctx3b": 15}
        if ev:
            tail = name[len("ev_radix_"):]
            slot = int(tail[2:]) if tail.startswith("ts") else (8 + int(tail[1:]) if tail.startswith("g") else 99)
        else:
            slot = idx[name[len("radix_"):]]
        if slot >= 16 or not slots[slot]["active"]:
            return 0.0
        out_n = int(slots[slot]["n_out"])  # records, events, or runs of one context
        elem = 12.0 + (4.0 if (wide and not ev) else 0.0)
        src = int(slots[slot]["src"])
        if src == 2:  # first pass: raw records / instances
            return (16.0 * n if not ev else 32.0 * nb) + elem * out_n
        return 2.0 * elem * out_n
    runs = plan.get("runs", 0)
    if name == "runs_base":  # chunk run counts scanned (read twice, written once)
        return 12.0 * (-(-n // 256)) if runs else 0.0
    if name == "runs_compact":  # raw runs and counts in; run keys, ids and lengths out
        return (12.0 * (-(-n // 256)) + 24.0 * plan["n_runs"]) if runs else 0.0
    if name == "runs_pos":  # run ids and lengths in (twice), positions out
        return 20.0 * plan["n_runs"] if runs else 0.0
    if name == "runs_scatter":  # raw records in, packed keys and payloads out
        return (16.0 * n + 12.0 * nv) if runs else 0.0
    if name == "tile_sums":
        # sorted keys and payloads: order check and per-tile depth maps (record radix path)
        return 0.0 if runs else (12.0 + (4.0 if wide else 0.0)) * nv
    if name == "runs_check":  # each run's count and position, the two keys where it meets the one before
        return 24.0 * plan["n_runs"] if runs else 0.0
    if name == "tile_sums_runs":  # sorted payloads (kind and context-start bits)
        return 4.0 * nv if runs else 0.0
    if name == "tile_sums_full":
        return (12.0 + (4.0 if wide else 0.0)) * nv if plan["unsorted"] else 0.0
    if name == "ts_hist":
        return 8.0 * nv if plan["unsorted"] else 0.0
    ev_words = K > 0 and plan["rec_ts_bits"] + (max(G - 1, 0)).bit_length() + 5 <= 64
    if name == "match":
        # sorted keys (+ context words) in; instances and one event word per record out
        return (12.0 + (4.0 if wide else 0.0) + (8.0 if ev_words else 0.0)) * nv + 40.0 * nb
    if name.startswith("merge") and name[5:].isdigit():
        # passes before the last: read and write one word per event
        return 16.0 * plan["merge_end"] if int(name[5:]) + 1 < plan["merge_rounds"] and plan["ev_merge"] else 0.0
    if name == "merge_sweep":
        # last pass: reads one word per event, merges and sweeps without storing
        return 8.0 * plan["merge_end"] if plan["ev_merge"] else 0.0
    if name == "agg":
        # instances and their exclusive times in (the caller's exclusive output
        # already holds them), histogram keys out when they do not fit in LDS
        return 40.0 * nb + (4.0 * nb if R > 167 else 0.0)
    if name == "hist":
        # the histogram keys are read from HBM once; the region slices of one
        # key range re-read them from the L2 of the XCD that holds them
        return 4.0 * nb if R > 167 else 0.0
    if name == "ev_hist":
        return 32.0 * nb
    if name == "sweep":
        return 0.0 if plan["ev_merge"] else 12.0 * nev
    if name == "init":
        return 8.0 * (R * 142 + (-(-n // 4096)) * 256 + (-(-nv // 2048)) * 4 + (-(-n // 2048)) * 8)
    if name == "ev_clear":
        return 8.0 * (-(-2 * nb // 4096)) * 256
    return 0.0


def traffic_for(kernel: str, n_begin: int):
    """HBM bytes per launch measured by rocprofv3 counters, if the committed
    measurement is for the current source of that kernel and for this trace
    (same number of BEGIN records)."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path)).get(kernel)
        if not rec:
            return None
        src = os.path.join(ROOT, "paper_2609_12299_amd", "csrc", rec["source"])
        sha = hashlib.sha256(open(src, "rb").read()).hexdigest()
        if sha != rec["source_sha256"] or int(rec.get("n_begin", -1)) != n_begin:
            return None
        return float(rec["bytes_per_launch"])
    except Exception:  # noqa: BLE001
        return None


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(records: np.ndarray, d: dict, sample: int, params: dict) -> dict:
    """The oracle, single-threaded, on the first `sample` records of the same
    trace the GPU runs (all of them by default)."""
    import oracle
    sub = records if sample >= len(records) else np.ascontiguousarray(records[:sample])
    t0 = time.perf_counter()
    oracle.run(sub, params["num_regions"], params["num_classes"], params["region_class"],
               params["group_shift"], params["num_groups"], instances=True)
    t = time.perf_counter() - t0
    what = ("all records of the trace the GPU runs" if sample >= len(records)
            else f"first {sample} records ({sample * 16 >> 20} MiB) of the trace the GPU runs")
    return {"value": sample / t, "unit": "records/s", "cores": 1, "kind": "oracle",
            "seconds": round(t, 3), "host_cpus": os.cpu_count(), "cpu_model": cpu_model(),
            "sample": f"{what}; single-threaded C++ oracle (validate, stable sort, stack replay, "
                      "sums, sweep) on 1 of the host's cores"}


def hbm_ceiling(dev, nbytes: int = 4 << 30, reps: int = 5) -> dict:
    """Practical HBM ceilings on this GPU: a plain device copy (read + write),
    a fill (write only) and a read-only reduction over `nbytes`, timed with
    events on the current stream (torch's own kernels)."""
    import torch
    src = torch.empty(nbytes // 8, dtype=torch.int64, device=dev).fill_(1)
    dst = torch.empty_like(src)
    res = {}

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps * 1e-3

    res["copy_gbs"] = round(2 * nbytes / timed(lambda: dst.copy_(src)) / 1e9, 1)
    res["fill_gbs"] = round(nbytes / timed(lambda: dst.fill_(3)) / 1e9, 1)
    res["read_gbs"] = round(nbytes / timed(lambda: src.sum()) / 1e9, 1)
    res["bytes"] = nbytes
    res["how"] = "torch copy_ (read+write), fill_ and sum of an int64 tensor, HIP events"
    del src, dst
    torch.cuda.empty_cache()
    return res


PART_DEFAULT_CONFIG = {"samples": 3, "scope": 5, "probes": 2, "handoffs": 3}


def bench_part(args, d: dict, rec_np: np.ndarray, dev) -> dict:
    """One of the steps that work on the instances of a run: PC-sample
    attribution, scoped statistics with iteration ordinals, the probe join,
    or the phase handoffs.  The run itself is done once, untimed; `value`
    is units per second of the timed calls (HIP events on the stream), with
    an algorithmic-byte model of the whole call."""
    import torch

    import tracegen
    from paper_2609_12299_amd import (RegionAttribution, attribute_samples, join_probes,
                                      phase_handoffs, scope_statistics)
    n = rec_np.shape[0]
    R = d["num_regions"]
    rec = torch.from_numpy(rec_np.reshape(-1)).to(dev)
    ra = RegionAttribution(R, d["num_classes"], d["region_class"], d["group_shift"],
                           d["num_groups"], max_records=n, device=dev)
    out = ra.run(rec)
    torch.cuda.synchronize()
    nb = int(out["counters"][4].item())
    inst, cnt = out["instances"], out["counters"][4:5]
    part = args.part
    if part == "samples":
        S, P = args.samples, args.pcs
        smp_np = tracegen.pc_samples(rec_np, S, P, R, seed=1)
        smp = torch.from_numpy(smp_np.view(np.uint8).reshape(-1)).to(dev)
        met = torch.from_numpy(np.stack([np.arange(P, dtype=np.float64) % 97, np.ones(P)])).to(dev)

        def call():
            return attribute_samples(inst, cnt, smp, R, P, metrics=met)
        units, unit_name = S, "samples"
        # each sample, its owner instance and a count update; the [P][R] table
        # cleared, read twice, alpha written and read (2 metrics)
        per_call = 56.0 * S + 8.0 * P * R * 6
        what = (f"{S} PC samples over {P} PCs (2 metrics) on the instances of the "
                f"{WORKLOADS[args.config]}")
    elif part == "scope":
        def call():
            return scope_statistics(inst, out["instance_excl"], cnt, R, iter_lo=0, iter_hi=15)
        units, unit_name = nb, "instances"
        if R <= 4096:
            # chunk-local ordinals (context and region half of each instance in,
            # ordinal out); the carry scan over the chunks' counts (R words per
            # chunk of 4096: written, read, read and written); statistics
            # (instance, exclusive time, ordinal in and out, histogram key out);
            # the histogram pass over the keys
            per_call = nb * (16.0 + 4.0 + 16.0 * R / 4096 + 32.0 + 8.0 + 4.0 + 4.0 + 4.0 + 4.0)
        else:
            passes = 2 if R > 256 else 1
            # sort passes; ordinals (sorted element in, pair out; pair in, ordinal
            # out); statistics (instance, exclusive time, ordinal in, histogram
            # key out); the histogram pass over the keys
            per_call = nb * (48.0 * passes + 24.0 + 12.0 + 48.0 + 4.0)
        what = f"iterations 0..15 of every region, on the instances of the {WORKLOADS[args.config]}"
    elif part == "probes":
        pr_np = tracegen.probes_for([1, 2, 7], d["blocks"] * d["warps"], 16, 5, seed=9)
        pr = torch.from_numpy(pr_np.view(np.uint8).reshape(-1)).to(dev)

        def call():
            return join_probes(inst, cnt, pr, R)
        units, unit_name = len(pr_np), "probes"

        def probe_bytes(r):
            # the reference sort pass(es); the join (probe and reference
            # instance in, outputs and sort element out); the sort passes the
            # library runs: those whose byte of the latency or the instance
            # code is not the same for every probe
            ref = r["ref"][:len(pr_np)].cpu().numpy().astype(np.uint64)
            joined = ref != np.uint64(0xFFFFFFFF)
            lat = np.where(joined, pr_np["t_end"] - pr_np["t_start"], np.uint64(0))
            # an unjoined probe's code is the instance capacity
            code = np.where(joined, ref, np.uint64(inst.shape[0]))

            def varying(v, nbytes):
                if len(v) == 0:
                    return 0
                d = np.bitwise_or.reduce(v) ^ np.bitwise_and.reduce(v)
                return sum(1 for k in range(nbytes) if (int(d) >> (8 * k)) & 0xFF)
            passes = varying(lat, 8) + varying(code, 4)
            return (nb * 48.0 * (2 if R > 256 else 1)
                    + len(pr_np) * (64.0 + 32.0 + 48.0 * passes))
        per_call = None
        what = (f"{len(pr_np)} probes (3 operations x 16 iterations x 5 repeats per warp) joined "
                f"to the {WORKLOADS[args.config]}")
    elif part == "handoffs":
        def call():
            return phase_handoffs(inst, cnt, R, level=1)
        units, unit_name = nb, "instances"
        # compaction (level word in, index out for level <= 1); pairs (index
        # and both instances in, for each level <= 1 instance); the per-parent
        # sums (one output word per instance)
        lv = inst.view(torch.int32).view(-1, 8)[:nb, 6]
        m = int(((lv >= 0) & (lv <= 1)).sum().item()) if nb else 0  # levels are below 2^31
        per_call = nb * (4.0 + 8.0) + m * (4.0 + 4.0 + 64.0)
        what = f"level-1 phases (operators within token steps) of the {WORKLOADS[args.config]}"
    else:
        raise ValueError(part)
    keep = [call() for _ in range(max(args.warmup, 1))]
    torch.cuda.synchronize()
    del keep
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    res = []
    e0.record()
    for _ in range(args.steps):
        res.append(call())
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    if per_call is None:
        per_call = probe_bytes(res[-1])
    del res
    ra.close()
    gbs = per_call / (ms * 1e-3) / 1e9
    return {
        "metric": f"{unit_name} per second ({part})", "value": units / (ms * 1e-3),
        "unit": f"{unit_name}/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f64" if part == "samples" else "u64",
        "data": "synthetic", "config": {"workload": what, "records": n, "instances": nb,
                                        "units": units, "regions": R},
        "roofline": {"bound": "hbm", "kernel": f"whole {part} call", "achieved": round(gbs, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4),
                     "traffic": None, "bytes_per_launch": per_call},
    }


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=0, choices=[0] + sorted(WORKLOADS),
                    help="workload (default: 5 for the run, the part's own otherwise)")
    ap.add_argument("--part", default="attr", choices=["attr", "samples", "scope", "probes",
                                                       "handoffs"],
                    help="attr: the whole attribution run (the headline); the others time one "
                         "step on the instances of a run")
    ap.add_argument("--samples", type=int, default=1 << 24, help="PC samples (--part samples)")
    ap.add_argument("--pcs", type=int, default=65536, help="PCs (--part samples)")
    ap.add_argument("--force-full-sort", action="store_true")
    ap.add_argument("--force-event-sort", action="store_true",
                    help="order overlap events with the radix sort instead of merging")
    ap.add_argument("--no-overlap", action="store_true",
                    help="run without the class-overlap step (num_classes = 0)")
    ap.add_argument("--graph", action="store_true",
                    help="also time the run captured once in a HIP graph and replayed")
    ap.add_argument("--no-ceiling", action="store_true",
                    help="skip the copy / fill / read ceiling measurement")
    ap.add_argument("--cpu-sample", type=int, default=0,
                    help="records the oracle runs on (0: all records of the trace)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--kernels", action="store_true", help="print per-launch timing to stderr")
    ap.add_argument("--profile-steps", type=int, default=3,
                    help="untimed steps with an event after every launch (per-kernel breakdown)")
    ap.add_argument("--copy-calibrate", action="store_true",
                    help="also run a plain 1 GiB device copy (reference for HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        err("bench.py measures one GPU: there is no multi-GPU path (the path would shard by "
            "context group with one all-reduce of the aggregates). Use --gpus 1.")
        return 2

    import torch

    import tracegen
    from paper_2609_12299_amd import RegionAttribution, load_library
    load_library()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")

    if args.config == 0:
        args.config = 5 if args.part == "attr" else PART_DEFAULT_CONFIG[args.part]
    t0 = time.perf_counter()
    d = tracegen.generate(args.config, threads=int(os.environ.get("OMP_NUM_THREADS", "16")))
    rec_np = d["records"]
    n = rec_np.shape[0]
    if args.part != "attr":
        err(f"generated config {args.config}: {n} records in {time.perf_counter() - t0:.1f}s")
        print(json.dumps(bench_part(args, d, rec_np, dev)), flush=True)
        return 0
    params = {k: d[k] for k in ("num_regions", "num_classes", "region_class", "group_shift",
                                "num_groups")}
    if args.no_overlap:
        params.update(num_classes=0, region_class=None, num_groups=0)
    err(f"generated config {args.config}: {n} records in {time.perf_counter() - t0:.1f}s")
    rec = torch.from_numpy(rec_np.reshape(-1)).to(dev)
    torch.cuda.synchronize()
    ra = RegionAttribution(params["num_regions"], params["num_classes"], params["region_class"],
                           params["group_shift"], params["num_groups"], max_records=n,
                           instances=True, instance_excl=True,
                           force_full_sort=args.force_full_sort,
                           force_event_sort=args.force_event_sort, device=dev)
    out = ra.alloc(n)
    for _ in range(max(args.warmup, 1)):
        ra.run(rec, out)
    torch.cuda.synchronize()
    cnt = out["counters"].cpu().numpy()
    assert int(cnt[31]) == 0, "internal error flag set"
    assert int(cnt[0]) == n
    err(f"warm: n_valid={int(cnt[1])} n_begin={int(cnt[4])} matched={int(cnt[9])} "
        f"max_level={int(cnt[14])}")

    if args.copy_calibrate:
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # Per-launch breakdown from instrumented steps outside the timed region
    # (an event after every launch); it names the dominant kernel.
    ra.set_timing(True)
    ra.kernel_times()  # discard
    for _ in range(args.profile_steps):
        ra.run(rec, out)
    times = ra.kernel_times()
    per = {}
    for name, ms in times:
        per.setdefault(name, []).append(ms)
    avg = {k: float(np.mean(v)) for k, v in per.items()}
    dom = max(avg, key=lambda k: avg[k])

    # Timed region: events only around the dominant kernel's launches, whose
    # durations give the roofline.
    ra.set_timing_filter(dom)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        ra.run(rec, out)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    dom_times = [ms for name, ms in ra.kernel_times() if name == dom]
    ra.set_timing_filter(None)
    ra.set_timing(False)
    plan = ra.plan()
    assert len(dom_times) == args.steps, f"expected {args.steps} timed launches of {dom}"
    avg[dom] = float(np.mean(dom_times))

    graph = None
    if args.graph:
        # the same run captured once and replayed: host launch work leaves the step
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            ra.run(rec, out)
        g.replay()
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        for _ in range(args.steps):
            g.replay()
        torch.cuda.synchronize()
        gms = (time.perf_counter() - t1) * 1e3 / args.steps
        graph = {"ms_per_step": round(gms, 4), "records_per_s": n / (gms * 1e-3)}
        gcnt = out["counters"].cpu().numpy()
        assert np.array_equal(gcnt, cnt), "graph replay changed the counters"
        del g

    c = dict(n=n, nv=int(cnt[1]), nb=int(cnt[4]))
    flags = ra.flags
    R, K, G = params["num_regions"], params["num_classes"], params["num_groups"]
    bytes_per = {k: byte_model(k, c, plan, R, K, G, flags) for k in avg}
    step_ms = elapsed * 1e3 / args.steps
    total_bytes = sum(bytes_per.values())
    achieved = bytes_per[dom] / (avg[dom] * 1e-3) / 1e9
    roofline = {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1),
                "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                "traffic": traffic_for(dom, c["nb"]), "avg_launch_ms": round(avg[dom], 4),
                "bytes_per_launch": bytes_per[dom]}
    if args.kernels:
        for k in sorted(avg, key=lambda k: -avg[k]):
            gbs = bytes_per[k] / (avg[k] * 1e-3) / 1e9 if avg[k] > 0 else 0.0
            err(f"  {k:16s} {avg[k]:8.4f} ms  {bytes_per[k] / 2**20:10.1f} MiB  {gbs:8.1f} GB/s")
        err(f"plan: unsorted={plan['unsorted']} n_ev={plan['n_ev']} ev_merge={plan['ev_merge']} "
            f"merge_rounds={plan['merge_rounds']} "
            f"rec_active={[int(s['pos']) for s in plan['rec_slots'] if s['active']]} "
            f"ev_active={[int(s['pos']) for s in plan['ev_slots'] if s['active']]}")

    result = {
        "metric": METRIC,
        "value": n * args.steps / elapsed,
        "unit": "records/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(step_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u64",
        "data": "synthetic",
        "config": {"workload": WORKLOADS[args.config] + ("; overlap step off" if args.no_overlap else ""),
                   "records": n, "record_bytes": 16,
                   "contexts": int(d["blocks"]) * int(d["warps"]), "regions": R, "classes": K,
                   "groups": G, "overlap_step": K > 0,
                   "force_full_sort": bool(args.force_full_sort),
                   "force_event_sort": bool(args.force_event_sort)},
        "trace": {"valid": c["nv"], "begins": c["nb"], "matched": int(cnt[9]),
                  "mismatched": int(cnt[10]), "unclosed": int(cnt[11]), "orphan_ends": int(cnt[12]),
                  "max_level": int(cnt[14])},
        "pipeline": {"bytes_per_record": round(total_bytes / n, 2),
                     "achieved_gbs": round(total_bytes / (step_ms * 1e-3) / 1e9, 1),
                     "frac_of_peak": round(total_bytes / (step_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                     "full_sort": bool(plan["unsorted"]),
                     "events": f"merged in {plan['merge_rounds']} passes" if plan["ev_merge"] else "radix sort"},
        "roofline": roofline,
        # per launch; the dominant kernel's from the timed steps, the others
        # from the instrumented steps before them
        "kernels_ms": {k: round(v, 4) for k, v in sorted(avg.items(), key=lambda kv: -kv[1])
                       if v >= 0.01},
    }
    if graph is not None:
        result["graph"] = graph
    if not args.no_ceiling:
        result["hbm_ceiling"] = hbm_ceiling(dev)
    if not args.no_cpu_baseline:
        sample = min(args.cpu_sample, n) if args.cpu_sample > 0 else n
        err(f"cpu baseline: oracle on {sample} records ...")
        result["cpu_baseline"] = cpu_baseline(rec_np, d, sample, params)
    print(json.dumps(result), flush=True)
    ra.close()
    return 0


if __name__ == "__main__":
    sys.exit(main())
