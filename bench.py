#!/usr/bin/env python3
"""Throughput of expand + FIFO batch + ordered gather on one MI355X.

One step = the whole path over one batch of the synthetic workload: ro_expand
(counts -> offsets and lineage keys), ro_batch over the ready queue for the
dispatched children, ro_batch over the list of children sealed before
dispatch, and ro_gather of all reports into parent slots.  Inputs
(counts, ready queue, masks, report states, report offsets and record bytes)
are resident in HBM before the timed region; record bytes are generated
untimed by the generator's device fill.

Prints one JSON line.  The default workload is 100,000 parents with Zipf(1.2)
child counts truncated to [1, 10^4] (about 41.1M children) and lognormal
16-4096-byte records (about 25 GB surviving payload).
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

HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E, published


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--parents", type=int, default=100_000, help="parents of the Zipf(1.2) workload")
    ap.add_argument("--cpu-parents", type=int, default=100_000,
                    help="parents in the CPU-oracle sample (same distributions; about 10 s of one core)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="also run a plain device copy of this many MiB (counter calibration)")
    ap.add_argument("--rocprof-summary", metavar="DIR", default=None,
                    help="print per-kernel averages from rocprofv3 CSV output under DIR and exit")
    return ap.parse_args()


# kernel whose HBM counters feed roofline.traffic, the file holding them, and
# the source they were taken from (a changed source voids the figure)
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gather_copy_zipf41M_counters.txt")
TRAFFIC_SOURCE = os.path.join(ROOT, "paper_2609_18703_amd", "csrc", "k_gather.hip")


def source_sha256(path):
    import hashlib
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def traffic_from_profile():
    """Calibrated HBM bytes per launch of the copy kernel, or None when the
    counters were taken on a different kernel source."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    vals = {}
    for line in open(TRAFFIC_FILE):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    if vals.get("source_sha256") != source_sha256(TRAFFIC_SOURCE):
        return None
    try:
        return int(vals["calibrated_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def rocprof_summary(root):
    """Per-kernel averages from rocprofv3 --output-format csv files under root."""
    import csv
    import glob
    from collections import defaultdict
    dur = defaultdict(list)
    ctr = defaultdict(list)
    for path in glob.glob(os.path.join(root, "**", "*kernel_trace.csv"), recursive=True):
        for row in csv.DictReader(open(path)):
            dur[row["Kernel_Name"].split("(")[0]].append(int(row["End_Timestamp"]) - int(row["Start_Timestamp"]))
    for path in glob.glob(os.path.join(root, "**", "*counter_collection.csv"), recursive=True):
        for row in csv.DictReader(open(path)):
            ctr[(row["Kernel_Name"].split("(")[0], row["Counter_Name"])].append(float(row["Counter_Value"]))
    if dur:
        print(f"{'kernel':48s} {'calls':>6s} {'avg_us':>12s} {'total_ms':>10s}")
        for k, v in sorted(dur.items(), key=lambda kv: -sum(kv[1])):
            print(f"{k[:48]:48s} {len(v):6d} {sum(v) / len(v) / 1e3:12.2f} {sum(v) / 1e6:10.3f}")
    if ctr:
        print(f"{'kernel':48s} {'counter':12s} {'n':>4s} {'avg_KiB':>14s}")
        for (k, c), v in sorted(ctr.items()):
            print(f"{k[:48]:48s} {c:12s} {len(v):4d} {sum(v) / len(v):14.1f}")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def alg_bytes(kind, P, N, M, S):
    """Algorithmic HBM bytes of one launch of each kernel kind.

    P parents, N children, M dispatched children, S surviving payload bytes.
    Reads and writes the path must do, counted once; cache-resident lookups
    (offsets searches, per-parent atomics) are not counted.
    """
    nsub = (N + 1023) // 1024
    return {
        "expand_scan": 12 * P + 8,                   # counts in, offsets out
        "expand_tags": 8 * N,                        # (parent, ordinal) out
        "batch_samples": 0,
        "batch": None,                               # per call, see below
        "gather_scatter": 17 * N + 16 * N + 12 * P,  # report tags/state/offsets in, canonical slot out, counters zeroed
        "gather_scan": 16 * N + 8 * P + 8 * nsub,    # canonical slots in, slot offsets and sub-tile bases out
        "gather_finalize": 30 * P,
        "gather_copy": 16 * N + 8 * nsub + 2 * S,    # canonical slots + payload in and out
        "gather_reset": 0,
    }[kind]


def main():
    args = parse()
    if args.rocprof_summary:
        rocprof_summary(args.rocprof_summary)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: this build has no multi-GPU path "
              f"(asked for --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)

    import torch
    import workloads as W
    from workloads import device as D
    import paper_2609_18703_amd as R
    from paper_2609_18703_amd import pipeline as PL

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)

    t0 = time.time()
    c = W.config2(n_parents=args.parents)
    r = c.reports
    P, N, M = c.n_parents, c.n_children, c.n_dispatched
    S = int(r.off[-1])
    log(f"[bench] workload: P={P} N={N} dispatched={M} surviving bytes={S} (gen {time.time() - t0:.1f}s)")

    data = torch.empty(max(S, 1), dtype=torch.uint8, device="cuda")
    D.fill_records_dev(D.to_dev(r.seed), D.to_dev(r.off), data)
    b = PL.SingleLevelBuffers(
        D.to_dev(c.counts), D.to_dev(c.queue.view(np.int32)), D.to_dev(c.keep), D.to_dev(c.sealed_ids.view(np.int32)),
        D.to_dev(r.state), D.to_dev(r.off), data, N, M, c.batch_size, out_cap=S)
    torch.cuda.synchronize()
    log(f"[bench] staged in HBM ({time.time() - t0:.1f}s)")

    ctx = R.Context()
    ctx.reserve(N, P, N)
    for _ in range(args.warmup):
        PL.single_level(ctx, b)
    ctx.check("warmup")
    torch.cuda.synchronize()
    log("[bench] warmup done")

    # timed region: K steps on the context's (torch's current) stream
    ctx.trace(True)
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record()
    for _ in range(args.steps):
        PL.single_level(ctx, b)
    ev1.record()
    torch.cuda.synchronize()
    ms_total = ev0.elapsed_time(ev1)
    kern = ctx.trace_read()
    ctx.trace(False)
    ctx.check("timed steps")
    ms_step = ms_total / args.steps
    log(f"[bench] {args.steps} steps: {ms_step:.3f} ms/step")

    # sanity: slot offsets and counts of the last step
    tot = int(b.out_off[P].item())
    assert tot == S, (tot, S)

    # per-kernel algorithmic rates
    per_kernel = {}
    total_alg = 0
    for k, (n_launch, ms) in kern.items():
        if k == "batch":
            # two launches per step: the ready queue (N entries in, M tags out) and
            # the sealed list (N-M entries in, N-M tags out)
            per_step = 5 * N + 4 * (N - M) + 8 * N
            ab = per_step / 2
        else:
            ab = alg_bytes(k, P, N, M, S)
        avg_ms = ms / n_launch
        per_kernel[k] = {"launches_per_step": n_launch / args.steps, "avg_ms": round(avg_ms, 4),
                         "alg_GBps": round(ab / (avg_ms * 1e-3) / 1e9, 1) if avg_ms > 0 and ab else None}
        total_alg += ab * n_launch / args.steps
    dom = max(kern.items(), key=lambda kv: kv[1][1])[0]
    dom_avg_ms = kern[dom][1] / kern[dom][0]
    dom_bytes = alg_bytes(dom, P, N, M, S) if dom != "batch" else 9 * N
    achieved = dom_bytes / (dom_avg_ms * 1e-3) / 1e9

    result = {
        "metric": "children/sec through expand+batch+gather; achieved HBM GB/s vs peak",
        "value": round(N / (ms_step * 1e-3), 1),
        "unit": "children/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u8",
        "data": "synthetic",
        "config": {
            "workload": f"single-level Zipf(1.2) fan-out: {P} parents, counts truncated to [1,10000], "
                        f"{N} children, lognormal(6,1) records clipped to [16,4096] B, 3% failed, "
                        f"2% skipped, random ready order, B={c.batch_size}, seed 1",
            "parents": P, "children": N, "dispatched": M, "surviving_bytes": S,
            "batch_size": c.batch_size,
        },
        "roofline": {
            "bound": "hbm", "kernel": dom, "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
            "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
            "traffic": traffic_from_profile() if dom == "gather_copy" else None,
            "alg_bytes_per_launch": dom_bytes, "avg_launch_ms": round(dom_avg_ms, 4),
        },
        "step_alg_GBps": round(total_alg / (ms_step * 1e-3) / 1e9, 1),
        "step_frac_of_peak": round(total_alg / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
        "kernels": per_kernel,
    }

    if args.calib_copy_mib:
        n = args.calib_copy_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(5):
            dst.copy_(src)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / 5
        result["calib_copy"] = {"bytes": n, "avg_ms": round(ms, 4), "GBps": round(2 * n / (ms * 1e-3) / 1e9, 1)}
        del src, dst

    del b, data
    torch.cuda.empty_cache()

    if not args.no_cpu:
        result["cpu_baseline"] = cpu_baseline(args.cpu_parents)

    print(json.dumps(result), flush=True)


def cpu_baseline(n_parents):
    """The oracle, single threaded, on a bounded sample of the same workload."""
    import torch
    import oracle as O
    import workloads as W
    from workloads import device as D

    c = W.config2(n_parents=n_parents)
    r = c.reports
    S = int(r.off[-1])
    dev = torch.empty(max(S, 1), dtype=torch.uint8, device="cuda")
    D.fill_records_dev(D.to_dev(r.seed), D.to_dev(r.off), dev)
    data = dev.cpu().numpy()
    del dev
    L = O.lib()
    t = time.perf_counter()
    offs, cp, co = O.expand(c.counts, L=L)
    b1 = O.batch(c.queue, c.keep, offs, c.batch_size, L=L)
    b2 = O.batch(c.sealed_ids, None, offs, c.batch_size, L=L)
    par = np.concatenate([b1[1], b2[1]])
    ordi = np.concatenate([b1[2], b2[2]])
    g = O.gather(par, ordi, r.state, r.off, data, offs, L=L)
    dt = time.perf_counter() - t
    assert int(g["out_off"][-1]) == S
    log(f"[bench] cpu oracle: {c.n_children} children in {dt:.2f}s")
    return {"value": round(c.n_children / dt, 1), "unit": "children/s", "cores": 1, "kind": "oracle",
            "sample": f"same distributions with {n_parents} parents: {c.n_children} children, "
                      f"{S} surviving bytes; expand + 2 batches + gather, single thread",
            "seconds": round(dt, 2)}


if __name__ == "__main__":
    main()
