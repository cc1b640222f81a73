#!/usr/bin/env python3
"""Throughput of expand + FIFO batch + ordered gather on one MI355X.

One step = the whole path over one batch of a synthetic workload, with every
input resident in HBM before the timed region (record bytes are generated
untimed by the generator's device fill):

  zipf-single   (default) ro_expand, ro_batch over the ready queue for the
                dispatched children, ro_batch over the children sealed before
                dispatch, ro_gather of all reports into parent slots.
                100,000 parents, Zipf(1.2) child counts truncated to
                [1, 10^4] (about 41.1M children), lognormal 16-4096-byte
                records (about 25 GB surviving payload), B = 256.
  docs-nested   two levels: 20,000 documents -> pages -> regions, B = 512.
  videos-nested two levels: 2,000 videos -> clips -> frames, 1,024-B frames.
  stream-waves  10^7 children under 500,000 parents turning terminal over 50
                waves: per wave ro_batch, ro_stream_report, ro_stream_emit.
  docs-ops      F.filter over the ~2.7M regions of the documents workload and
                F.broadcast of a document-level Item to every region.
  zipf-pbatch   parent-bound reservation of zipf-single's ready queue (41M
                entries, B = 256): batches of up to B siblings of the first
                ready parent.
  zipf-fence    Grain phases and the generation fence over the dispatched
                children of zipf-single: reset, dispatch at generation 0,
                commit (with identical and conflicting repeats), retry of the
                2% lost attempts, dispatch at generation 1, commit (with
                stale generation-0 reports).
  zipf-canonical zipf-single with every child ready in canonical order: the
                reports and their records arrive in slot order, so the
                gather reads sequentially (the path's best-case ordering,
                for comparison with the random order of zipf-single).

Prints one JSON line.  Children/s counts every child entity created at every
level (pages + regions, clips + frames).  With the default workload the line
also carries, under "docs_nested", the same measurement of the two-level
documents workload (its own roofline, config and CPU baseline): the
single-level Zipf workload and the documents workload are the two readings
of the throughput target's "config 2".
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E, published
WORKLOADS = ("zipf-single", "docs-nested", "videos-nested", "stream-waves", "docs-ops", "zipf-fence",
             "zipf-pbatch", "zipf-canonical")


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", choices=WORKLOADS, default="zipf-single")
    ap.add_argument("--parents", type=int, default=None,
                    help="top-level parents (default: the workload's own size)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-docs", action="store_true",
                    help="with the default workload, skip the second line of the documents workload")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="also run a plain device copy of this many MiB (counter calibration)")
    ap.add_argument("--rocprof-summary", metavar="DIR", default=None,
                    help="print per-kernel averages from rocprofv3 CSV output under DIR and exit")
    return ap.parse_args()


# kernel whose HBM counters feed roofline.traffic, the workload and file
# holding them, and the source they were taken from (a changed source voids
# the figure)
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gather_copy_zipf41M_counters.txt")
TRAFFIC_SOURCES = [os.path.join(ROOT, "paper_2609_18703_amd", "csrc", f)
                   for f in ("k_gather.hip", "ro_copy.h", "ro_device.h", "ro_internal.h")]
TRAFFIC_WORKLOAD = ("zipf-single", "gather_copy")


def source_sha256(paths=TRAFFIC_SOURCES):
    """SHA-256 over the copy kernel's sources, concatenated in order."""
    import hashlib
    h = hashlib.sha256()
    for path in paths:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


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
    if vals.get("source_sha256") != source_sha256():
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


def cdiv(a, b):
    return (a + b - 1) // b


# ---------------------------------------------------------------- algorithmic bytes
#
# Reads and writes the path must do, counted once per step and per kernel
# kind; cache-resident lookups (offsets searches, per-parent atomics, seen
# bits) are not counted.  A kind launched several times per step sums its
# launches.

def _gather_bytes(P, N, S):
    """One ro_gather of N reports into P parents moving S payload bytes."""
    nsub = cdiv(N, 256)
    return {
        # report parent/ordinal/state/offset in, canonical 16-B slot out, counters zeroed
        "gather_scatter": 33 * N + 12 * P,
        # canonical slots in, parent slot offsets and sub-tile bases out
        "gather_scan": 16 * N + 8 * P + 8 * nsub,
        # counters and offsets in, complete and state out
        "gather_finalize": 22 * P,
        # canonical slots and sub-tile bases in, payload read and written
        "gather_copy": 16 * N + 8 * nsub + 2 * S,
    }


def _add(acc, d):
    for k, v in d.items():
        acc[k] = acc.get(k, 0) + v
    return acc


def alg_single(P, N, M, S):
    a = {"expand_scan": 12 * P + 8, "expand_tags": 8 * N,
         "batch_samples": 2 * 4 * cdiv(N, 64),            # coarse child->parent map, per batch call
         # ready queue: ids + mask in, tags of M out; sealed list: ids in, tags out
         "batch": 5 * N + 8 * M + 12 * (N - M)}
    return _add(a, _gather_bytes(P, N, S))


def alg_nested(P1, N1, N2, S2, S1, upper_in_place):
    """Two levels; when every mid slot survives, the top slots are the mid
    slots as they lie, so the top level moves no payload (in-place gather)."""
    a = {"expand_scan": 12 * P1 + 12 * N1 + 16, "expand_tags": 8 * N1 + 8 * N2,
         "batch_samples": 4 * cdiv(N1, 64) + 4 * cdiv(N2, 64),
         "batch": 12 * N1 + 12 * N2}
    _add(a, _gather_bytes(N1, N2, S2))
    return _add(a, _gather_bytes(P1, N1, 0 if upper_in_place else S1))


def alg_stream(P, N, S, n_waves, emit_wave):
    """emit_wave[p]: the wave in which parent p completes."""
    nsub = cdiv(N, 256)
    alive = int((emit_wave.astype(np.int64) + 1).sum())   # parent-waves a parent is still open
    return {
        "expand_scan": 12 * P + 8,
        "batch_samples": n_waves * 4 * cdiv(N, 64),
        "batch": 12 * N,                                   # wave ids in, tags out
        "stream_report": 33 * N,                           # report in, canonical slot out
        # per wave: emitted flags of every parent, counters of the open ones;
        # once per parent: its emission record; virtual expansion: offsets in,
        # per-child slot map out
        "stream_select": n_waves * P + 20 * alive + 30 * P + 24 * P + 4 * N,
        "stream_scan": 20 * N + 8 * P + 8 * nsub,
        "stream_copy": 20 * N + 8 * nsub + 2 * S,
        "stream_finish": 16 * P,
        "misc": cdiv(N, 8) + 13 * P,                       # reset of seen bits, counters, flags
    }


# ---------------------------------------------------------------- workloads

class Job:
    """A staged workload: step() enqueues one step; alg maps kernel kinds to
    algorithmic bytes per step."""

    def __init__(self, name, step, children, alg, config, check, leaves=None, metric=None):
        self.name, self.step, self.children, self.alg = name, step, children, alg
        self.config, self.check, self.leaves = config, check, leaves
        self.metric = metric or "children/sec through expand+batch+gather; achieved HBM GB/s vs peak"


def stage_zipf(ctx, parents, canonical=False):
    """The single-level Zipf(1.2) fan-out (100,000 parents, 41.1M children,
    25.2 GB of surviving records).  With canonical=True every child becomes ready in canonical
    order, so the reports (and their records) arrive in slot order and the
    gather's reads are sequential: the same path at its best-case ordering."""
    import torch
    import workloads as W
    from workloads import device as D
    from paper_2609_18703_amd import pipeline as PL
    c = W.config2(n_parents=parents or 100_000, canonical_order=canonical)
    r = c.reports
    P, N, M = c.n_parents, c.n_children, c.n_dispatched
    S = int(r.off[-1])
    name = "zipf-canonical" if canonical else "zipf-single"
    log(f"[bench] {name}: P={P} N={N} dispatched={M} surviving bytes={S}")
    data = torch.empty(max(S, 1), dtype=torch.uint8, device="cuda")
    D.fill_records_dev(D.to_dev(r.seed), D.to_dev(r.off), data)
    b = PL.SingleLevelBuffers(
        D.to_dev(c.counts), D.to_dev(c.queue.view(np.int32)), D.to_dev(c.keep),
        D.to_dev(c.sealed_ids.view(np.int32)), D.to_dev(r.state), D.to_dev(r.off), data, N, M,
        c.batch_size, out_cap=S)
    ctx.reserve(N, P, N)

    def check():
        assert int(b.out_off[P].item()) == S

    cfg = {"workload": f"single-level Zipf(1.2) fan-out: {P} parents, counts truncated to [1,10000], "
                       f"{N} children, lognormal(6,1) records clipped to [16,4096] B, 3% failed, "
                       f"2% skipped, {'canonical' if canonical else 'random'} ready order, "
                       f"B={c.batch_size}, seed 1",
           "parents": P, "children": N, "dispatched": M, "surviving_bytes": S, "batch_size": c.batch_size}
    return Job(name, lambda: PL.single_level(ctx, b), N, alg_single(P, N, M, S), cfg, check)


def stage_nested(ctx, which, parents):
    import workloads as W
    from workloads import device as D
    from paper_2609_18703_amd import pipeline as PL
    if which == "docs-nested":
        n = W.config3(n_docs=parents or 20_000)
        desc = "two-level documents->pages->regions: {P} docs, pages lognormal(2.3,0.9) clipped to " \
               "[1,2000], regions Poisson(8)+1, records uniform [32,1024] B, all succeed, B=512, seed 2"
    else:
        n = W.config4(n_videos=parents or 2_000)
        desc = "two-level videos->clips->frames: {P} videos, clips Pareto(1.1, x_min 5) clipped to " \
               "[1,50000], frames uniform [16,300], 1024-B frames, 1% failed, B=1024, seed 3"
    r = n.reports
    P1, N1, N2 = len(n.counts1), len(n.queue1), len(n.queue2)
    S2 = int(r.off[-1])
    log(f"[bench] {which}: top={P1} mid={N1} leaves={N2} leaf bytes={S2}")
    # surviving bytes at the top level: mid slots whose leaves all succeeded
    off2 = np.concatenate([[0], np.cumsum(n.counts2.astype(np.int64))])
    ok_leaf = (n.states == W.SUCCESS)
    lens = np.where(ok_leaf, n.lengths, 0)
    mid_bytes = np.add.reduceat(lens, off2[:-1]) if N2 else np.zeros(N1, np.int64)
    mid_failed = np.add.reduceat((n.states == W.FAILED).astype(np.int64), off2[:-1]) if N2 else np.zeros(N1)
    mid_bytes = np.where(n.counts2 > 0, mid_bytes, 0)
    mid_failed = np.where(n.counts2 > 0, mid_failed, 0)
    S1 = int(mid_bytes[mid_failed == 0].sum())
    # no leaf fails: the top level aliases the mid bytes (nothing to move)
    in_place = S1 == S2 and not (n.states == W.FAILED).any()
    data = D.reports_data_dev(r)
    b = PL.NestedBuffers(D.to_dev(n.counts1), D.to_dev(n.queue1.view(np.int32)), n.batch1,
                         D.to_dev(n.counts2), D.to_dev(n.queue2.view(np.int32)), n.batch2,
                         D.to_dev(r.state), D.to_dev(r.off), data, N1, N2, upper_in_place=in_place)
    ctx.reserve(N2, max(N1, P1), N2)

    def check():
        assert int(b.mid_off[N1].item()) == S2 and int(b.top_off[P1].item()) == S1

    cfg = {"workload": desc.format(P=P1), "top_parents": P1, "mid_children": N1, "leaf_children": N2,
           "leaf_bytes": S2, "top_bytes": S1, "batch_size": [n.batch1, n.batch2], "upper_in_place": in_place}
    return Job(which, lambda: PL.nested(ctx, b), N1 + N2, alg_nested(P1, N1, N2, S2, S1, in_place), cfg,
               check, leaves=N2)


def stage_stream(ctx, parents):
    import torch
    import workloads as W
    from workloads import device as D
    from paper_2609_18703_amd import pipeline as PL
    P0 = parents or 500_000
    s = W.config5(n_parents=P0, n_children=20 * P0)
    P, N = s.n_parents, s.n_children
    total = int(s.wave_reports[-1].off[-1])
    log(f"[bench] stream-waves: P={P} N={N} waves={len(s.waves)} bytes={total}")
    arena = torch.empty(max(total, 1), dtype=torch.uint8, device="cuda")
    for rep in s.wave_reports:
        D.fill_records_dev(D.to_dev(rep.seed), D.to_dev(rep.off), arena)
    b = PL.StreamingBuffers(D.to_dev(s.counts), [D.to_dev(q.view(np.int32)) for q in s.waves],
                            [D.to_dev(rep.state) for rep in s.wave_reports],
                            [D.to_dev(rep.off) for rep in s.wave_reports], arena, N, s.batch_size, total)
    ctx.reserve(N, P, max(len(q) for q in s.waves))
    ctx.expand(b.counts, b.offsets)
    st = ctx.stream(b.offsets, N)
    # wave in which each parent completes
    wave_of = np.empty(N, np.int64)
    for w, q in enumerate(s.waves):
        wave_of[q] = w
    offs = np.concatenate([[0], np.cumsum(s.counts.astype(np.int64))])
    ew = np.maximum.reduceat(wave_of, offs[:-1]) if N else np.zeros(P, np.int64)
    ew = np.where(s.counts > 0, ew, 0)

    def step():
        PL.streaming(ctx, b, st=st)

    def check():
        # the last wave emits exactly the parents completing in it
        assert int(b.scalars[2].item()) == int((ew == len(s.waves) - 1).sum())

    cfg = {"workload": f"streaming completion: {P} parents, {N} children, rank-frequency Zipf(1.1) counts "
                       f"clipped to [1,100000], records uniform [64,512] B, all succeed, "
                       f"{len(s.waves)} waves of {N // len(s.waves)} in random order, B={s.batch_size}, seed 4",
           "parents": P, "children": N, "waves": len(s.waves), "bytes": total, "batch_size": s.batch_size}
    return Job("stream-waves", step, N, alg_stream(P, N, total, len(s.waves), ew), cfg, check)


def stage_ops(ctx, parents):
    import torch
    import workloads as W
    from workloads import device as D
    n = W.config3(n_docs=parents or 20_000)
    P1, N1, N2 = len(n.counts1), len(n.queue1), len(n.queue2)
    log(f"[bench] docs-ops: docs={P1} pages={N1} regions={N2}")
    rng = np.random.default_rng(7)
    st = np.array([0, 0, 0, 1, 2, 3], np.uint8)
    xs = D.to_dev(rng.choice(st, N2))
    ms = D.to_dev(rng.choice(st, N2))
    mv = D.to_dev((rng.random(N2) < 0.5).astype(np.uint8))
    doc_x = D.to_dev(rng.choice(st, P1))
    like = D.to_dev(n.states)
    o1 = torch.empty(P1 + 1, dtype=torch.int64, device="cuda")
    o2 = torch.empty(N1 + 1, dtype=torch.int64, device="cuda")
    p1 = torch.empty(N1, dtype=torch.int32, device="cuda")
    p2 = torch.empty(N2, dtype=torch.int32, device="cuda")
    ctx.reserve(N2, max(N1, P1), N2)
    ctx.expand(D.to_dev(n.counts1), o1, p1, None)
    ctx.expand(D.to_dev(n.counts2), o2, p2, None)
    fout = torch.empty(N2, dtype=torch.uint8, device="cuda")
    bst = torch.empty(N2, dtype=torch.uint8, device="cuda")
    banc = torch.empty(N2, dtype=torch.int32, device="cuda")

    def step():
        ctx.filter(xs, mv, fout, mask_state=ms)
        ctx.broadcast([p2, p1], doc_x, bst, banc, like)

    def check():
        assert int(fout.max().item()) <= 3 and int(bst.max().item()) <= 3

    cfg = {"workload": f"F.filter over {N2} regions (state, mask state, mask) and F.broadcast of a document "
                       f"Item to every region through two child->parent levels; documents workload, seed 2",
           "regions": N2, "pages": N1, "documents": P1}
    # filter: three state bytes in, one out; broadcast: region map, region state, ancestor and state out
    # (the page map and document states stay in cache)
    return Job("docs-ops", step, N2, {"filter": 4 * N2, "broadcast": 10 * N2}, cfg, check)


def alg_fence(P, N, M, L, n0, n1, rep_bytes):
    """Algorithmic bytes of one fence step: the grain fill (phase, generation
    and fence key, 16 B a child); dispatch and retry, 20 B an entry (id in,
    phase read and written, generation in or out); the first fence pass, 45 B
    a report (key, ordinal, state, generation, the next offset, the grain's
    phase and generation, the key's read and write) plus the offsets; the
    deciding pass, 30 B a report (key, ordinal, state, generation, fence key,
    grain generation, state out, phase out) plus the bytes of compared
    repeats."""
    return {"grains": 16 * N + 20 * (M + 2 * L),
            "fence_first": 45 * (n0 + n1) + 2 * 8 * (P + 1),
            "fence_decide": 30 * (n0 + n1) + 2 * 8 * (P + 1) + rep_bytes}


def stage_fence(ctx, parents):
    import torch
    import workloads as W
    from workloads import device as D
    c = W.config2(n_parents=parents or 100_000)
    f = W.fence_trace(c)
    P, N = c.n_parents, c.n_children
    M, L = len(f.dispatch0), len(f.lost)
    r0, r1 = f.rounds
    log(f"[bench] zipf-fence: P={P} N={N} dispatched={M} lost={L} reports={r0.n}+{r1.n} "
        f"repeats={f.n_repeat} conflicts={f.n_conflict} stale={f.n_stale}")
    offs = torch.empty(P + 1, dtype=torch.int64, device="cuda")
    ctx.expand(D.to_dev(c.counts), offs)

    def dev_round(r):
        d = dict(parent=D.to_dev(r.parent.view(np.int32)), ordinal=D.to_dev(r.ordinal.view(np.int32)),
                 state=D.to_dev(r.state), off=D.to_dev(r.off), gen=D.to_dev(r.generation.view(np.int32)),
                 out=torch.empty(max(r.n, 1), dtype=torch.uint8, device="cuda"),
                 cnt=torch.zeros(4, dtype=torch.int64, device="cuda"))
        d["data"] = D.reports_data_dev(r)
        return d

    d0, d1 = dev_round(r0), dev_round(r1)
    disp0 = D.to_dev(f.dispatch0.view(np.int32))
    lost = D.to_dev(f.lost.view(np.int32))
    gen0 = torch.empty(max(M, 1), dtype=torch.int32, device="cuda")
    gen1 = torch.empty(max(L, 1), dtype=torch.int32, device="cuda")
    g = ctx.grains(N)
    # bytes the deciding pass compares: both copies of every same-state,
    # same-length successful repeat
    lens0 = np.diff(r0.off)
    na = r0.n - f.n_repeat - f.n_conflict
    first_len = {}
    rep_bytes = 0
    key0 = r0.parent.astype(np.int64) << 32 | r0.ordinal
    pos = dict(zip(key0[:na].tolist(), range(na)))
    for i in range(na, r0.n):
        w = pos[int(key0[i])]
        if r0.state[i] == r0.state[w] == W.SUCCESS and lens0[i] == lens0[w]:
            rep_bytes += 2 * int(lens0[i])

    def commit(d, n):
        g.commit(d["parent"], d["ordinal"], d["state"], d["off"], d["data"], d["gen"], offs, d["out"], d["cnt"],
                 n=n)

    def step():
        g.reset()
        g.dispatch(disp0, gen0, n=M)
        commit(d0, r0.n)
        g.retry(lost, n=L)
        g.dispatch(lost, gen1, n=L)
        commit(d1, r1.n)

    def check():
        c0 = tuple(int(x) for x in d0["cnt"].cpu().numpy())
        c1 = tuple(int(x) for x in d1["cnt"].cpu().numpy())
        assert c0 == (na, 0, f.n_repeat, f.n_conflict), c0
        assert c1 == (L, f.n_stale, 0, 0), c1
        assert int(gen1[:L].max().item()) == 1 and int(gen0[:M].max().item()) == 0

    cfg = {"workload": f"generation fence over the dispatched children of the single-level Zipf(1.2) fan-out "
                       f"({P} parents, {N} children, {M} dispatched): 2% of attempts lost and retried at "
                       f"generation 1, 1% identical and 0.2% conflicting repeats, stale reports for half of "
                       f"the lost attempts, seeds 1 and 6",
           "parents": P, "children": N, "dispatched": M, "lost": L, "reports": [r0.n, r1.n],
           "repeats": f.n_repeat, "conflicts": f.n_conflict, "stale": f.n_stale}
    return Job("zipf-fence", step, M, alg_fence(P, N, M, L, r0.n, r1.n, rep_bytes), cfg, check,
               metric="children/sec through dispatch + generation-fenced commit over two attempts; "
                      "achieved HBM GB/s vs peak")


def stage_pbatch(ctx, parents):
    import torch
    import workloads as W
    from workloads import device as D
    c = W.config2(n_parents=parents or 100_000)
    P, N, M = c.n_parents, c.n_children, c.n_dispatched
    Q = len(c.queue)
    log(f"[bench] zipf-pbatch: P={P} N={N} queue={Q} ready={M} B={c.batch_size}")
    ctx.reserve(N, P, Q)
    offs = torch.empty(P + 1, dtype=torch.int64, device="cuda")
    ctx.expand(D.to_dev(c.counts), offs)
    q = D.to_dev(c.queue.view(np.int32))
    keep = D.to_dev(c.keep)
    oc = torch.empty(M, dtype=torch.int32, device="cuda")
    op = torch.empty(M, dtype=torch.int32, device="cuda")
    oo = torch.empty(M, dtype=torch.int32, device="cuda")
    boff = torch.empty(M + 1, dtype=torch.int64, device="cuda")
    sc = torch.zeros(2, dtype=torch.int64, device="cuda")
    # batches: one per started group of B siblings of a parent
    offs_h = np.concatenate([[0], np.cumsum(c.counts.astype(np.int64))])
    par = np.searchsorted(offs_h, c.queue[c.keep == 1].astype(np.int64), side="right") - 1
    n_b = int((-(-np.bincount(par, minlength=P) // c.batch_size)).sum())

    def step():
        ctx.batch_parent(q, keep, offs, c.batch_size, boff, oc, op, oo, sc[0:1], sc[1:2])

    def check():
        assert int(sc[0].item()) == M and int(sc[1].item()) == n_b

    cfg = {"workload": f"parent-bound reservation of the single-level Zipf(1.2) fan-out's ready queue: {P} "
                       f"parents, {N} children in random ready order, {M} ready (sealed ones masked), "
                       f"B={c.batch_size}, seed 1",
           "parents": P, "queue": Q, "ready": M, "batches": n_b, "batch_size": c.batch_size}
    bits = max(int(P - 1).bit_length(), 0)
    passes = max(-(-bits // 9), 1)
    tiles = -(-Q // 16384)                 # histogram columns: spans of 8 sort tiles
    hist = 512 * tiles if passes * 9 == bits or bits > 9 else (1 << bits) * tiles
    alg = {
        # compaction: queue id and ready flag in, child and parent out
        "batch": 5 * Q + 8 * M, "batch_samples": 4 * (N // 64),
        # radix passes: the histogram reads the keys; the first scatter reads
        # keys and compacted children and writes keys and (child, position)
        # values, later ones read and write keys and values
        "pbatch_sort": passes * 4 * M + 20 * M + (passes - 1) * 24 * M,
        "expand_scan": passes * 12 * hist,
        # bounds (keys in, group sizes cleared), group firsts (keys), group
        # scan (sizes in, batch numbers and offsets out), placement (keys,
        # values in; child, parent, ordinal out)
        "pbatch": 8 * M + 4 * M + 4 * M + 12 * n_b + 24 * M,
    }
    return Job("zipf-pbatch", step, M, alg, cfg, check,
               metric="children/sec through parent-bound reservation; achieved HBM GB/s vs peak")


# ---------------------------------------------------------------- main

def main():
    args = parse()
    if args.rocprof_summary:
        rocprof_summary(args.rocprof_summary)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: the library has no multi-GPU path "
              f"(asked for --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)

    import torch

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)

    # everything runs on a stream of its own: work on the null stream
    # synchronises implicitly with other streams and pays for it per launch
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        result = run(args)
    result["device"] = _device_info(torch)
    print(json.dumps(result), flush=True)


def run(args):
    """The workload of the line; for the default one (single-level Zipf) also
    the two-level documents workload, timed the same way, under the key
    "docs_nested": the two workloads a reading of "config 2" can mean."""
    result = run_workload(args, args.workload)
    second = args.workload == "zipf-single" and not args.no_docs
    if second:
        result["docs_nested"] = run_workload(args, "docs-nested")
    if not args.no_cpu:
        result["cpu_baseline"] = cpu_baseline(args.workload)
        if second:
            result["docs_nested"]["cpu_baseline"] = cpu_baseline("docs-nested")
    return result


def _device_info(torch):
    """Which GPU unit ran the line: the same build has measured about 6% apart
    on different MI355X units in its HBM-bound kernels."""
    props = torch.cuda.get_device_properties(0)
    info = {"name": props.name, "arch": getattr(props, "gcnArchName", "")}
    uuid = getattr(props, "uuid", None)
    if uuid is not None:
        info["uuid"] = str(uuid)
    return info


def run_workload(args, workload):
    import torch
    import paper_2609_18703_amd as R

    t0 = time.time()
    ctx = R.Context()
    parents = args.parents if workload == args.workload else None
    if workload in ("zipf-single", "zipf-canonical"):
        job = stage_zipf(ctx, parents, canonical=workload == "zipf-canonical")
    elif workload == "stream-waves":
        job = stage_stream(ctx, parents)
    elif workload == "docs-ops":
        job = stage_ops(ctx, parents)
    elif workload == "zipf-fence":
        job = stage_fence(ctx, parents)
    elif workload == "zipf-pbatch":
        job = stage_pbatch(ctx, parents)
    else:
        job = stage_nested(ctx, workload, parents)
    torch.cuda.synchronize()
    log(f"[bench] staged in HBM ({time.time() - t0:.1f}s)")

    for _ in range(args.warmup):
        job.step()
    ctx.check("warmup")
    torch.cuda.synchronize()
    log("[bench] warmup done")

    # timed region: K steps on the context's (torch's current) stream, one
    # event pair per step
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    evs[0].record()
    for i in range(args.steps):
        job.step()
        evs[i + 1].record()
    torch.cuda.synchronize()
    per_step = [evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)]
    ms_total = evs[0].elapsed_time(evs[-1])
    ctx.check("timed steps")
    ms_step = ms_total / args.steps
    log(f"[bench] {args.steps} steps: {ms_step:.3f} ms/step (median {float(np.median(per_step)):.3f}, "
        f"min {min(per_step):.3f})")
    job.check()

    # second timed region, K more steps with every kernel bracketed by HIP
    # events on the same stream: per-kernel durations.  The events cost a
    # few microseconds per launch, so the step time above comes from the
    # untraced pass.
    ctx.trace(True)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(args.steps):
        job.step()
    e1.record()
    torch.cuda.synchronize()
    traced_ms_step = e0.elapsed_time(e1) / args.steps
    kern = ctx.trace_read()
    ctx.trace(False)
    ctx.check("traced steps")
    job.check()

    # per-kernel algorithmic rates; the dominant kernel kind is the one with
    # the most device time
    per_kernel = {}
    total_alg = 0
    for k, (n_launch, ms) in kern.items():
        ab = job.alg.get(k)
        rate = None
        if ab and ms > 0:
            rate = round(ab * args.steps / (ms * 1e-3) / 1e9, 1)
            total_alg += ab
        per_kernel[k] = {"launches_per_step": n_launch / args.steps, "avg_ms": round(ms / n_launch, 4),
                         "ms_per_step": round(ms / args.steps, 4), "alg_GBps": rate}
    dom = max(kern.items(), key=lambda kv: kv[1][1])[0]
    dom_launches = kern[dom][0] / args.steps
    dom_avg_ms = kern[dom][1] / kern[dom][0]
    dom_bytes = job.alg.get(dom, 0) / dom_launches
    achieved = dom_bytes / (dom_avg_ms * 1e-3) / 1e9
    value = job.children / (ms_step * 1e-3)
    traffic = traffic_from_profile() if (job.name, dom) == TRAFFIC_WORKLOAD else None

    result = {
        "metric": job.metric,
        "value": round(value, 1),
        "unit": "children/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "ms_per_step_median": round(float(np.median(per_step)), 4),
        "ms_per_step_min": round(min(per_step), 4),
        "traced_ms_per_step": round(traced_ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u8",
        "data": "synthetic",
        "config": job.config,
        "roofline": {
            "bound": "hbm", "kernel": dom, "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
            "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
            "traffic": traffic,
            "alg_bytes_per_launch": int(dom_bytes), "avg_launch_ms": round(dom_avg_ms, 4),
            "launches_per_step": dom_launches,
        },
        # the measured HBM bytes of the dominant kernel (rocprofv3 counters) over its live duration
        "traffic_GBps": round(traffic / (dom_avg_ms * 1e-3) / 1e9, 1) if traffic else None,
        "traffic_frac": round(traffic / (dom_avg_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4) if traffic else None,
        "step_alg_GBps": round(total_alg / (ms_step * 1e-3) / 1e9, 1),
        "step_frac_of_peak": round(total_alg / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
        # the whole step against the HBM peak: algorithmic bytes of every
        # kernel of the step over the untimed-event step time (the target's
        # figure); roofline above is the dominant kernel alone
        "step_roofline": {"bound": "hbm", "achieved": round(total_alg / (ms_step * 1e-3) / 1e9, 1),
                          "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                          "frac": round(total_alg / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
                          "alg_bytes_per_step": int(total_alg)},
        "kernels": per_kernel,
    }
    if job.leaves is not None:
        result["leaf_children_per_s"] = round(job.leaves / (ms_step * 1e-3), 1)

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

    del job
    torch.cuda.empty_cache()
    return result


def _cpu_info():
    """Model name of the host CPU as /proc/cpuinfo gives it, with its
    family / model / stepping numbers, and the host's CPU count."""
    fields = {}
    try:
        for line in open("/proc/cpuinfo"):
            if ":" in line:
                k, v = line.split(":", 1)
                fields.setdefault(k.strip(), v.strip())
            if not line.strip() and fields:
                break
    except OSError:
        pass
    model = fields.get("model name") or platform.processor() or "unknown"
    ids = [f"{k} {fields[k]}" for k in ("cpu family", "model", "stepping") if k in fields]
    if ids:
        model = f"{model} ({', '.join(ids)})"
    return model, os.cpu_count()


class _OneCore:
    """Pins this process to one CPU (the first it may use) while the oracle
    runs, and restores the previous set afterwards; the oracle is single
    threaded, so the pin only keeps it from migrating."""

    def __enter__(self):
        self.prev = os.sched_getaffinity(0)
        self.cpu = min(self.prev)
        os.sched_setaffinity(0, {self.cpu})
        return self

    def __exit__(self, *exc):
        os.sched_setaffinity(0, self.prev)
        return False


def _host_bytes(rep):
    """A report layout's record bytes on the host, written by the generator's
    device fill (the same content definition, much faster than numpy)."""
    import torch
    from workloads import device as D
    total = int(rep.off[-1])
    dev = torch.zeros(max(total, 1), dtype=torch.uint8, device="cuda")
    D.fill_records_dev(D.to_dev(rep.seed), D.to_dev(rep.off), dev)
    host = dev.cpu().numpy()[rep.base:total]
    del dev
    return host


def cpu_baseline(workload):
    """The oracle, single threaded and pinned to one CPU, on the workload
    (the full one: each takes under 15 s of one core here)."""
    with _OneCore() as pin:
        r = _cpu_baseline(workload)
    r["pinned_cpu"] = pin.cpu
    return r


def _cpu_baseline(workload):
    import torch
    import oracle as O
    import workloads as W
    from workloads import device as D

    L = O.lib()
    if workload in ("zipf-single", "zipf-canonical"):
        n_parents = 100_000
        c = W.config2(n_parents=n_parents, canonical_order=workload == "zipf-canonical")
        r = c.reports
        S = int(r.off[-1])
        dev = torch.empty(max(S, 1), dtype=torch.uint8, device="cuda")
        D.fill_records_dev(D.to_dev(r.seed), D.to_dev(r.off), dev)
        data = dev.cpu().numpy()
        del dev
        t = time.perf_counter()
        offs, cp, co = O.expand(c.counts, L=L)
        b1 = O.batch(c.queue, c.keep, offs, c.batch_size, L=L)
        b2 = O.batch(c.sealed_ids, None, offs, c.batch_size, L=L)
        par = np.concatenate([b1[1], b2[1]])
        ordi = np.concatenate([b1[2], b2[2]])
        g = O.gather(par, ordi, r.state, r.off, data, offs, L=L)
        dt = time.perf_counter() - t
        assert int(g["out_off"][-1]) == S
        n_child = c.n_children
        sample = (f"the full workload ({n_parents} parents: {n_child} children, {S} surviving bytes); "
                  f"expand + 2 batches + gather")
    elif workload in ("docs-nested", "videos-nested"):
        n = W.config3() if workload == "docs-nested" else W.config4()
        r = n.reports
        data = _host_bytes(r)
        t = time.perf_counter()
        want = O.nested(n.counts1, n.queue1, None, n.batch1, n.counts2, n.queue2, None, n.batch2,
                        r.state, r.off, data, L=L)
        dt = time.perf_counter() - t
        assert int(want["low"]["out_off"][-1]) == int(r.off[-1])
        n_child = len(n.queue1) + len(n.queue2)
        sample = (f"{len(n.counts1)} top parents, {len(n.queue1)} + {len(n.queue2)} children, "
                  f"{int(r.off[-1])} leaf bytes; expand, batch, expand, batch, gather, gather")
    elif workload == "docs-ops":
        n = W.config3()
        rng = np.random.default_rng(7)
        N2, P1 = len(n.queue2), len(n.counts1)
        stv = np.array([0, 0, 0, 1, 2, 3], np.uint8)
        xs, ms = rng.choice(stv, N2), rng.choice(stv, N2)
        mv = (rng.random(N2) < 0.5).astype(np.uint8)
        doc_x = rng.choice(stv, P1)
        t = time.perf_counter()
        _, p1, _ = O.expand(n.counts1, L=L)
        _, p2, _ = O.expand(n.counts2, L=L)
        O.filter(xs, mv, ms, L=L)
        O.broadcast([p2, p1], doc_x, n.states, L=L)
        dt = time.perf_counter() - t
        n_child = N2
        sample = f"the full workload ({N2} regions); two expands for the maps, filter, broadcast"
    elif workload == "zipf-pbatch":
        c = W.config2()
        t = time.perf_counter()
        offs = O.expand(c.counts, tags=False, L=L)
        _, _, _, sizes = O.batch(c.queue, c.keep, offs, c.batch_size, L=L, parent_bound=True)
        dt = time.perf_counter() - t
        n_child = c.n_dispatched
        sample = (f"the full workload ({len(c.queue)} queue entries, {n_child} ready, {len(sizes)} batches); "
                  f"expand and parent-bound reservations")
    elif workload == "zipf-fence":
        c = W.config2()
        f = W.fence_trace(c)
        datas = [r.repeated_data() for r in f.rounds]
        t = time.perf_counter()
        offs = O.expand(c.counts, tags=False, L=L)
        g = O.Grains(c.n_children, L=L)
        g.dispatch(f.dispatch0)
        r0, r1 = f.rounds
        g.commit(r0.parent, r0.ordinal, r0.state, r0.off, datas[0], r0.generation, offs)
        g.retry(f.lost)
        g.dispatch(f.lost)
        g.commit(r1.parent, r1.ordinal, r1.state, r1.off, datas[1], r1.generation, offs)
        dt = time.perf_counter() - t
        g.close()
        n_child = len(f.dispatch0)
        sample = (f"the full workload ({c.n_children} children, {n_child} dispatched, the same fence trace; "
                  f"the oracle holds the bytes of repeated reports only, the rest it never reads); "
                  f"expand, dispatch, commit, retry, dispatch, commit")
    else:
        s = W.config5()
        total = int(s.wave_reports[-1].off[-1])
        dev = torch.zeros(total + 1, dtype=torch.uint8, device="cuda")
        for rep in s.wave_reports:
            D.fill_records_dev(D.to_dev(rep.seed), D.to_dev(rep.off), dev)
        arena = dev.cpu().numpy()
        del dev
        t = time.perf_counter()
        offs = O.expand(s.counts, tags=False, L=L)
        st = O.Stream(offs, L=L)
        for q, rep in zip(s.waves, s.wave_reports):
            _, par, ordi, _ = O.batch(q, None, offs, s.batch_size, L=L)
            st.report(par, ordi, rep.state, rep.off, arena)
            st.emit()
        st.close()
        dt = time.perf_counter() - t
        n_child = s.n_children
        sample = (f"the full workload ({s.n_parents} parents, {n_child} children over {len(s.waves)} waves); "
                  f"expand + per wave batch, report, emit")
    model, ncpu = _cpu_info()
    log(f"[bench] cpu oracle: {n_child} children in {dt:.2f}s")
    return {"value": round(n_child / dt, 1), "unit": "children/s", "cores": 1, "kind": "oracle",
            "sample": sample + ", single thread", "seconds": round(dt, 2), "cpu_model": model,
            "host_cpus": ncpu}


if __name__ == "__main__":
    main()
