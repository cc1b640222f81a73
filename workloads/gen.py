"""Seeded synthetic inputs shaped like the paper's long-tailed fan-out workloads.

Five workloads are defined (counts, record lengths, terminal states, ready
orders).  Every draw uses ``numpy.random.default_rng(seed)`` in a fixed order:
child counts, then second-level counts, then record lengths, then terminal
states, then ready-order permutations.

The generator also plays the part of the user function (the "UDF stand-in"):
it lays out one result record per dispatched child in dispatch order, followed
by the sealed (never dispatched) children, whose reports carry no bytes.
Record contents are the little-endian output stream of splitmix64 (Steele,
Lea and Flood, OOPSLA 2014) seeded with ``parent << 32 | ordinal``, truncated
to the record length.  The generator enumerates each child's key only to seed
that content; it computes no output of the method.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

SUCCESS, FAILED, SKIPPED, PENDING, GROUP_FAILED = 0, 1, 2, 3, 4

_GAMMA = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)

__all__ = [
    "SUCCESS", "FAILED", "SKIPPED", "PENDING", "GROUP_FAILED",
    "splitmix64_words", "record_bytes", "content_seed",
    "trunc_zipf", "lognormal_int", "pareto_int", "rank_zipf_counts",
    "Reports", "SingleLevel", "Nested", "Streaming",
    "single_level", "config1", "config2", "config3", "config4", "config5",
    "nested", "streaming", "CONFIG_NAMES", "FailureTrace", "failure_trace",
    "FenceRound", "FenceTrace", "fence_trace",
]


# --------------------------------------------------------------------------
# splitmix64 content
# --------------------------------------------------------------------------
def splitmix64_words(seed, k):
    """Output number ``k`` (0-based) of splitmix64 started from ``seed``.

    The generator state after k+1 steps is ``seed + (k+1)*gamma`` (mod 2^64);
    each output is that state passed through the published 64-bit finaliser.
    """
    seed = np.asarray(seed, dtype=np.uint64)
    k = np.asarray(k, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = seed + (k + np.uint64(1)) * _GAMMA
        z = (z ^ (z >> np.uint64(30))) * _M1
        z = (z ^ (z >> np.uint64(27))) * _M2
        return z ^ (z >> np.uint64(31))


def content_seed(parent, ordinal):
    return (np.asarray(parent, np.uint64) << np.uint64(32)) | np.asarray(ordinal, np.uint64)


def record_bytes(seeds, lengths, chunk_words=1 << 22):
    """Concatenate the records ``splitmix64(seed_r)[:len_r]`` for all r."""
    seeds = np.asarray(seeds, dtype=np.uint64)
    lengths = np.asarray(lengths, dtype=np.int64)
    total = int(lengths.sum())
    out = np.empty(total, dtype=np.uint8)
    nw = (lengths + 7) // 8
    r0, pos = 0, 0
    n = len(lengths)
    cum_all = np.cumsum(nw)
    while r0 < n:
        # records [r0, r1) hold at most ~chunk_words words (at least one record)
        base = int(cum_all[r0 - 1]) if r0 else 0
        r1 = r0 + max(1, int(np.searchsorted(cum_all[r0:] - base, chunk_words, side="right")))
        w = nw[r0:r1]
        W = int(w.sum())
        if W:
            first = np.cumsum(w) - w
            k = np.arange(W, dtype=np.int64) - np.repeat(first, w)
            words = splitmix64_words(np.repeat(seeds[r0:r1], w), k).astype("<u8")
            b = words.view(np.uint8)
            # drop the 0..7 bytes past each record's length in its last word
            pad = 8 * w - lengths[r0:r1]
            npad = int(pad.sum())
            if npad:
                wend = np.cumsum(w)
                rp = np.repeat(np.arange(r1 - r0), pad)
                t = np.arange(npad, dtype=np.int64) - np.repeat(np.cumsum(pad) - pad, pad)
                keep = np.ones(b.size, dtype=bool)
                keep[8 * wend[rp] - pad[rp] + t] = False
                seg = b[keep]
            else:
                seg = b
            out[pos:pos + seg.size] = seg
            pos += seg.size
        r0 = r1
    assert pos == total
    return out


# --------------------------------------------------------------------------
# integer draws
# --------------------------------------------------------------------------
def trunc_zipf(rng, s, lo, hi, n):
    """Truncated Zipf: pmf proportional to k^-s on [lo, hi], by inverse CDF."""
    k = np.arange(lo, hi + 1, dtype=np.float64)
    cdf = np.cumsum(k ** (-s))
    cdf /= cdf[-1]
    u = rng.random(n)
    idx = np.minimum(np.searchsorted(cdf, u, side="right"), len(k) - 1)
    return (lo + idx).astype(np.int64)


def lognormal_int(rng, mu, sigma, lo, hi, n):
    """round-half-even(lognormal(mu, sigma)) clamped to [lo, hi]."""
    return np.clip(np.rint(rng.lognormal(mu, sigma, n)), lo, hi).astype(np.int64)


def pareto_int(rng, alpha, xmin, lo, hi, n):
    """round-half-even(xmin * U^(-1/alpha)) clamped to [lo, hi]."""
    u = 1.0 - rng.random(n)            # (0, 1]
    return np.clip(np.rint(xmin * u ** (-1.0 / alpha)), lo, hi).astype(np.int64)


def rank_zipf_counts(rng, n_parents, n_children, s, lo, hi):
    """Rank-frequency Zipf counts that sum to exactly ``n_children``.

    Rank r (1-based) gets clip(rint(C * r^-s), lo, hi), with C found by
    bisection; a residual left by rounding is closed by +-1 steps on the
    unclamped ranks whose rounding moved them furthest.  Ranks are assigned to
    parents by a seeded permutation.
    """
    counts = _rank_counts(np.arange(1, n_parents + 1), n_children, s, lo, hi)
    perm = rng.permutation(n_parents)
    return counts[perm]


def _rank_counts(ranks, n_children, s, lo, hi):
    """clip(rint(C * r^-s), lo, hi) over the given ranks, summing to n_children."""
    w = np.asarray(ranks, dtype=np.float64) ** (-s)
    lo_c, hi_c = 0.0, float(n_children) / w[-1] + 1.0

    def total(c):
        return int(np.clip(np.rint(c * w), lo, hi).sum())

    for _ in range(200):
        mid = 0.5 * (lo_c + hi_c)
        if total(mid) <= n_children:
            lo_c = mid
        else:
            hi_c = mid
    x = lo_c * w
    counts = np.clip(np.rint(x), lo, hi).astype(np.int64)
    resid = n_children - int(counts.sum())
    if resid > 0:
        cand = np.nonzero(counts < hi)[0]
        order = cand[np.argsort(-(x[cand] - counts[cand]), kind="stable")]
        counts[order[:resid]] += 1
    elif resid < 0:
        cand = np.nonzero(counts > lo)[0]
        order = cand[np.argsort(-(counts[cand] - x[cand]), kind="stable")]
        counts[order[:-resid]] -= 1
    assert int(counts.sum()) == n_children
    return counts


# --------------------------------------------------------------------------
# workload containers
# --------------------------------------------------------------------------
@dataclass
class Reports:
    """UDF stand-in output: one report slot per child, in report order.

    ``child`` and ``seed`` are generator-side bookkeeping (which canonical
    child the slot belongs to, and its content key); the method never sees
    them.  ``state``/``off`` (and the bytes from :meth:`data`) are the report
    fields handed to the gather; the lineage tags come from batching.
    """
    child: np.ndarray      # uint32[n]
    state: np.ndarray      # uint8[n]
    off: np.ndarray        # int64[n+1]
    seed: np.ndarray       # uint64[n]
    base: int = 0          # byte offset of off[0] inside a shared arena

    @property
    def n(self):
        return len(self.child)

    @property
    def lengths(self):
        return np.diff(self.off)

    def data(self):
        return record_bytes(self.seed, self.lengths)


@dataclass
class SingleLevel:
    name: str
    seed: int
    counts: np.ndarray      # int32[P]
    lengths: np.ndarray     # int64[N] canonical record length (bytes if SUCCESS)
    states: np.ndarray      # uint8[N] canonical terminal state
    queue: np.ndarray       # uint32[N] ready order (canonical child ids)
    keep: np.ndarray        # uint8[N] 1 = dispatched, 0 = sealed before dispatch
    batch_size: int
    reports: Reports = field(default=None)

    @property
    def n_parents(self):
        return len(self.counts)

    @property
    def n_children(self):
        return len(self.lengths)

    @property
    def sealed(self):
        return (1 - self.keep).astype(np.uint8)

    @property
    def sealed_ids(self):
        """Children that turned terminal without dispatch, in queue order."""
        return np.ascontiguousarray(self.queue[self.keep == 0])

    @property
    def n_dispatched(self):
        return int(self.keep.sum())


@dataclass
class Nested:
    name: str
    seed: int
    counts1: np.ndarray     # int32[P1]   top parents -> level-1 children
    queue1: np.ndarray      # uint32[N1]
    counts2: np.ndarray     # int32[N1]   level-1 children -> leaves (canonical level-1 order)
    lengths: np.ndarray     # int64[N2]   leaf record length
    states: np.ndarray      # uint8[N2]   leaf terminal state
    queue2: np.ndarray      # uint32[N2]
    batch1: int
    batch2: int
    reports: Reports = field(default=None)   # leaf reports in level-2 dispatch order


@dataclass
class Streaming:
    name: str
    seed: int
    counts: np.ndarray      # int32[P]
    lengths: np.ndarray     # int64[N]
    states: np.ndarray      # uint8[N]
    waves: list             # list of uint32[Q_w] ready children per wave
    batch_size: int
    wave_reports: list = field(default=None)   # Reports per wave, offsets into one arena

    @property
    def n_parents(self):
        return len(self.counts)

    @property
    def n_children(self):
        return len(self.lengths)


def _child_keys(counts):
    """(parent, ordinal) of every child in canonical order, for content seeds."""
    counts = np.asarray(counts, dtype=np.int64)
    parent = np.repeat(np.arange(len(counts), dtype=np.uint64), counts)
    first = np.cumsum(counts) - counts
    ordinal = np.arange(int(counts.sum()), dtype=np.int64) - np.repeat(first, counts)
    return parent, ordinal.astype(np.uint64)


def _states(rng, n, p_failed, p_skipped):
    u = rng.random(n)
    st = np.full(n, SUCCESS, dtype=np.uint8)
    st[u < p_failed] = FAILED
    st[(u >= p_failed) & (u < p_failed + p_skipped)] = SKIPPED
    return st


def _report_layout(order, counts, lengths, states, base=0):
    """Reports for children in ``order``; only SUCCESS reports carry bytes."""
    order = np.asarray(order, dtype=np.int64)
    parent, ordinal = _child_keys(counts)
    st = states[order].astype(np.uint8)
    ln = np.where(st == SUCCESS, lengths[order], 0).astype(np.int64)
    off = np.empty(len(order) + 1, dtype=np.int64)
    off[0] = base
    np.cumsum(ln, out=off[1:])
    off[1:] += base
    seed = content_seed(parent[order], ordinal[order])
    return Reports(child=order.astype(np.uint32), state=st, off=off, seed=seed, base=base)


def single_level(name, seed, counts_fn, length_fn, p_failed, p_skipped, batch_size,
                 canonical_order=False):
    rng = np.random.default_rng(seed)
    counts = counts_fn(rng).astype(np.int64)
    n = int(counts.sum())
    lengths = length_fn(rng, n).astype(np.int64)
    states = _states(rng, n, p_failed, p_skipped)
    if canonical_order:
        queue = np.arange(n, dtype=np.int64)
    else:
        queue = rng.permutation(n)
    keep = (states[queue] != SKIPPED).astype(np.uint8)
    order = np.concatenate([queue[keep == 1], queue[keep == 0]])
    rep = _report_layout(order, counts, lengths, states)
    return SingleLevel(name=name, seed=seed, counts=counts.astype(np.int32), lengths=lengths,
                       states=states, queue=queue.astype(np.uint32), keep=keep,
                       batch_size=batch_size, reports=rep)


def config1(n_parents=1000, seed=0, canonical_order=False):
    """1,000 parents, counts ~ lognormal(1.5, 1.0) clipped to [1, 500], 64-byte
    records, 5% failed, random ready order, B = 64."""
    return single_level(
        "single-level lognormal fan-out, 64-B records", seed,
        lambda r: lognormal_int(r, 1.5, 1.0, 1, 500, n_parents),
        lambda r, n: np.full(n, 64, dtype=np.int64),
        0.05, 0.0, 64, canonical_order)


def config2(n_parents=100_000, seed=1, canonical_order=False):
    """100,000 parents, counts ~ Zipf(1.2) truncated to [1, 10^4], records
    lognormal(6, 1) bytes clipped to [16, 4096], 3% failed, 2% skipped,
    random ready order, B = 256."""
    return single_level(
        "single-level Zipf(1.2) fan-out, 16-4096-B records", seed,
        lambda r: trunc_zipf(r, 1.2, 1, 10_000, n_parents),
        lambda r, n: lognormal_int(r, 6.0, 1.0, 16, 4096, n),
        0.03, 0.02, 256, canonical_order)


def nested(name, seed, n_top, counts1_fn, counts2_fn, length_fn, p_failed, batch1, batch2,
           canonical_order=False):
    rng = np.random.default_rng(seed)
    counts1 = counts1_fn(rng, n_top).astype(np.int64)
    n1 = int(counts1.sum())
    counts2 = counts2_fn(rng, n1).astype(np.int64)
    n2 = int(counts2.sum())
    lengths = length_fn(rng, n2).astype(np.int64)
    states = _states(rng, n2, p_failed, 0.0)
    if canonical_order:
        q1 = np.arange(n1, dtype=np.int64)
        q2 = np.arange(n2, dtype=np.int64)
    else:
        q1 = rng.permutation(n1)
        q2 = rng.permutation(n2)
    rep = _report_layout(q2, counts2, lengths, states)
    return Nested(name=name, seed=seed, counts1=counts1.astype(np.int32), queue1=q1.astype(np.uint32),
                  counts2=counts2.astype(np.int32), lengths=lengths, states=states,
                  queue2=q2.astype(np.uint32), batch1=batch1, batch2=batch2, reports=rep)


def config3(n_docs=20_000, seed=2, canonical_order=False):
    """Two levels: 20,000 documents, pages ~ lognormal(2.3, 0.9) clipped to
    [1, 2000], regions per page ~ Poisson(8)+1, region records uniform in
    [32, 1024] bytes, all succeed, B = 512 at both levels."""
    return nested(
        "two-level documents->pages->regions", seed, n_docs,
        lambda r, n: lognormal_int(r, 2.3, 0.9, 1, 2000, n),
        lambda r, n: r.poisson(8, n) + 1,
        lambda r, n: r.integers(32, 1025, n),
        0.0, 512, 512, canonical_order)


def config4(n_videos=2_000, seed=3, canonical_order=False):
    """Two levels: 2,000 videos, clips ~ Pareto(1.1, x_min 5) clipped to
    [1, 50000], frames per clip uniform in [16, 300], 1,024-byte frame
    records, 1% of frames failed, B = 1,024 at both levels."""
    return nested(
        "two-level videos->clips->frames", seed, n_videos,
        lambda r, n: pareto_int(r, 1.1, 5.0, 1, 50_000, n),
        lambda r, n: r.integers(16, 301, n),
        lambda r, n: np.full(n, 1024, dtype=np.int64),
        0.01, 1024, 1024, canonical_order)


def streaming(name, seed, counts_fn, length_fn, n_waves, batch_size):
    rng = np.random.default_rng(seed)
    counts = counts_fn(rng).astype(np.int64)
    n = int(counts.sum())
    lengths = length_fn(rng, n).astype(np.int64)
    states = np.full(n, SUCCESS, dtype=np.uint8)
    perm = rng.permutation(n)
    waves = [w.astype(np.uint32) for w in np.array_split(perm, n_waves)]
    reps, base = [], 0
    for w in waves:
        r = _report_layout(w.astype(np.int64), counts, lengths, states, base=base)
        reps.append(r)
        base = int(r.off[-1])
    return Streaming(name=name, seed=seed, counts=counts.astype(np.int32), lengths=lengths,
                     states=states, waves=waves, batch_size=batch_size, wave_reports=reps)


def config5(n_parents=500_000, n_children=10_000_000, n_waves=50, seed=4):
    """10^7 children under 500,000 parents, rank-frequency Zipf(1.1) counts
    clipped to [1, 10^5], records uniform in [64, 512] bytes, children turn
    terminal over 50 waves in random order, B = 1,024."""
    return streaming(
        "streaming completion, rank-Zipf(1.1) fan-out", seed,
        lambda r: rank_zipf_counts(r, n_parents, n_children, 1.1, 1, 100_000),
        lambda r, n: r.integers(64, 513, n),
        n_waves, 1024)


@dataclass
class FailureTrace:
    """A Call whose ready queue holds every child of a long-tailed document
    set, pages of one document in page order and documents interleaved; the
    first page of each of the largest documents reports a group failure."""
    name: str
    seed: int
    counts: np.ndarray      # int32[P]
    queue: np.ndarray       # uint32[N] ready order (canonical child ids)
    states: np.ndarray      # uint8[N] canonical report state
    lengths: np.ndarray     # int64[N] record length
    poisoned: np.ndarray    # int64[n_poisoned] parent ids
    wave: int               # entries reserved per wave (actors x batch)
    batch_size: int

    @property
    def n_parents(self):
        return len(self.counts)

    @property
    def n_children(self):
        return len(self.lengths)


def failure_trace(seed=5, n_parents=1_885, n_children=45_507, n_poisoned=99, poisoned_children=23_613,
                  max_pages=427, actors=4, batch_size=48):
    """Group-failure workload shaped by the paper's failure-containment
    numbers (1,885 documents, 45,507 pages, the 99 largest documents poisoned
    at page 0, 23,514 of their other pages; 1-427 pages per document; 4
    actors with batches of 48).  Rank-frequency counts: the 99 largest
    follow r^-0.5 and hold 23,613 pages, the rest follow r^-1 below the
    smallest of them.  The ready queue is a seeded interleaving that keeps
    each document's pages in page order.  Records are uniform in
    [64, 512] bytes; every report succeeds except the poisoned first pages."""
    rng = np.random.default_rng(seed)
    top = _rank_counts(np.arange(1, n_poisoned + 1), poisoned_children, 0.5, 1, max_pages)
    rest = _rank_counts(np.arange(n_poisoned + 1, n_parents + 1), n_children - poisoned_children, 1.0, 1,
                        int(top.min()) - 1)
    by_rank = np.concatenate([top, rest])
    perm = rng.permutation(n_parents)            # parent perm[r] gets rank r
    counts = np.empty(n_parents, np.int64)
    counts[perm] = by_rank
    poisoned = np.sort(perm[:n_poisoned])
    # interleave documents, pages in order: draw a position for every page,
    # then hand each document's positions to its pages in ascending order
    n = int(counts.sum())
    parent = np.repeat(np.arange(n_parents), counts)
    pos = rng.permutation(n)
    idx = np.lexsort((pos, parent))
    pos_of_child = pos[idx]
    queue = np.argsort(pos_of_child, kind="stable")
    offsets = np.concatenate([[0], np.cumsum(counts)])
    states = np.full(n, SUCCESS, np.uint8)
    states[offsets[poisoned]] = GROUP_FAILED
    lengths = rng.integers(64, 513, n).astype(np.int64)
    return FailureTrace(name="group-failure trace", seed=seed, counts=counts.astype(np.int32),
                        queue=queue.astype(np.uint32), states=states, lengths=lengths, poisoned=poisoned,
                        wave=actors * batch_size, batch_size=batch_size)


CONFIG_NAMES = {
    1: "lognormal(1.5,1) x 1,000 parents, 64-B records",
    2: "Zipf(1.2) x 100,000 parents, lognormal 16-4096-B records",
    3: "20,000 docs -> pages -> regions",
    4: "2,000 videos -> clips -> frames",
    5: "10M children / 500,000 parents over 50 waves",
}


# --------------------------------------------------------------------------
# Generation-fence trace: retries, stale and repeated reports
# --------------------------------------------------------------------------

@dataclass
class FenceRound:
    """One commit call: report keys, state, generation and the record layout
    (``off`` into a shared arena, ``seed`` the content key of each record)."""
    parent: np.ndarray      # uint32[n]
    ordinal: np.ndarray     # uint32[n]
    state: np.ndarray       # uint8[n]
    generation: np.ndarray  # uint32[n]
    off: np.ndarray         # int64[n+1]
    seed: np.ndarray        # uint64[n]
    base: int = 0

    @property
    def n(self):
        return len(self.state)

    def data(self):
        return record_bytes(self.seed, np.diff(self.off))

    def repeated_data(self):
        """Host bytes of the records of every report whose child is reported
        more than once in the call, at their offsets; the rest of the buffer
        stays zero and its pages are never touched (so never allocated)."""
        key = self.parent.astype(np.int64) << 32 | self.ordinal.astype(np.int64)
        _, inv, cnt = np.unique(key, return_inverse=True, return_counts=True)
        idx = np.flatnonzero(cnt[inv] > 1)
        host = np.zeros(max(int(self.off[-1]), 1), np.uint8)
        lens = np.diff(self.off)[idx]
        if len(idx):
            starts = self.off[idx] - np.concatenate([[0], np.cumsum(lens)[:-1]])
            host[np.repeat(starts, lens) + np.arange(int(lens.sum()))] = record_bytes(self.seed[idx], lens)
        return host


@dataclass
class FenceTrace:
    """A Call's dispatched children through two attempts.  Attempt 0
    dispatches them in queue order at generation 0; the reports of a fraction
    of them never arrive, and those children are retried and dispatched again
    at generation 1.  Some attempt-0 reports arrive twice (an identical
    repeat, or a conflicting one: another state, or the same length with other
    bytes), always after the first copy; in the second call, late reports of
    lost attempts arrive at generation 0 (stale) among the new ones."""
    counts: np.ndarray      # int32[P]
    dispatch0: np.ndarray   # uint32[M] children dispatched at generation 0
    lost: np.ndarray        # uint32[L] children retried and dispatched at generation 1
    rounds: list            # [FenceRound, FenceRound]
    n_repeat: int
    n_conflict: int
    n_stale: int


def fence_trace(c, seed=6, p_lost=0.02, p_repeat=0.01, p_conflict=0.002, p_stale=0.5):
    """Fence trace over a single-level workload ``c`` (its dispatched
    children, canonical states and lengths).  Record bytes follow the content
    definition: a report's bytes are splitmix64 of its content seed, which is
    the child's (parent, ordinal) key, with its top bit flipped for a
    conflicting repeat of the same length."""
    rng = np.random.default_rng(seed)
    parent, ordinal = _child_keys(c.counts)
    disp = np.ascontiguousarray(c.queue[c.keep == 1]).astype(np.int64)
    M = len(disp)
    lost_mask = rng.random(M) < p_lost
    arrived = disp[~lost_mask]
    u = rng.random(len(arrived))
    rep = arrived[u < p_repeat]
    conf = arrived[(u >= p_repeat) & (u < p_repeat + p_conflict)]
    lost = disp[lost_mask]

    def build(children, state, gen, seed_xor):
        ln = np.where(state == SUCCESS, c.lengths[children], 0).astype(np.int64)
        off = np.zeros(len(children) + 1, np.int64)
        np.cumsum(ln, out=off[1:])
        sd = content_seed(parent[children], ordinal[children]) ^ seed_xor
        return FenceRound(parent=parent[children].astype(np.uint32), ordinal=ordinal[children].astype(np.uint32),
                          state=state.astype(np.uint8), generation=gen.astype(np.uint32), off=off, seed=sd)

    # call 0: first copies in dispatch order, then the repeats in random order
    rep_all = np.concatenate([rep, conf])
    perm = rng.permutation(len(rep_all))
    rep_all = rep_all[perm]
    is_conf = np.concatenate([np.zeros(len(rep), bool), np.ones(len(conf), bool)])[perm]
    st_rep = c.states[rep_all].copy()
    xor_rep = np.zeros(len(rep_all), np.uint64)
    # a conflict of a successful record keeps its length and changes its bytes;
    # any other conflict changes the state
    same_len = is_conf & (st_rep == SUCCESS) & (rng.random(len(rep_all)) < 0.5)
    xor_rep[same_len] = np.uint64(1 << 63)
    flip = is_conf & ~same_len
    st_rep[flip] = np.where(st_rep[flip] == SUCCESS, FAILED, SUCCESS)
    ch0 = np.concatenate([arrived, rep_all])
    st0 = np.concatenate([c.states[arrived], st_rep])
    xor0 = np.concatenate([np.zeros(len(arrived), np.uint64), xor_rep])
    r0 = build(ch0, st0, np.zeros(len(ch0), np.uint32), xor0)
    # call 1: every retried child at generation 1, and stale generation-0
    # reports of some of them, shuffled together
    stale = lost[rng.random(len(lost)) < p_stale]
    ch1 = np.concatenate([lost, stale])
    g1 = np.concatenate([np.ones(len(lost), np.uint32), np.zeros(len(stale), np.uint32)])
    perm = rng.permutation(len(ch1))
    ch1, g1 = ch1[perm], g1[perm]
    r1 = build(ch1, c.states[ch1], g1, np.zeros(len(ch1), np.uint64))
    return FenceTrace(counts=c.counts, dispatch0=disp.astype(np.uint32), lost=lost.astype(np.uint32),
                      rounds=[r0, r1], n_repeat=len(rep), n_conflict=len(conf), n_stale=len(stale))
