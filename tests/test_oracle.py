"""Pins for the CPU oracle (no GPU): worked examples from the paper's figures,
brute-force enumeration on tiny inputs, closed forms and invariants."""
import itertools
import json
import os

import numpy as np
import pytest

import oracle as O
from oracle import brute
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _key_ids(fx):
    names = fx["parents"]
    counts = fx["counts"]
    offs = np.concatenate([[0], np.cumsum(counts)])
    return lambda k: int(offs[names.index(k[0])] + k[1]), offs


# ---------------------------------------------------------------- worked examples
def test_teaser_fifo_batches_and_completion():
    fx = json.load(open(os.path.join(GOLDEN, "teaser_fifo.json")))
    cid, _ = _key_ids(fx)
    offsets = O.expand(fx["counts"], tags=False)
    queue = np.array([cid(k) for k in fx["queue"]], np.uint32)
    child, parent, ordinal, sizes = O.batch(queue, None, offsets, fx["reserve"])
    assert list(sizes) == [len(b) for b in fx["batches"]]
    flat = [tuple(k) for b in fx["batches"] for k in b]
    got = [(fx["parents"][p], o) for p, o in zip(parent, ordinal)]
    assert got == flat
    # the eight batched children turn terminal (SUCCESS, one byte each)
    n = len(child)
    g = O.gather(parent, ordinal, np.zeros(n, np.uint8), np.arange(n + 1), np.arange(n, dtype=np.uint8),
                 offsets)
    for i, name in enumerate(fx["parents"]):
        done, total = fx["terminal_over_total"][name]
        assert g["n_success"][i] + g["n_failed"][i] + g["n_skipped"][i] == done
        assert offsets[i + 1] - offsets[i] == total
        assert bool(g["complete"][i]) == fx["proceeds"][name]
        assert g["parent_state"][i] == (O.SUCCESS if fx["proceeds"][name] else O.PENDING)


def test_failure_figure_reservation():
    fx = json.load(open(os.path.join(GOLDEN, "failure_fifo.json")))
    cid, _ = _key_ids(fx)
    offsets = O.expand(fx["counts"], tags=False)
    queue = np.array([cid(k) for k in fx["queue"]], np.uint32)
    child, parent, ordinal, sizes = O.batch(queue, None, offsets, fx["reserve"])
    first = [(fx["parents"][p], o) for p, o in zip(parent[:sizes[0]], ordinal[:sizes[0]])]
    rest = [(fx["parents"][p], o) for p, o in zip(parent[sizes[0]:], ordinal[sizes[0]:])]
    assert first == [tuple(k) for k in fx["first_batch"]]
    assert rest == [tuple(k) for k in fx["left_in_queue"]]


# ---------------------------------------------------------------- expand
def test_expand_exhaustive_vs_brute():
    for P in range(0, 4):
        for counts in itertools.product(range(4), repeat=P):
            offs, par, ordi = O.expand(np.array(counts, np.int32))
            bo, bp, bord = brute.expand(counts)
            assert list(offs) == bo
            assert list(par) == bp and list(ordi) == bord


def test_expand_invariants_config2_small():
    c = W.config2(n_parents=3000)
    offs, par, ordi = O.expand(c.counts)
    assert offs[0] == 0 and offs[-1] == c.counts.astype(np.int64).sum()
    assert np.all(np.diff(par.astype(np.int64)) >= 0)               # parents nondecreasing
    # ordinals run 0..k-1 for every parent, each child exactly once
    for p in np.random.default_rng(0).choice(len(c.counts), 200, replace=False):
        seg = ordi[offs[p]:offs[p + 1]]
        assert np.array_equal(seg, np.arange(c.counts[p]))
        assert np.all(par[offs[p]:offs[p + 1]] == p)
    keys = par.astype(np.int64) * (1 << 32) + ordi
    assert len(np.unique(keys)) == len(keys)


def test_expand_errors(olib):
    with pytest.raises(O.OracleError) as e:
        O.expand(np.array([1, -1, 2], np.int32))
    assert e.value.code == O.EINVAL
    big = np.full(3, 2 ** 31 - 1, np.int32)
    with pytest.raises(O.OracleError) as e:
        O.expand(big, tags=False)
    assert e.value.code == O.EOVERFLOW


def test_expand_empty():
    offs, par, ordi = O.expand(np.zeros(0, np.int32))
    assert list(offs) == [0] and len(par) == 0
    offs, par, ordi = O.expand(np.zeros(5, np.int32))
    assert list(offs) == [0] * 6 and len(par) == 0


# ---------------------------------------------------------------- batch
def test_batch_exhaustive_vs_brute():
    for counts in [(2, 1), (0, 3, 1), (1, 0, 0, 2), (4,)]:
        n = sum(counts)
        offsets = O.expand(np.array(counts, np.int32), tags=False)
        keys = brute.children(counts)
        for perm in itertools.permutations(range(n)):
            for mask in itertools.product((0, 1), repeat=n):
                for B in range(1, n + 2):
                    q = np.array(perm, np.uint32)
                    keep = np.array(mask, np.uint8)
                    child, parent, ordinal, sizes = O.batch(q, keep, offsets, B)
                    bb, _ = brute.batch(list(perm), list(mask), counts, B)
                    assert list(sizes) == [len(b) for b in bb]
                    flat = [c for b in bb for c in b]
                    assert list(child) == flat
                    assert [(int(p), int(o)) for p, o in zip(parent, ordinal)] == [keys[c] for c in flat]


def test_batch_fifo_order_and_chunking():
    c = W.config2(n_parents=2000)
    offs = O.expand(c.counts, tags=False)
    child, parent, ordinal, sizes = O.batch(c.queue, c.keep, offs, c.batch_size)
    kept = np.nonzero(c.keep)[0]
    # FIFO: kept entries appear once each, in queue order
    assert np.array_equal(child, c.queue[kept])
    m = len(kept)
    B = c.batch_size
    assert len(sizes) == -(-m // B)
    assert np.all(sizes[:-1] == B) and 1 <= sizes[-1] <= B
    assert np.all(offs[parent] + ordinal == child)


def test_batch_parent_exhaustive_vs_brute():
    """Sec. 4 "Scheduling Ready Grains": parent-bound reservations, the C
    oracle against the literal list simulation on every queue order, keep
    mask and batch size of tiny expansions."""
    for counts in [(2, 1), (0, 3, 1), (1, 0, 0, 2), (4,), (2, 2)]:
        n = sum(counts)
        offsets = O.expand(np.array(counts, np.int32), tags=False)
        keys = brute.children(counts)
        for perm in itertools.permutations(range(n)):
            for mask in itertools.product((0, 1), repeat=n):
                for B in range(1, n + 2):
                    q = np.array(perm, np.uint32)
                    keep = np.array(mask, np.uint8)
                    child, parent, ordinal, sizes = O.batch(q, keep, offsets, B, parent_bound=True)
                    bb, _ = brute.batch_parent(list(perm), list(mask), counts, B)
                    assert list(sizes) == [len(b) for b in bb]
                    flat = [c for b in bb for c in b]
                    assert list(child) == flat
                    assert [(int(p), int(o)) for p, o in zip(parent, ordinal)] == [keys[c] for c in flat]


def test_batch_parent_teaser_queue():
    """The teaser figure's ready queue A0 B0 C0 A1 B1 C1 B2 C2 under
    parent-bound reservations of B = 2 (worked by hand from the definition):
    A0 A1 | B0 B1 | C0 C1 | B2 | C2."""
    counts = np.array([2, 3, 3], np.int32)            # A, B, C
    offs = O.expand(counts, tags=False)
    A, Bp, Cp = 0, 2, 5
    q = np.array([A, Bp, Cp, A + 1, Bp + 1, Cp + 1, Bp + 2, Cp + 2], np.uint32)
    child, parent, ordinal, sizes = O.batch(q, None, offs, 2, parent_bound=True)
    assert list(sizes) == [2, 2, 2, 1, 1]
    assert list(zip(parent.tolist(), ordinal.tolist())) == [(0, 0), (0, 1), (1, 0), (1, 1), (2, 0), (2, 1),
                                                            (1, 2), (2, 2)]


def test_batch_parent_closed_form():
    """An equivalent formulation: rank every kept entry within its parent in
    queue order; the entries of ranks jB .. jB + B - 1 of a parent form one
    batch, and batches follow the queue position of their first entry (the
    head is always the earliest entry left, and batches leave whole)."""
    for B, seed in [(1, 0), (3, 1), (256, 2), (10_000, 3)]:
        c = W.config2(n_parents=300, seed=seed)
        offs = O.expand(c.counts, tags=False)
        child, parent, ordinal, sizes = O.batch(c.queue, c.keep, offs, B, parent_bound=True)
        kept = c.queue[c.keep == 1].astype(np.int64)
        par = np.searchsorted(offs, kept, side="right") - 1
        rank = np.zeros(len(kept), np.int64)
        seen = {}
        for i, p in enumerate(par.tolist()):
            rank[i] = seen.get(p, 0)
            seen[p] = rank[i] + 1
        # queue position of the first entry of each entry's batch
        pos_by_parent = {}
        for i, p in enumerate(par.tolist()):
            pos_by_parent.setdefault(p, []).append(i)
        first = np.array([pos_by_parent[p][(r // B) * B] for p, r in zip(par.tolist(), rank.tolist())])
        order = np.lexsort((rank, first))                      # by batch, then rank inside it
        bounds = np.flatnonzero(np.diff(first[order])) + 1
        want = np.split(kept[order], bounds)
        assert list(sizes) == [len(w) for w in want]
        assert np.array_equal(child, np.concatenate(want))
        assert np.all(offs[parent] + ordinal == child)


def test_batch_parent_barrier_is_a_filter():
    c = W.config2(n_parents=800, seed=4)
    offs = O.expand(c.counts, tags=False)
    rng = np.random.default_rng(4)
    bar = (rng.random(800) < 0.3).astype(np.uint8)
    par = np.searchsorted(offs, c.queue.astype(np.int64), side="right") - 1
    keep2 = c.keep & (bar[par] == 0)
    a = O.batch(c.queue, c.keep, offs, 7, barrier=bar, parent_bound=True)
    b = O.batch(c.queue, keep2.astype(np.uint8), offs, 7, parent_bound=True)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


def test_batch_errors():
    offs = O.expand(np.array([2, 1], np.int32), tags=False)
    with pytest.raises(O.OracleError) as e:
        O.batch(np.array([0, 3], np.uint32), None, offs, 2)
    assert e.value.code == O.ERANGE
    # an out-of-range id that is not kept is never looked at
    child, *_ = O.batch(np.array([0, 3], np.uint32), np.array([1, 0], np.uint8), offs, 2)
    assert list(child) == [0]
    child, parent, ordinal, sizes = O.batch(np.zeros(0, np.uint32), None, offs, 4)
    assert len(child) == 0 and len(sizes) == 0


# ---------------------------------------------------------------- gather
def _random_reports(rng, counts, p_report=1.0, states=(0, 1, 2), max_len=5):
    reports = []
    for p, k in enumerate(counts):
        for o in range(k):
            if rng.random() >= p_report:
                continue
            s = int(rng.choice(states))
            ln = int(rng.integers(0, max_len + 1))
            reports.append([p, o, s, bytes(rng.integers(0, 256, ln, dtype=np.uint8))])
    order = rng.permutation(len(reports))
    return [reports[i] for i in order]


def _run_gather(reports, counts):
    offsets = O.expand(np.array(counts, np.int32), tags=False)
    n = len(reports)
    par = np.array([r[0] for r in reports], np.uint32)
    ordi = np.array([r[1] for r in reports], np.uint32)
    st = np.array([r[2] for r in reports], np.uint8)
    lens = np.array([len(r[3]) for r in reports], np.int64)
    off = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    data = np.frombuffer(b"".join(r[3] for r in reports) or b"\0", np.uint8)
    return O.gather(par, ordi, st, off, data, offsets)


def _compare_brute(g, b):
    for p, (ns, nf, nk, done, state, slot) in enumerate(b):
        assert g["n_success"][p] == ns and g["n_failed"][p] == nf and g["n_skipped"][p] == nk
        assert g["complete"][p] == done and g["parent_state"][p] == state
        got = bytes(g["out_data"][g["out_off"][p]:g["out_off"][p + 1]])
        assert got == slot


def test_gather_vs_brute_exhaustive_states():
    rng = np.random.default_rng(7)
    for counts in [(1, 2), (0, 3), (2, 0, 2), (3,)]:
        n = sum(counts)
        for states in itertools.product((0, 1, 2, 3), repeat=n):
            reports = []
            i = 0
            for p, k in enumerate(counts):
                for o in range(k):
                    reports.append([p, o, states[i], bytes([p * 16 + o] * (o + 1))])
                    i += 1
            order = rng.permutation(n)
            reports = [reports[j] for j in order]
            _compare_brute(_run_gather(reports, counts), brute.gather(reports, counts))


def test_gather_vs_brute_random():
    rng = np.random.default_rng(11)
    for trial in range(300):
        P = int(rng.integers(0, 7))
        counts = [int(x) for x in rng.integers(0, 5, P)]
        reports = _random_reports(rng, counts, p_report=float(rng.choice([1.0, 0.7])),
                                  states=(0, 0, 1, 2, 3))
        _compare_brute(_run_gather(reports, counts), brute.gather(reports, counts))


def test_gather_child_positions():
    """Per-child output positions: the bytes between a child's position and
    the next child's are exactly its own SUCCESS record (empty for any other
    state or no report), and a parent's first child starts its slot."""
    rng = np.random.default_rng(23)
    for trial in range(200):
        P = int(rng.integers(0, 8))
        counts = [int(x) for x in rng.integers(0, 5, P)]
        reports = _random_reports(rng, counts, p_report=float(rng.choice([1.0, 0.6])),
                                  states=(0, 0, 1, 2, 3), max_len=7)
        offsets = O.expand(np.array(counts, np.int32), tags=False)
        par = np.array([r[0] for r in reports], np.uint32)
        ordi = np.array([r[1] for r in reports], np.uint32)
        st = np.array([r[2] for r in reports], np.uint8)
        lens = np.array([len(r[3]) for r in reports], np.int64)
        off = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
        data = np.frombuffer(b"".join(r[3] for r in reports) or b"\0", np.uint8)
        g = O.gather(par, ordi, st, off, data, offsets, child_dst=True)
        cd = g["child_dst_off"]
        N = int(offsets[-1])
        assert len(cd) == N + 1 and cd[N] == g["out_off"][P]
        want = {}
        for p_, o_, s_, b_ in reports:
            if s_ == O.SUCCESS:
                want[int(offsets[p_]) + o_] = b_
        for c in range(N):
            assert bytes(g["out_data"][cd[c]:cd[c + 1]]) == want.get(c, b""), (trial, c)
        for p_ in range(P):
            if counts[p_] > 0:
                assert cd[offsets[p_]] == g["out_off"][p_]


def test_gather_round_trip_and_content():
    """gather(batch(expand(x))) puts every record of parent p back in ordinal
    order; each record's bytes are the splitmix64 stream of its own key."""
    c = W.config1()
    offs, cpar, cord = O.expand(c.counts)
    child, parent, ordinal, _ = O.batch(c.queue, c.keep, offs, c.batch_size)
    r = c.reports
    m = len(child)
    data = r.data()
    g = O.gather(parent, ordinal, r.state[:m], r.off[:m + 1], data, offs)
    # reference slot of each parent from the content definition
    for p in range(c.n_parents):
        ords = np.arange(c.counts[p])
        ok = c.states[offs[p]:offs[p + 1]] == W.SUCCESS
        seeds = W.content_seed(np.full(ok.sum(), p), ords[ok])
        want = W.record_bytes(seeds, c.lengths[offs[p]:offs[p + 1]][ok])
        got = g["out_data"][g["out_off"][p]:g["out_off"][p + 1]]
        assert np.array_equal(got, want)
        assert g["n_success"][p] == ok.sum() and g["n_failed"][p] == (~ok).sum()
        assert g["complete"][p] == 1
        assert g["parent_state"][p] == (O.FAILED if (~ok).any() else O.SUCCESS)


def _full_reports(c, B=None, perm=None):
    """oracle batch tags for the dispatched + sealed children of a workload."""
    offs = O.expand(c.counts, tags=False)
    B = B or c.batch_size
    ch1, p1, o1, _ = O.batch(c.queue, c.keep, offs, B)
    ch2, p2, o2, _ = O.batch(c.queue, c.sealed, offs, B)
    par = np.concatenate([p1, p2])
    ordi = np.concatenate([o1, o2])
    return offs, par, ordi


def test_gather_schedule_invariance():
    """Eq. (schedule-invariance): report order and batch size do not change
    the gathered items."""
    c = W.config2(n_parents=1500)
    r = c.reports
    data = r.data()
    offs, par, ordi = _full_reports(c)
    g0 = O.gather(par, ordi, r.state, r.off, data, offs)
    offs, par_b, ordi_b = _full_reports(c, B=7)
    assert np.array_equal(par_b, par) and np.array_equal(ordi_b, ordi)   # B never reorders
    rng = np.random.default_rng(3)
    perm = rng.permutation(len(par))
    # permute the reports (their bytes move with them)
    lens = np.diff(r.off)[perm]
    off2 = np.concatenate([[0], np.cumsum(lens)])
    data2 = np.concatenate([data[r.off[i]:r.off[i + 1]] for i in perm])
    g1 = O.gather(par[perm], ordi[perm], r.state[perm], off2, data2, offs)
    for k in g0:
        assert np.array_equal(g0[k], g1[k]), k


def test_gather_complete_iff_all_terminal():
    c = W.config2(n_parents=800)
    r = c.reports
    data = r.data()
    offs, par, ordi = _full_reports(c)
    rng = np.random.default_rng(5)
    st = r.state.copy()
    drop = rng.random(len(st)) < 0.01
    st[drop] = W.PENDING
    g = O.gather(par, ordi, st, r.off, data, offs)
    missing = np.zeros(c.n_parents, np.int64)
    np.add.at(missing, par[drop], 1)
    assert np.array_equal(g["complete"] == 1, missing == 0)
    assert np.all(g["parent_state"][missing > 0] == O.PENDING)
    # an incomplete parent still packs the SUCCESS bytes it has, in ordinal order
    p = int(np.nonzero(missing)[0][0])
    sel = np.nonzero((par == p) & (st == W.SUCCESS))[0]
    sel = sel[np.argsort(ordi[sel])]
    want = np.concatenate([data[r.off[i]:r.off[i + 1]] for i in sel]) if len(sel) else np.zeros(0, np.uint8)
    assert np.array_equal(g["out_data"][g["out_off"][p]:g["out_off"][p + 1]], want)


def test_gather_empty_expansion_and_all_skipped():
    counts = [0, 2, 0, 3, 0]
    reports = [[1, 0, W.SKIPPED, b"xx"], [1, 1, W.SKIPPED, b""], [3, 2, W.SUCCESS, b"abc"],
               [3, 0, W.FAILED, b"zz"], [3, 1, W.SUCCESS, b"d"]]
    g = _run_gather(reports, counts)
    assert list(g["complete"]) == [1, 1, 1, 1, 1]
    assert list(g["parent_state"]) == [O.SUCCESS, O.SUCCESS, O.SUCCESS, O.FAILED, O.SUCCESS]
    assert list(g["out_off"]) == [0, 0, 0, 0, 4, 4]
    assert bytes(g["out_data"]) == b"dabc"        # failed bytes never copied; ordinal order


def test_gather_errors():
    counts = [2, 1]
    with pytest.raises(O.OracleError) as e:
        _run_gather([[0, 0, 0, b"a"], [0, 0, 1, b""]], counts)
    assert e.value.code == O.EDUP
    with pytest.raises(O.OracleError) as e:
        _run_gather([[2, 0, 0, b"a"]], counts)
    assert e.value.code == O.ERANGE
    with pytest.raises(O.OracleError) as e:
        _run_gather([[1, 1, 0, b"a"]], counts)
    assert e.value.code == O.ERANGE
    with pytest.raises(O.OracleError) as e:
        _run_gather([[0, 0, 4, b"a"]], counts)
    assert e.value.code == O.ESTATE
    # a PENDING slot is no report: duplicates of it are not conflicts
    g = _run_gather([[0, 0, 3, b""], [0, 0, 3, b""], [0, 0, 0, b"q"]], counts)
    assert g["n_success"][0] == 1
    offsets = O.expand(np.array(counts, np.int32), tags=False)
    with pytest.raises(O.OracleError) as e:           # decreasing offsets
        O.gather(np.array([0, 0], np.uint32), np.array([0, 1], np.uint32), np.zeros(2, np.uint8),
                 np.array([0, 3, 2]), np.zeros(3, np.uint8), offsets)
    assert e.value.code == O.EINVAL


# ---------------------------------------------------------------- nested
def test_nested_closed_form_documents():
    """All leaves succeed and the mid level is canonical: each document's
    slot is the concatenation, over (page ordinal, region ordinal) in
    lexicographic order, of the region records."""
    n = W.config3(n_docs=150)
    r = n.reports
    data = r.data()
    res = O.nested(n.counts1, n.queue1, None, n.batch1, n.counts2, n.queue2, None, n.batch2,
                   r.state, r.off, data)
    low, up = res["low"], res["up"]
    off1, off2 = res["offsets1"], res["offsets2"]
    assert np.array_equal(up["out_data"], low["out_data"])
    assert np.array_equal(up["out_off"], low["out_off"][off1])
    assert np.all(up["complete"] == 1) and np.all(up["parent_state"] == O.SUCCESS)
    # spot-check a document directly from the content definition
    for d in (0, len(n.counts1) // 2, len(n.counts1) - 1):
        parts = []
        for g in range(off1[d], off1[d + 1]):
            seeds = W.content_seed(np.full(n.counts2[g], g), np.arange(n.counts2[g]))
            parts.append(W.record_bytes(seeds, n.lengths[off2[g]:off2[g + 1]]))
        want = np.concatenate(parts)
        assert np.array_equal(up["out_data"][up["out_off"][d]:up["out_off"][d + 1]], want)


def test_nested_failed_frames_drop_clips():
    """A clip with a failed frame is FAILED; its bytes stay in the clip slot
    but never reach the video slot, which is then FAILED too."""
    n = W.config4(n_videos=40)
    r = n.reports
    data = r.data()
    res = O.nested(n.counts1, n.queue1, None, n.batch1, n.counts2, n.queue2, None, n.batch2,
                   r.state, r.off, data)
    low, up = res["low"], res["up"]
    off1 = res["offsets1"]
    assert np.all(low["complete"] == 1)
    for v in range(len(n.counts1)):
        clips = np.arange(off1[v], off1[v + 1])
        ok = clips[low["parent_state"][clips] == O.SUCCESS]
        want = np.concatenate([low["out_data"][low["out_off"][g]:low["out_off"][g + 1]] for g in ok]) \
            if len(ok) else np.zeros(0, np.uint8)
        assert np.array_equal(up["out_data"][up["out_off"][v]:up["out_off"][v + 1]], want)
        assert up["parent_state"][v] == (O.FAILED if len(ok) < len(clips) else O.SUCCESS)
        assert up["n_failed"][v] == len(clips) - len(ok)


# ---------------------------------------------------------------- streaming
def _stream_run(s, with_brute=False):
    offs = O.expand(s.counts, tags=False)
    st = O.Stream(offs)
    arena = np.concatenate([r.data() for r in s.wave_reports])
    emitted = []
    for w, (q, r) in enumerate(zip(s.waves, s.wave_reports)):
        ch, par, ordi, _ = O.batch(q, None, offs, s.batch_size)
        st.report(par, ordi, r.state, r.off, arena)
        emitted.append(st.emit())
    st.close()
    return offs, arena, emitted


def test_stream_emits_each_parent_once_at_its_last_wave():
    s = W.config5(n_parents=3000, n_children=40000, n_waves=6)
    offs, arena, emitted = _stream_run(s)
    wave_of = np.empty(s.n_children, np.int64)
    for w, q in enumerate(s.waves):
        wave_of[q] = w
    last = np.zeros(s.n_parents, np.int64)
    par_of_child = np.repeat(np.arange(s.n_parents), s.counts)
    np.maximum.at(last, par_of_child, wave_of)
    seen = np.zeros(s.n_parents, np.int64)
    for w, e in enumerate(emitted):
        assert np.all(np.diff(e["parent"].astype(np.int64)) > 0)      # ascending
        assert np.all(last[e["parent"]] == w)
        seen[e["parent"]] += 1
    assert np.all(seen == 1)
    # union over waves equals the one-shot gather of all reports
    allpar, allord, allst, alloff = [], [], [], []
    for q, r in zip(s.waves, s.wave_reports):
        _, p, o, _ = O.batch(q, None, offs, s.batch_size)
        allpar.append(p); allord.append(o); allst.append(r.state); alloff.append(r.off[:-1])
    alloff.append(s.wave_reports[-1].off[-1:])
    g = O.gather(np.concatenate(allpar), np.concatenate(allord), np.concatenate(allst),
                 np.concatenate(alloff), arena, offs)
    for e in emitted:
        for j, p in enumerate(e["parent"]):
            got = e["data"][e["off"][j]:e["off"][j + 1]]
            assert np.array_equal(got, g["out_data"][g["out_off"][p]:g["out_off"][p + 1]])
            assert e["n_success"][j] == g["n_success"][p]


def test_stream_vs_brute_small():
    rng = np.random.default_rng(2)
    for trial in range(60):
        P = int(rng.integers(1, 6))
        counts = [int(x) for x in rng.integers(0, 4, P)]
        reps = _random_reports(rng, counts, states=(0, 1, 2))
        cuts = sorted(rng.integers(0, len(reps) + 1, 2))
        waves = [reps[:cuts[0]], reps[cuts[0]:cuts[1]], reps[cuts[1]:]]
        want = brute.stream(waves, counts)
        offs = O.expand(np.array(counts, np.int32), tags=False)
        st = O.Stream(offs)
        for w, wave in enumerate(waves):
            lens = [len(x[3]) for x in wave]
            off = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
            data = np.frombuffer(b"".join(x[3] for x in wave) or b"\0", np.uint8).copy()
            st.report(np.array([x[0] for x in wave], np.uint32), np.array([x[1] for x in wave], np.uint32),
                      np.array([x[2] for x in wave], np.uint8), off, data)
            e = st.emit()
            got = [(int(p), int(e["n_success"][j]), int(e["n_failed"][j]), int(e["n_skipped"][j]),
                    int(e["parent_state"][j]), bytes(e["data"][e["off"][j]:e["off"][j + 1]]))
                   for j, p in enumerate(e["parent"])]
            assert got == want[w]
        st.close()


def test_stream_duplicate_across_waves():
    offs = O.expand(np.array([2, 1], np.int32), tags=False)
    st = O.Stream(offs)
    one = np.array([0, 1], np.int64)
    st.report(np.array([0], np.uint32), np.array([1], np.uint32), np.zeros(1, np.uint8), one,
              np.zeros(1, np.uint8))
    with pytest.raises(O.OracleError) as e:
        st.report(np.array([0], np.uint32), np.array([1], np.uint32), np.zeros(1, np.uint8), one,
                  np.zeros(1, np.uint8))
    assert e.value.code == O.EDUP
    st.close()


# ---------------------------------------------------------------- group failure
def test_group_failure_figure():
    """Fig. recovery-protocol: B1's group failure rejects the in-flight B2,
    suppresses the queued B3, keeps B0 committed earlier, and leaves A and C
    to pass on their own."""
    fx = json.load(open(os.path.join(GOLDEN, "failure_group.json")))
    names = {n: i for i, n in enumerate("ABC")}
    codes = {"SUCCESS": O.SUCCESS, "GROUP_FAILED": O.GROUP_FAILED}
    counts = np.array(fx["counts"], np.int32)
    offs = O.expand(counts, tags=False)
    st = O.Stream(offs)

    def wave(reports):
        par = np.array([names[r[0]] for r in reports], np.uint32)
        ordi = np.array([r[1] for r in reports], np.uint32)
        state = np.array([codes[r[2]] for r in reports], np.uint8)
        data = np.array([16 * names[r[0]] + r[1] for r in reports], np.uint8)
        off = np.arange(len(reports) + 1, dtype=np.int64)
        return st.report(par, ordi, state, off, data)

    ex = fx["expect"]
    assert wave(fx["wave1"]["reports"]) == 0
    assert len(st.emit()["parent"]) == len(ex["wave1_emitted"]) == 0
    queue = np.array([offs[names[p]] + o for p, o in fx["queue"]], np.uint32)
    child, par, ordi, sizes = O.batch(queue, None, offs, fx["reserve"], barrier=st.barrier())
    assert [(int(p), int(o)) for p, o in zip(par[:sizes[0]], ordi[:sizes[0]])] == \
        [(names[p], o) for p, o, _ in fx["wave2"]["reports"]]
    assert wave(fx["wave2"]["reports"]) == ex["wave2_rejected"]
    e = st.emit()
    assert [("ABC"[p]) for p in e["parent"]] == ex["wave2_emitted"]
    for j, p in enumerate(e["parent"]):
        n = "ABC"[p]
        assert e["parent_state"][j] == codes.get(ex["states"][n], O.FAILED)
        assert e["n_success"][j] == ex["n_success"][n] and e["n_failed"][j] == ex["n_failed"][n]
        assert list(e["data"][e["off"][j]:e["off"][j + 1]]) == ex["bytes"][n]
    # the next reservation over what is left (B3) suppresses it
    left = queue[sizes[0]:]
    assert len(O.batch(left, None, offs, fx["reserve"], barrier=st.barrier())[0]) == len(ex["next_reservation"])
    st.close()


def _gf_expected(reports, counts, barrier_in):
    """Group failure from its first-failure form: a report of parent p is
    accepted iff p was not barred before the call and no group failure of p
    comes earlier in report order."""
    P = len(counts)
    first = {}
    for i, (p, o, s, b) in enumerate(reports):
        if s == O.GROUP_FAILED and p not in first and not barrier_in[p]:
            first[p] = i
    acc = [s != O.PENDING and not barrier_in[p] and (p not in first or i <= first[p])
           for i, (p, o, s, b) in enumerate(reports)]
    bar = np.array([1 if barrier_in[p] or p in first else 0 for p in range(P)], np.uint8)
    out = []
    for p in range(P):
        mine = sorted((o, s, b) for (pp, o, s, b), a in zip(reports, acc) if a and pp == p)
        ns = sum(1 for _, s, _ in mine if s == O.SUCCESS)
        nf = sum(1 for _, s, _ in mine if s in (O.FAILED, O.GROUP_FAILED))
        nk = sum(1 for _, s, _ in mine if s == O.SKIPPED)
        done = bool(bar[p]) or ns + nf + nk == counts[p]
        state = O.PENDING if not done else (O.FAILED if bar[p] or nf else O.SUCCESS)
        slot = b"".join(b for _, s, b in mine if s == O.SUCCESS)
        out.append((ns, nf, nk, int(done), state, slot))
    n_rej = sum(1 for (p, o, s, b), a in zip(reports, acc) if s != O.PENDING and not a)
    return out, bar, n_rej


def test_group_failure_vs_first_failure_form():
    rng = np.random.default_rng(31)
    for trial in range(400):
        P = int(rng.integers(1, 6))
        counts = [int(x) for x in rng.integers(0, 5, P)]
        reports = _random_reports(rng, counts, p_report=float(rng.choice([1.0, 0.7])),
                                  states=(0, 0, 1, 2, 3, 4, 4), max_len=4)
        barrier_in = (rng.random(P) < 0.2).astype(np.uint8)
        offsets = O.expand(np.array(counts, np.int32), tags=False)
        par = np.array([r[0] for r in reports], np.uint32)
        ordi = np.array([r[1] for r in reports], np.uint32)
        st = np.array([r[2] for r in reports], np.uint8)
        lens = np.array([len(r[3]) for r in reports], np.int64)
        off = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
        data = np.frombuffer(b"".join(r[3] for r in reports) or b"\0", np.uint8)
        g = O.gather(par, ordi, st, off, data, offsets, barrier=barrier_in)
        want, bar, n_rej = _gf_expected([tuple(r) for r in reports], counts, barrier_in)
        _compare_brute(g, want)
        assert np.array_equal(g["barrier"], bar) and g["n_rejected"] == n_rej, trial


def test_group_failure_rejected_repeat_is_not_a_duplicate():
    """A repeat of a committed child that arrives after its parent's group
    failure is rejected before any duplicate check."""
    offs = O.expand(np.array([3], np.int32), tags=False)
    par = np.zeros(3, np.uint32)
    ordi = np.array([0, 1, 0], np.uint32)
    st = np.array([O.SUCCESS, O.GROUP_FAILED, O.SUCCESS], np.uint8)
    off = np.array([0, 1, 1, 2], np.int64)
    g = O.gather(par, ordi, st, off, np.array([7, 9], np.uint8), offs, barrier=np.zeros(1, np.uint8))
    assert g["n_rejected"] == 1 and g["complete"][0] == 1 and g["parent_state"][0] == O.FAILED
    assert list(g["out_data"]) == [7]
    with pytest.raises(O.OracleError) as e:           # without a barrier array the state is bad
        O.gather(par, ordi, st, off, np.array([7, 9], np.uint8), offs)
    assert e.value.code == O.ESTATE


def test_batch_barrier_is_a_filter():
    """Dropping barred parents' children is the same as filtering the queue
    first (suppressed before dispatch), order kept."""
    rng = np.random.default_rng(37)
    for trial in range(200):
        counts = rng.integers(0, 6, int(rng.integers(1, 9))).astype(np.int32)
        offs, cpar, _ = O.expand(counts)
        N = int(offs[-1])
        q = rng.permutation(N).astype(np.uint32)
        keep = (rng.random(N) < 0.8).astype(np.uint8)
        bar = (rng.random(len(counts)) < 0.3).astype(np.uint8)
        B = int(rng.integers(1, 6))
        got = O.batch(q, keep, offs, B, barrier=bar)
        k2 = keep & (1 - bar[cpar[q]]) if N else keep
        want = O.batch(q, k2, offs, B)
        for a, b in zip(got, want):
            assert np.array_equal(a, b), trial


def test_stream_group_failure_emits_at_barrier():
    """Waves committed in order equal one gather over all reports with the
    barrier carried along; each parent is emitted once, in the wave where it
    completes or is barred."""
    rng = np.random.default_rng(41)
    for trial in range(60):
        counts = rng.integers(0, 6, int(rng.integers(1, 12))).astype(np.int32)
        offs = O.expand(counts, tags=False)
        N = int(offs[-1])
        reports = _random_reports(rng, list(counts), states=(0, 0, 1, 2, 4), max_len=3)
        cuts = np.sort(rng.integers(0, len(reports) + 1, 3))
        waves = np.split(np.arange(len(reports)), cuts)
        st = O.Stream(offs)
        emitted_in = {}
        got_bytes = {}
        for w, idx in enumerate(waves):
            rs = [reports[i] for i in idx]
            par = np.array([r[0] for r in rs], np.uint32)
            ordi = np.array([r[1] for r in rs], np.uint32)
            stt = np.array([r[2] for r in rs], np.uint8)
            off = np.concatenate([[0], np.cumsum([len(r[3]) for r in rs])]).astype(np.int64)
            data = np.frombuffer(b"".join(r[3] for r in rs) or b"\0", np.uint8)
            st.report(par, ordi, stt, off, data)
            e = st.emit()
            for j, p in enumerate(e["parent"]):
                assert p not in emitted_in
                emitted_in[int(p)] = w
                got_bytes[int(p)] = bytes(e["data"][e["off"][j]:e["off"][j + 1]])
        want, bar, _ = _gf_expected([tuple(r) for r in reports], list(counts),
                                    np.zeros(len(counts), np.uint8))
        for p in range(len(counts)):
            if want[p][3]:
                assert p in emitted_in and got_bytes[p] == want[p][5], (trial, p)
            else:
                assert p not in emitted_in
        st.close()


def test_group_failure_trace_schedule():
    """The failure-containment analog on the oracle: every page is either
    dispatched or suppressed, every dispatched report either commits or is
    rejected, the 99 poisoned first pages all commit, only poisoned documents
    lose pages, and every document is emitted once (poisoned ones FAILED with
    the pages committed before their barrier)."""
    from failure_sched import oracle_waves
    t = W.failure_trace()
    N, P = t.n_children, t.n_parents
    assert (N, P, len(t.poisoned)) == (45_507, 1_885, 99)
    assert N - len(t.poisoned) == 45_408                       # non-trigger pages
    assert int(t.counts[t.poisoned].sum()) - len(t.poisoned) == 23_514
    offs, waves = oracle_waves(t)
    disp = np.concatenate([w["dispatched"] for w in waves])
    supp = sum(w["suppressed"] for w in waves)
    rej = sum(w["rejected"] for w in waves)
    assert len(disp) + supp == N and len(np.unique(disp)) == len(disp)
    parent_of = np.repeat(np.arange(P), t.counts)
    poisoned = np.zeros(P, bool)
    poisoned[t.poisoned] = True
    assert poisoned[parent_of[np.setdiff1d(np.arange(N), disp)]].all()   # only their pages are suppressed
    trig = offs[t.poisoned]
    assert np.isin(trig, disp).all()
    emitted = np.concatenate([w["emitted"]["parent"] for w in waves])
    states = np.concatenate([w["emitted"]["parent_state"] for w in waves])
    assert np.array_equal(np.sort(emitted), np.arange(P))
    assert (states[poisoned[emitted]] == O.FAILED).all() and (states[~poisoned[emitted]] == O.SUCCESS).all()
    ns = np.concatenate([w["emitted"]["n_success"] for w in waves])
    nf = np.concatenate([w["emitted"]["n_failed"] for w in waves])
    assert (nf[poisoned[emitted]] == 1).all()
    committed = len(disp) - rej
    assert int(ns.sum() + nf.sum()) == committed
    print(f"group-failure trace: {len(waves)} waves, {len(disp)} dispatched, {supp} suppressed, "
          f"{rej} rejected, {committed} committed")


# ---------------------------------------------------------------- filter / broadcast
S, F, K, Pd = O.SUCCESS, O.FAILED, O.SKIPPED, O.PENDING


def test_filter_mask_table_and_precedence():
    """Table "primitives": on a present x and a present mask the output passes
    x on true and is dropped on false; Sec. 4 propagation: a failed input
    suppresses, an unresolved one waits (even next to a dropped one), a
    dropped one drops; the two inputs play symmetric roles."""
    xs, ms, mv = [], [], []
    for x in (S, F, K, Pd):
        for m in (S, F, K, Pd):
            for v in (0, 1):
                xs.append(x); ms.append(m); mv.append(v)
    out = O.filter(np.array(xs), np.array(mv), np.array(ms))
    got = {(x, m, v): o for x, m, v, o in zip(xs, ms, mv, out)}
    assert got[(S, S, 1)] == S and got[(S, S, 0)] == K
    for v in (0, 1):
        for a in (S, F, K, Pd):
            assert got[(F, a, v)] == F and got[(a, F, v)] == F
            assert got[(a, S, 1)] == a                         # a true mask is the identity
        assert got[(Pd, K, v)] == Pd and got[(K, Pd, v)] == Pd
        assert got[(K, S, v)] == K and got[(S, K, v)] == K
        for a in (S, F, K, Pd):
            for b in (S, F, K, Pd):
                if a != S and b != S:
                    assert got[(a, b, v)] == got[(b, a, v)]
    assert O.filter(np.zeros(0, np.uint8), np.zeros(0, np.uint8)).size == 0


def test_filter_then_reduce_drops_masked_members():
    """Filtered-out members are dropped, so the parent's slot is its
    surviving members' bytes in ordinal order and they count as skipped."""
    rng = np.random.default_rng(43)
    counts = rng.integers(0, 6, 200).astype(np.int32)
    offs, cp, co = O.expand(counts)
    N = int(offs[-1])
    lens = rng.integers(0, 9, N)
    off = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    data = rng.integers(0, 256, int(off[-1]) + 1, dtype=np.uint8)
    mask = (rng.random(N) < 0.6).astype(np.uint8)
    st = O.filter(np.zeros(N, np.uint8), mask)
    g = O.gather(cp, co, st, off, data, offs)
    for p in range(len(counts)):
        cs = range(int(offs[p]), int(offs[p + 1]))
        want = b"".join(bytes(data[off[c]:off[c + 1]]) for c in cs if mask[c])
        assert bytes(g["out_data"][g["out_off"][p]:g["out_off"][p + 1]]) == want
        assert g["n_skipped"][p] == sum(1 for c in cs if not mask[c])


def test_broadcast_ancestor_by_composed_offsets():
    """The ancestor of a leaf two levels down, by searching the two offset
    arrays, equals the chained child->parent maps; its state follows x at
    the ancestor and the leaf's own state."""
    rng = np.random.default_rng(47)
    for trial in range(20):
        c1 = rng.integers(0, 5, int(rng.integers(1, 40))).astype(np.int32)
        o1, p1, _ = O.expand(c1)
        c2 = rng.integers(0, 5, int(o1[-1])).astype(np.int32)
        o2, p2, _ = O.expand(c2)
        n = int(o2[-1])
        x = rng.choice(np.array([S, S, F, K, Pd], np.uint8), len(c1))
        like = rng.choice(np.array([S, S, S, F, K, Pd], np.uint8), n)
        anc, st = O.broadcast([p2, p1], x, like)
        mid = np.searchsorted(o2, np.arange(n), side="right") - 1
        top = np.searchsorted(o1, mid, side="right") - 1
        assert np.array_equal(anc, top), trial
        for d in range(n):
            a, b = x[top[d]], like[d]
            want = F if F in (a, b) else (Pd if Pd in (a, b) else (K if K in (a, b) else S))
            assert st[d] == want
    anc, st = O.broadcast([np.zeros(0, np.uint32)], np.zeros(1, np.uint8))
    assert anc.size == 0 and st.size == 0


# ---------------------------------------------------------------- generation fence
def test_generation_fence_cases():
    """Eq. (generation-fence) case by case: a report commits only while its
    Grain is in flight at the report's generation; a repeat of the committed
    report in the same call is a duplicate, a different one a conflict; a
    retry moves the Grain to the next generation, after which the old
    attempt's report is stale."""
    offs = O.expand(np.array([3], np.int32), tags=False)
    g = O.Grains(3)
    assert list(g.phase()) == [O.READY] * 3
    gen = g.dispatch([0, 1, 2])
    assert list(gen) == [0, 0, 0] and list(g.phase()) == [O.IN_FLIGHT] * 3
    data = np.array([5, 6, 7, 9], np.uint8)
    # child 0: committed, then an identical repeat and a conflicting one
    # child 1: a report at a wrong generation (stale) and a right one
    par = np.zeros(5, np.uint32)
    ordi = np.array([0, 0, 0, 1, 1], np.uint32)
    st = np.array([O.SUCCESS, O.SUCCESS, O.SUCCESS, O.SUCCESS, O.FAILED], np.uint8)
    off = np.array([0, 1, 1, 2, 3, 3], np.int64)            # bytes 5 | - | 6 | 7 | -
    data = np.array([5, 6, 7], np.uint8)
    out, counts = g.commit(par, ordi, st, off, data, np.array([0, 0, 0, 7, 0], np.uint32), offs)
    # report 1 has no bytes while report 0 has one: conflict; report 2 has a different byte: conflict
    assert list(out) == [O.SUCCESS, O.PENDING, O.PENDING, O.PENDING, O.FAILED]
    assert counts == (2, 1, 0, 2)
    assert list(g.phase()) == [O.SEALED, O.SEALED, O.IN_FLIGHT]
    # an identical repeat in one call is a duplicate
    g2 = O.Grains(1)
    g2.dispatch([0])
    o1 = O.expand(np.array([1], np.int32), tags=False)
    out, counts = g2.commit(np.zeros(2, np.uint32), np.zeros(2, np.uint32), np.zeros(2, np.uint8),
                            np.array([0, 2, 4], np.int64), np.array([1, 2, 1, 2], np.uint8), np.zeros(2, np.uint32), o1)
    assert list(out) == [O.SUCCESS, O.PENDING] and counts == (1, 0, 1, 0)
    # child 2 retried: the old attempt's report is stale, the new one commits
    g.retry([2])
    assert g.phase()[2] == O.READY and g.gen()[2] == 1
    assert list(g.dispatch([2])) == [1]
    out, counts = g.commit(np.zeros(2, np.uint32), np.array([2, 2], np.uint32), np.zeros(2, np.uint8),
                           np.array([0, 1, 2], np.int64), np.array([8, 9], np.uint8), np.array([0, 1], np.uint32), offs)
    assert list(out) == [O.PENDING, O.SUCCESS] and counts == (1, 1, 0, 0)
    # phase errors: dispatching a sealed Grain, retrying one not in flight
    with pytest.raises(O.OracleError) as e:
        g.dispatch([0])
    assert e.value.code == O.ESTATE
    with pytest.raises(O.OracleError) as e:
        g.retry([1])
    assert e.value.code == O.ESTATE
    g.close(); g2.close()


def _fenced_run(rng, counts, outcomes, lens, payload, B, retry_p=0.3, stale_p=0.3, dup_p=0.2):
    """A legal schedule with retries, stale and repeated reports; returns the
    gather of everything the fence accepted."""
    offs, cp, co = O.expand(counts)
    N = int(offs[-1])
    g = O.Grains(N)
    ready = list(rng.permutation(N))
    committed = np.zeros(N, bool)
    old_attempts = []                    # (child, generation) of retried attempts
    all_par, all_ord, all_st, all_gen, all_data, all_len = [], [], [], [], [], []
    while not committed.all():
        batch = ready[:B]
        ready = ready[B:]
        gens = g.dispatch(np.array(batch, np.uint32)) if batch else []
        par, ordi, st, gn, blobs = [], [], [], [], []
        for c, gen in zip(batch, gens):
            if rng.random() < retry_p:               # the attempt is lost: retried later
                old_attempts.append((c, gen))
                continue
            reps = 2 if rng.random() < dup_p else 1
            for _ in range(reps):
                par.append(cp[c]); ordi.append(co[c]); st.append(outcomes[c]); gn.append(gen)
                blobs.append(payload[c] if outcomes[c] == O.SUCCESS else b"")
        # stale reports of earlier lost attempts arrive late
        for c, gen in list(old_attempts):
            if rng.random() < stale_p:
                par.append(cp[c]); ordi.append(co[c]); st.append(outcomes[c]); gn.append(gen)
                blobs.append(payload[c] if outcomes[c] == O.SUCCESS else b"")
        order = rng.permutation(len(par))
        par = np.array(par, np.uint32)[order] if par else np.zeros(0, np.uint32)
        ordi = np.array(ordi, np.uint32)[order] if len(order) else np.zeros(0, np.uint32)
        st = np.array(st, np.uint8)[order] if len(order) else np.zeros(0, np.uint8)
        gn = np.array(gn, np.uint32)[order] if len(order) else np.zeros(0, np.uint32)
        blobs = [blobs[i] for i in order]
        off = np.concatenate([[0], np.cumsum([len(b) for b in blobs])]).astype(np.int64)
        data = np.frombuffer(b"".join(blobs) or b"\0", np.uint8)
        out, cnt = g.commit(par, ordi, st, off, data, gn, offs)
        acc = out != O.PENDING
        committed[offs[par[acc]] + ordi[acc]] = True
        all_par.append(par[acc]); all_ord.append(ordi[acc]); all_st.append(st[acc])
        all_data += [blobs[i] for i in np.flatnonzero(acc)]
        # lost attempts go back to the queue at the next generation
        lost = [c for c in batch if not committed[c] and g.phase()[c] == O.IN_FLIGHT]
        if lost:
            g.retry(np.array(lost, np.uint32))
            ready += lost
    par = np.concatenate(all_par); ordi = np.concatenate(all_ord); st = np.concatenate(all_st)
    off = np.concatenate([[0], np.cumsum([len(b) for b in all_data])]).astype(np.int64)
    data = np.frombuffer(b"".join(all_data) or b"\0", np.uint8)
    g.close()
    return O.gather(par, ordi, st, off, data, offs)


def test_generation_fence_schedule_invariance():
    """Eq. (schedule-invariance) under retries: whatever the batches, lost
    attempts, late stale reports and repeats, the fence commits each Grain
    exactly once with its fixed outcome, so the gather equals the one-shot
    gather of one report per child."""
    rng = np.random.default_rng(53)
    for trial in range(25):
        counts = rng.integers(0, 6, int(rng.integers(1, 30))).astype(np.int32)
        offs, cp, co = O.expand(counts)
        N = int(offs[-1])
        outcomes = rng.choice(np.array([0, 0, 0, 1, 2], np.uint8), N)
        payload = [bytes(rng.integers(0, 256, int(rng.integers(0, 6)), dtype=np.uint8)) for _ in range(N)]
        lens = np.array([len(p) if o == 0 else 0 for p, o in zip(payload, outcomes)], np.int64)
        off = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
        data = np.frombuffer(b"".join(p for p, o in zip(payload, outcomes) if o == 0) or b"\0", np.uint8)
        want = O.gather(cp, co, outcomes, off, data, offs)
        for B in (1, 3, 7):
            got = _fenced_run(rng, counts, outcomes, lens, payload, B)
            for k in ("out_off", "n_success", "n_failed", "n_skipped", "complete", "parent_state", "out_data"):
                assert np.array_equal(got[k], want[k]), (trial, B, k)


def test_generation_fence_trace_outcome():
    """Sec. 4, Eq. generation-fence with the publication rules, on the fence
    trace: whatever is lost, repeated or late, every dispatched child ends
    sealed with exactly one accepted report carrying its own outcome; the
    first call accepts every first copy, calls the identical repeats
    duplicates and the altered ones conflicts; the second accepts every
    retried child and rejects the generation-0 reports as stale."""
    c = W.config2(n_parents=400)
    f = W.fence_trace(c, p_repeat=0.05, p_conflict=0.03, p_lost=0.1)
    offs = O.expand(c.counts, tags=False)
    g = O.Grains(c.n_children)
    assert np.array_equal(g.dispatch(f.dispatch0), np.zeros(len(f.dispatch0), np.uint32))
    r0, r1 = f.rounds
    out0, cnt0 = g.commit(r0.parent, r0.ordinal, r0.state, r0.off, r0.data(), r0.generation, offs)
    g.retry(f.lost)
    assert np.array_equal(g.dispatch(f.lost), np.ones(len(f.lost), np.uint32))
    out1, cnt1 = g.commit(r1.parent, r1.ordinal, r1.state, r1.off, r1.data(), r1.generation, offs)
    na = len(f.dispatch0) - len(f.lost)
    assert f.n_conflict > 0 and f.n_repeat > 0 and f.n_stale > 0
    assert tuple(cnt0) == (na, 0, f.n_repeat, f.n_conflict)
    assert tuple(cnt1) == (len(f.lost), f.n_stale, 0, 0)
    ph = g.phase()
    assert (ph[f.dispatch0] == O.SEALED).all()
    assert (ph[c.queue[c.keep == 0]] == O.READY).all()
    acc_child, acc_state = [], []
    for r, out in ((r0, out0), (r1, out1)):
        a = out != O.PENDING
        acc_child.append(offs[r.parent[a]] + r.ordinal[a])
        acc_state.append(out[a])
        assert np.array_equal(out[a], r.state[a])
    ch = np.concatenate(acc_child)
    assert len(np.unique(ch)) == len(ch) == len(f.dispatch0)
    assert np.array_equal(np.concatenate(acc_state), c.states[ch])
    g.close()
    # the fence reads the bytes of repeated reports only: the same outcome
    # from a buffer that holds nothing else
    g = O.Grains(c.n_children)
    g.dispatch(f.dispatch0)
    out0b, cnt0b = g.commit(r0.parent, r0.ordinal, r0.state, r0.off, r0.repeated_data(), r0.generation, offs)
    assert np.array_equal(out0b, out0) and tuple(cnt0b) == tuple(cnt0)
    g.close()
