"""GPU parity at the workloads' full sizes, in the benchmark's launch
configuration.  Every integer output is compared with the oracle in full.
The payload bytes are checked on sampled parents against the content
definition (each record is the splitmix64 stream of its own (parent,
ordinal)) computed on the host, and then all of them on the device against
the same definition written by the generator's fill, at the oracle's slot
offsets."""
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

import oracle as O  # noqa: E402
import workloads as W  # noqa: E402
from workloads import device as D  # noqa: E402
import gpu_common as G  # noqa: E402


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def ctx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_18703_amd as R
    c = R.Context()
    yield c
    c.close()


def _expected_slot(counts_row_start, states, lengths, p, k):
    """Bytes of parent p's slot from the content definition: SUCCESS children
    in ordinal order."""
    o = np.arange(k)
    ok = states[counts_row_start:counts_row_start + k] == W.SUCCESS
    seeds = W.content_seed(np.full(int(ok.sum()), p), o[ok])
    return W.record_bytes(seeds, lengths[counts_row_start:counts_row_start + k][ok])


def _sample_parents(rng, counts, n, n_big=10):
    big = np.argsort(-counts.astype(np.int64), kind="stable")[:n_big]
    rnd = rng.choice(len(counts), n, replace=False)
    return np.unique(np.concatenate([big, rnd, [0, len(counts) - 1]]))


def _expected_bytes_dev(counts, lengths, mask):
    """Device bytes of every child with mask set, in canonical order, each
    its record by the content definition (splitmix64 of its (parent,
    ordinal)); these are the packed slots of a gather whose surviving
    children are the masked ones."""
    counts = np.asarray(counts, np.int64)
    parent = np.repeat(np.arange(len(counts), dtype=np.int64), counts)
    first = np.cumsum(counts) - counts
    ordinal = np.arange(int(counts.sum()), dtype=np.int64) - np.repeat(first, counts)
    idx = np.flatnonzero(mask)
    lens = np.asarray(lengths, np.int64)[idx]
    off = np.zeros(len(idx) + 1, np.int64)
    np.cumsum(lens, out=off[1:])
    out = torch.empty(max(int(off[-1]), 1), dtype=torch.uint8, device="cuda")
    if len(idx):
        D.fill_records_dev(D.to_dev(W.content_seed(parent[idx], ordinal[idx])), D.to_dev(off), out)
    return out[:int(off[-1])]


def test_config2_full(ctx):
    from paper_2609_18703_amd import pipeline as PL
    c = W.config2()
    r = c.reports
    _say("config2 full: N =", c.n_children, "bytes =", int(r.off[-1]))
    b = G.stage_single(c)
    ctx.reserve(c.n_children, c.n_parents, c.n_children)
    PL.single_level(ctx, b)
    ctx.check("config2 full")
    _say("config2: oracle metadata")
    want = G.oracle_single(c, with_data=False)
    G.compare_single(b, want, with_data=False)
    g = want["g"]
    rng = np.random.default_rng(11)
    offs = want["offsets"]
    for p in _sample_parents(rng, c.counts, 150):
        k = int(c.counts[p])
        exp = _expected_slot(int(offs[p]), c.states, c.lengths, int(p), k)
        lo, hi = int(g["out_off"][p]), int(g["out_off"][p + 1])
        assert hi - lo == len(exp)
        assert np.array_equal(b.out_data[lo:hi].cpu().numpy(), exp), p
    # every byte: the surviving children's records in canonical order (the
    # slot offsets above are the oracle's)
    _say("config2: all bytes")
    exp = _expected_bytes_dev(c.counts, c.lengths, c.states == W.SUCCESS)
    S = int(g["out_off"][-1])
    assert exp.numel() == S and torch.equal(b.out_data[:S], exp)
    del exp


def _nested_full(ctx, n, sample_top=60, n_big=10):
    from paper_2609_18703_amd import pipeline as PL
    r = n.reports
    data = D.reports_data_dev(r)
    b = PL.NestedBuffers(D.to_dev(n.counts1), D.to_dev(n.queue1.view(np.int32)), n.batch1, D.to_dev(n.counts2),
                         D.to_dev(n.queue2.view(np.int32)), n.batch2, D.to_dev(r.state), D.to_dev(r.off), data,
                         len(n.queue1), len(n.queue2))
    ctx.reserve(len(n.queue2), max(len(n.queue1), len(n.counts1)), len(n.queue2))
    PL.nested(ctx, b)
    ctx.check("nested full")
    _say("nested: oracle metadata")
    want = O.nested(n.counts1, n.queue1, None, n.batch1, n.counts2, n.queue2, None, n.batch2,
                    r.state, r.off, None, with_data=False)
    low, up = want["low"], want["up"]
    N1, N2, P1 = b.N1, b.N2, b.P1
    # every integer output of both levels, in full
    assert np.array_equal(b.offsets1.cpu().numpy()[:P1 + 1], want["offsets1"])
    assert np.array_equal(G.u32(b.mid_parent)[:N1], want["parent1"])
    assert np.array_equal(G.u32(b.mid_ordinal)[:N1], want["ordinal1"])
    sc = b.scalars.cpu().numpy()
    assert int(sc[0]) == len(want["batch1"][0]) == N1
    assert np.array_equal(G.u32(b.b1_parent)[:N1], want["batch1"][1])
    assert np.array_equal(G.u32(b.b1_ordinal)[:N1], want["batch1"][2])
    assert int(sc[1]) == len(want["batch1"][3])
    assert np.array_equal(b.offsets2.cpu().numpy()[:N1 + 1], want["offsets2"])
    assert np.array_equal(G.u32(b.leaf_parent)[:N2], want["parent2"])
    assert np.array_equal(G.u32(b.leaf_ordinal)[:N2], want["ordinal2"])
    assert int(sc[2]) == len(want["batch2"][0]) == N2
    assert np.array_equal(G.u32(b.b2_parent)[:N2], want["batch2"][1])
    assert np.array_equal(G.u32(b.b2_ordinal)[:N2], want["batch2"][2])
    assert int(sc[3]) == len(want["batch2"][3])
    for k in ("out_off",):
        assert np.array_equal(b.mid_off.cpu().numpy()[:N1 + 1], low[k])
        assert np.array_equal(b.top_off.cpu().numpy()[:P1 + 1], up[k])
    assert np.array_equal(b.mid_state.cpu().numpy()[:N1], low["parent_state"])
    assert np.array_equal(b.mid_complete.cpu().numpy()[:N1], low["complete"])
    assert np.array_equal(b.mid_cnt.cpu().numpy()[:N1], low["n_success"])
    assert np.array_equal(b.mid_cnt.cpu().numpy()[N1:2 * N1], low["n_failed"])
    assert np.array_equal(b.mid_cnt.cpu().numpy()[2 * N1:3 * N1], low["n_skipped"])
    assert np.array_equal(b.top_state.cpu().numpy()[:P1], up["parent_state"])
    assert np.array_equal(b.top_complete.cpu().numpy()[:P1], up["complete"])
    assert np.array_equal(b.top_cnt.cpu().numpy()[:P1], up["n_success"])
    assert np.array_equal(b.top_cnt.cpu().numpy()[P1:2 * P1], up["n_failed"])
    assert np.array_equal(b.top_cnt.cpu().numpy()[2 * P1:3 * P1], up["n_skipped"])
    # content: a top slot is its surviving mid slots' bytes in order, and each
    # mid slot is its leaves' splitmix64 records in ordinal order
    off1, off2 = want["offsets1"], want["offsets2"]
    rng = np.random.default_rng(5)
    for d in _sample_parents(rng, n.counts1, sample_top, n_big):
        parts = []
        for gmid in range(int(off1[d]), int(off1[d + 1])):
            if low["parent_state"][gmid] != W.SUCCESS:
                continue
            parts.append(_expected_slot(int(off2[gmid]), n.states, n.lengths, gmid, int(n.counts2[gmid])))
        exp = np.concatenate(parts) if parts else np.zeros(0, np.uint8)
        lo, hi = int(up["out_off"][d]), int(up["out_off"][d + 1])
        assert hi - lo == len(exp)
        assert np.array_equal(b.top_data[lo:hi].cpu().numpy(), exp), d
    # every byte of both levels: a mid slot packs its successful leaves; a
    # top slot packs the leaves of its successful mid slots
    _say("nested: all bytes")
    ok = n.states == W.SUCCESS
    exp = _expected_bytes_dev(n.counts2, n.lengths, ok)
    S2 = int(low["out_off"][-1])
    assert exp.numel() == S2 and torch.equal(b.mid_data[:S2], exp)
    del exp
    mid_ok = np.repeat(low["parent_state"] == W.SUCCESS, n.counts2.astype(np.int64))
    exp = _expected_bytes_dev(n.counts2, n.lengths, ok & mid_ok)
    S1 = int(up["out_off"][-1])
    assert exp.numel() == S1 and torch.equal(b.top_data[:S1], exp)
    del exp


def test_config3_full(ctx):
    n = W.config3()
    _say("config3 full: mid =", len(n.queue1), "leaves =", len(n.queue2))
    _nested_full(ctx, n)


def test_config4_full(ctx):
    n = W.config4()
    _say("config4 full: mid =", len(n.queue1), "leaves =", len(n.queue2))
    _nested_full(ctx, n, sample_top=25, n_big=1)   # the largest videos hold about 1 GB each


def test_config5_full_streaming(ctx):
    """50 waves over 10^7 children: every wave's emitted parents, slot
    offsets, counts, states and bytes in full."""
    from paper_2609_18703_amd import pipeline as PL
    s = W.config5()
    _say("config5 full: N =", s.n_children, "waves =", len(s.waves))
    total = int(s.wave_reports[-1].off[-1])
    arena = torch.empty(max(total, 1), dtype=torch.uint8, device="cuda")
    for rep in s.wave_reports:
        D.fill_records_dev(D.to_dev(rep.seed), D.to_dev(rep.off), arena)
    b = PL.StreamingBuffers(D.to_dev(s.counts), [D.to_dev(q.view(np.int32)) for q in s.waves],
                            [D.to_dev(rep.state) for rep in s.wave_reports],
                            [D.to_dev(rep.off) for rep in s.wave_reports], arena, s.n_children,
                            s.batch_size, total)
    offs = O.expand(s.counts, tags=False)
    ost = O.Stream(offs)
    rng = np.random.default_rng(9)
    P = s.n_parents
    checked = [0]

    def on_wave(w):
        q, rep = s.waves[w], s.wave_reports[w]
        _, par, ordi, _ = O.batch(q, None, offs, s.batch_size)
        ost.report(par, ordi, rep.state, rep.off, None)
        want = ost.emit(with_data=False)
        sc = b.scalars.cpu().numpy()
        E, nb = int(sc[2]), int(sc[3])
        assert E == len(want["parent"]) and nb == want["n_bytes"], w
        assert np.array_equal(G.u32(b.emit_parent)[:E], want["parent"]), w
        assert np.array_equal(b.emit_off.cpu().numpy()[:E + 1], want["off"]), w
        assert np.array_equal(b.emit_cnt.cpu().numpy()[:E], want["n_success"]), w
        assert np.array_equal(b.emit_state.cpu().numpy()[:E], want["parent_state"]), w
        if E:
            # every emitted byte: the emitted parents' children in order
            ep = want["parent"].astype(np.int64)
            ks = s.counts[ep].astype(np.int64)
            cidx = np.repeat(offs[ep] - np.cumsum(ks) + ks, ks) + np.arange(int(ks.sum()))
            mask = np.zeros(s.n_children, bool)
            mask[cidx] = s.states[cidx] == W.SUCCESS
            exp = _expected_bytes_dev(s.counts, s.lengths, mask)
            assert exp.numel() == nb and torch.equal(b.emit_data[:nb], exp), w
            for j in np.unique(rng.integers(0, E, 4)):
                p = int(want["parent"][j])
                exp = _expected_slot(int(offs[p]), s.states, s.lengths, p, int(s.counts[p]))
                lo, hi = int(want["off"][j]), int(want["off"][j + 1])
                assert np.array_equal(b.emit_data[lo:hi].cpu().numpy(), exp), (w, p)
                checked[0] += 1
        if w % 10 == 0:
            _say("  wave", w, "emitted", E)

    ctx.reserve(s.n_children, P, max(len(q) for q in s.waves))
    PL.streaming(ctx, b, on_wave)
    ctx.check("config5 streaming")
    ost.close()
    assert checked[0] > 20
