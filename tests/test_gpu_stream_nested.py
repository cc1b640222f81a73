"""GPU parity for nested composition and streaming completion (HIP path vs the
CPU oracle, bit-exact)."""
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

import oracle as O  # noqa: E402
import workloads as W  # noqa: E402
from workloads import device as D  # noqa: E402


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def ctx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_18703_amd as R
    c = R.Context()
    c.reserve(1 << 22, 1 << 20, 1 << 22)
    yield c
    c.close()


def _i32(a):
    return D.to_dev(np.ascontiguousarray(a).view(np.int32))


def _u32(t, n):
    return t.cpu().numpy().view(np.uint32)[:n]


# ------------------------------------------------------------------ nested
def _nested_case(ctx, n, upper_in_place=False):
    from paper_2609_18703_amd import pipeline as PL
    r = n.reports
    data = r.data()
    b = PL.NestedBuffers(D.to_dev(n.counts1), _i32(n.queue1), n.batch1, D.to_dev(n.counts2), _i32(n.queue2),
                         n.batch2, D.to_dev(r.state), D.to_dev(r.off), D.to_dev(data), len(n.queue1),
                         len(n.queue2), upper_in_place=upper_in_place)
    PL.nested(ctx, b)
    ctx.check("nested")
    want = O.nested(n.counts1, n.queue1, None, n.batch1, n.counts2, n.queue2, None, n.batch2,
                    r.state, r.off, data)
    N1, P1 = b.N1, b.P1
    assert np.array_equal(b.offsets1.cpu().numpy()[:P1 + 1], want["offsets1"])
    assert np.array_equal(b.offsets2.cpu().numpy()[:N1 + 1], want["offsets2"])
    assert np.array_equal(_u32(b.mid_parent, N1), want["parent1"])
    assert np.array_equal(_u32(b.b1_parent, N1), want["batch1"][1])
    assert np.array_equal(_u32(b.b2_parent, b.N2), want["batch2"][1])
    low, up = want["low"], want["up"]
    assert np.array_equal(b.mid_off.cpu().numpy()[:N1 + 1], low["out_off"])
    assert np.array_equal(b.mid_state.cpu().numpy()[:N1], low["parent_state"])
    assert np.array_equal(b.mid_cnt.cpu().numpy()[N1:2 * N1], low["n_failed"])
    assert np.array_equal(b.mid_data.cpu().numpy()[:int(low["out_off"][-1])], low["out_data"])
    assert np.array_equal(b.top_off.cpu().numpy()[:P1 + 1], up["out_off"])
    assert np.array_equal(b.top_state.cpu().numpy()[:P1], up["parent_state"])
    assert np.array_equal(b.top_complete.cpu().numpy()[:P1], up["complete"])
    assert np.array_equal(b.top_cnt.cpu().numpy()[:P1], up["n_success"])
    assert np.array_equal(b.top_cnt.cpu().numpy()[P1:2 * P1], up["n_failed"])
    assert np.array_equal(b.top_data.cpu().numpy()[:int(up["out_off"][-1])], up["out_data"])


@pytest.mark.parametrize("n_docs", [1, 37, 400])
def test_nested_documents_upper_in_place(ctx, n_docs):
    """No region fails, so each document slot is its pages' slots as they
    already lie: the upper gather aliases the page buffer and copies nothing,
    with the same results as a separate buffer."""
    _say("nested docs in place", n_docs)
    _nested_case(ctx, W.config3(n_docs=n_docs), upper_in_place=True)


def test_nested_upper_in_place_rejects_moves(ctx):
    """With a failed frame, clips drop out of their video's slot and later
    clips would have to move: an in-place upper gather is RO_EINVAL."""
    from paper_2609_18703_amd import pipeline as PL
    n = W.config4(n_videos=40)
    assert (n.states == W.FAILED).any()
    r = n.reports
    b = PL.NestedBuffers(D.to_dev(n.counts1), _i32(n.queue1), n.batch1, D.to_dev(n.counts2), _i32(n.queue2),
                         n.batch2, D.to_dev(r.state), D.to_dev(r.off), D.to_dev(r.data()), len(n.queue1),
                         len(n.queue2), upper_in_place=True)
    PL.nested(ctx, b)
    assert ctx.status() == O.EINVAL
    ctx.check("after in-place rejection")


@pytest.mark.parametrize("n_docs", [1, 37, 400])
def test_nested_documents(ctx, n_docs):
    _say("nested docs", n_docs)
    _nested_case(ctx, W.config3(n_docs=n_docs))


@pytest.mark.parametrize("n_videos", [3, 30])
def test_nested_videos_with_failed_frames(ctx, n_videos):
    _say("nested videos", n_videos)
    _nested_case(ctx, W.config4(n_videos=n_videos))


def test_nested_canonical_order(ctx):
    _nested_case(ctx, W.config3(n_docs=120, canonical_order=True))


# ------------------------------------------------------------------ streaming
def _stream_case(ctx, counts, waves, B=64, runs=1, run_left=0):
    """waves: list of (child ids, states, lengths); all reports of a wave are in
    its queue order; bytes of every wave live in one arena.  With runs > 1 the
    whole stream is replayed on one stream state, reset between runs."""
    from paper_2609_18703_amd import pipeline as PL
    counts = np.asarray(counts, np.int32)
    offs = O.expand(counts, tags=False)
    N = int(offs[-1])
    rng = np.random.default_rng(len(waves) + N)
    offsets_list, states, arena_parts, base = [], [], [], 0
    for (ids, st, ln) in waves:
        ln = np.where(st == W.SUCCESS, ln, 0).astype(np.int64)
        off = base + np.concatenate([[0], np.cumsum(ln)]).astype(np.int64)
        offsets_list.append(off)
        states.append(np.asarray(st, np.uint8))
        arena_parts.append(rng.integers(0, 256, int(ln.sum()), dtype=np.uint8))
        base = int(off[-1])
    arena = np.concatenate(arena_parts + [np.zeros(1, np.uint8)])
    # oracle, wave by wave
    ost = O.Stream(offs)
    want = []
    for (ids, _, _), st, off in zip(waves, states, offsets_list):
        _, par, ordi, _ = O.batch(np.asarray(ids, np.uint32), None, offs, B)
        ost.report(par, ordi, st, off, arena)
        want.append(ost.emit())
    ost.close()
    # GPU
    b = PL.StreamingBuffers(D.to_dev(counts) if len(counts) else torch.zeros(1, dtype=torch.int32, device="cuda")[:0],
                            [_i32(np.asarray(w[0], np.uint32)) for w in waves],
                            [D.to_dev(s) for s in states], [D.to_dev(o) for o in offsets_list],
                            D.to_dev(arena), N, B, max(base, 1))
    P = len(counts)
    got = []

    def on_wave(w):
        sc = b.scalars.cpu().numpy()
        E, nb = int(sc[2]), int(sc[3])
        got.append(dict(parent=_u32(b.emit_parent, E), off=b.emit_off.cpu().numpy()[:E + 1],
                        data=b.emit_data.cpu().numpy()[:nb], ns=b.emit_cnt.cpu().numpy()[:E],
                        nf=b.emit_cnt.cpu().numpy()[P:P + E], nk=b.emit_cnt.cpu().numpy()[2 * P:2 * P + E],
                        state=b.emit_state.cpu().numpy()[:E], nbytes=nb))
    if runs == 1:
        PL.streaming(ctx, b, on_wave)
    else:
        ctx.expand(b.counts, b.offsets)          # the stream validates its offsets when created
        st = ctx.stream(b.offsets, N)
        ctx.debug_epochs(stream=st, run_left=run_left)
        for _ in range(runs):
            PL.streaming(ctx, b, on_wave, st=st)
        st.close()
    ctx.check("stream")
    assert len(got) == runs * len(want)
    for w, (g, o) in enumerate(zip(got, want * runs)):
        assert np.array_equal(g["parent"], o["parent"]), w
        assert np.array_equal(g["off"], o["off"]), w
        assert g["nbytes"] == o["n_bytes"], w
        assert np.array_equal(g["data"], o["data"]), w
        assert np.array_equal(g["ns"], o["n_success"]) and np.array_equal(g["nf"], o["n_failed"]), w
        assert np.array_equal(g["nk"], o["n_skipped"]) and np.array_equal(g["state"], o["parent_state"]), w
    return got


def test_stream_config5_shape(ctx):
    s = W.config5(n_parents=3000, n_children=40_000, n_waves=6)
    waves = [(q, r.state, np.diff(r.off)) for q, r in zip(s.waves, s.wave_reports)]
    _say("stream config5-shaped", len(waves))
    _stream_case(ctx, s.counts, waves, B=s.batch_size)


@pytest.mark.parametrize("run_left", [0, 2])
def test_stream_reset_replays(ctx, run_left):
    """A reset stream forgets every report and emission: three runs over one
    stream state give the oracle's emissions each time (empty parents are
    emitted again by each run's first call).  With run_left the slot epoch
    wraps after the second reset (test aid)."""
    rng = np.random.default_rng(21)
    counts = rng.integers(0, 9, 4000).astype(np.int32)
    N = int(counts.sum())
    parts = np.split(rng.permutation(N).astype(np.uint32), [N // 3, N // 2])
    waves = [(ids, rng.choice(np.array([0, 0, 1, 2], np.uint8), len(ids)),
              rng.integers(1, 200, len(ids)).astype(np.int64)) for ids in parts]
    _say("stream reset replays", [len(p) for p in parts])
    got = _stream_case(ctx, counts, waves, B=100, runs=3, run_left=run_left)
    empties = set(np.flatnonzero(counts == 0).tolist())
    assert empties
    for r in range(3):
        assert empties <= set(got[r * len(waves)]["parent"].tolist()), r


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_stream_mixed_states_and_empty_parents(ctx, seed):
    rng = np.random.default_rng(seed)
    counts = rng.integers(0, 6, 5000).astype(np.int32)
    counts[:7] = 0                        # empty expansions: emitted by the first call
    N = int(counts.sum())
    perm = rng.permutation(N).astype(np.uint32)
    cuts = np.sort(rng.integers(0, N + 1, 4))
    parts = np.split(perm, cuts)
    waves = []
    for ids in parts:
        st = rng.choice(np.array([0, 0, 0, 1, 2], np.uint8), len(ids))
        ln = rng.choice(np.array([0, 1, 15, 16, 17, 64, 300], np.int64), len(ids))
        waves.append((ids, st, ln))
    _say("stream mixed", seed, [len(p) for p in parts])
    got = _stream_case(ctx, counts, waves, B=37)
    assert set(range(7)) <= set(got[0]["parent"].tolist())


def test_stream_empty_runs(ctx):
    """Runs of thousands of empty parents: the first emission's 1,024-child
    scan tiles span more emitted parents than they hold children (their
    parent search runs in global memory), and later waves emit parents far
    apart."""
    rng = np.random.default_rng(33)
    counts = np.concatenate([rng.integers(1, 5, 500), np.zeros(3000), rng.integers(0, 3, 2000), np.zeros(5000),
                             [3000], np.zeros(2000), rng.integers(0, 4, 800)]).astype(np.int32)
    N = int(counts.sum())
    parts = np.split(rng.permutation(N).astype(np.uint32), [N // 4, N // 2, (3 * N) // 4])
    waves = [(ids, rng.choice(np.array([0, 0, 0, 1, 2], np.uint8), len(ids)),
              rng.choice(np.array([0, 1, 16, 33, 200], np.int64), len(ids))) for ids in parts]
    _say("stream empty runs", len(counts), N, [len(p) for p in parts])
    got = _stream_case(ctx, counts, waves, B=64)
    assert set(np.flatnonzero(counts == 0).tolist()) <= set(got[0]["parent"].tolist())


def test_stream_single_wave_equals_gather(ctx):
    """One wave holding every report emits every parent: the same slots as a
    one-shot gather."""
    c = W.config2(n_parents=900)
    r = c.reports
    offs = O.expand(c.counts, tags=False)
    order = np.concatenate([c.queue[c.keep == 1], c.sealed_ids])
    got = _stream_case(ctx, c.counts, [(order, r.state, np.diff(r.off))], B=256)
    g = O.gather(*O.batch(order, None, offs, 256)[1:3], r.state, r.off, r.data(), offs)
    assert np.array_equal(got[0]["parent"], np.arange(c.n_parents))
    assert np.array_equal(got[0]["off"], g["out_off"])


def test_stream_duplicate_across_waves(ctx):
    from paper_2609_18703_amd import pipeline as PL
    counts = np.array([3, 2], np.int32)
    waves = [np.array([0, 1], np.uint32), np.array([1, 4], np.uint32)]   # child 1 twice
    b = PL.StreamingBuffers(D.to_dev(counts), [_i32(w) for w in waves],
                            [D.to_dev(np.zeros(2, np.uint8))] * 2,
                            [D.to_dev(np.array([0, 1, 2], np.int64)), D.to_dev(np.array([2, 3, 4], np.int64))],
                            D.to_dev(np.zeros(8, np.uint8)), 5, 4, 8)
    PL.streaming(ctx, b)
    assert ctx.status() == O.EDUP
    ctx.check("after duplicate")


def test_stream_batch_matches_batch_and_oracle(ctx):
    """A stream's own batch (parents from the map it built at creation) gives
    the slots, tags and counts of the oracle's FIFO batch, with and without a
    ready mask, with the stream's barrier, and rejects ids past the
    expansion."""
    import paper_2609_18703_amd as R
    rng = np.random.default_rng(21)
    counts = rng.integers(0, 12, 30_000).astype(np.int32)
    counts[5] = 20_000
    offs = O.expand(counts, tags=False)
    N = int(offs[-1])
    od = D.to_dev(offs)
    bar = torch.zeros(len(counts), dtype=torch.uint8, device="cuda")
    st = ctx.stream(od, N, barrier=bar)
    try:
        for wave, (Q, masked, barred) in enumerate([(50_000, False, False), (7_000, True, False),
                                                     (N, True, False), (30_000, False, True)]):
            q = rng.choice(N, Q, replace=False).astype(np.uint32)
            keep = (rng.random(Q) < 0.8).astype(np.uint8) if masked else None
            hb = np.zeros(len(counts), np.uint8)
            if barred:
                hb[rng.random(len(counts)) < 0.3] = 1
            bar.copy_(torch.from_numpy(hb))
            oc = torch.full((Q,), -1, dtype=torch.int32, device="cuda")
            op = torch.full((Q,), -1, dtype=torch.int32, device="cuda")
            oo = torch.full((Q,), -1, dtype=torch.int32, device="cuda")
            sc = torch.full((2,), -1, dtype=torch.int64, device="cuda")
            st.batch(_i32(q), None if keep is None else D.to_dev(keep), 1024, oc, op, oo, sc[0:1], sc[1:2])
            ctx.check(f"stream batch wave {wave}")
            want = O.batch(q, keep, offs, 1024, barrier=hb if barred else None)
            m = int(sc[0].item())
            assert m == len(want[0]) and int(sc[1].item()) == len(want[3]), wave
            assert np.array_equal(_u32(oc, m), want[0]), wave
            assert np.array_equal(_u32(op, m), want[1]), wave
            assert np.array_equal(_u32(oo, m), want[2]), wave
        bar.zero_()
        bad = np.array([0, N, 3], np.uint32)
        t = torch.zeros(9, dtype=torch.int32, device="cuda")
        st.batch(_i32(bad), None, 4, t[0:3], t[3:6], t[6:9])
        assert ctx.status() == R.ERANGE
        # tag arrays sharing memory are rejected on the host
        with pytest.raises(R.RoError) as e:
            st.batch(_i32(bad), None, 4, t[0:3], t[2:5], None)
        assert e.value.code == R.EINVAL
    finally:
        st.close()
