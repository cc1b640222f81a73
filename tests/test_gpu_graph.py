"""Steps of the library captured in one HIP graph.

A streaming step (expand, stream reset, then per wave the stream's batch,
report and emission: Sec. 1 and Sec. 4, a parent proceeds once all its
children are terminal, in parent order) and a nested documents step (two
expansions, two batches, a gather into the mid slots and an in-place gather
into the top slots: Sec. 4, nested F.expand / F.reduce) are each captured on
the context's stream with a torch CUDA graph.  Every replay, with eager steps
and synchronisations between replays, must leave the same outputs as an eager
step, and the eager step must equal the oracle.  The outputs are overwritten
before each replay, so a replay that writes nothing fails.
"""
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


def _outputs(b, P):
    torch.cuda.synchronize()
    sc = b.scalars.cpu().numpy().copy()
    E, nb = int(sc[2]), int(sc[3])
    cnt = b.emit_cnt.cpu().numpy()
    return dict(scalars=sc, parent=b.emit_parent.cpu().numpy().view(np.uint32)[:E].copy(),
                off=b.emit_off.cpu().numpy()[:E + 1].copy(), data=b.emit_data.cpu().numpy()[:nb].copy(),
                ns=cnt[:E].copy(), nf=cnt[P:P + E].copy(), nk=cnt[2 * P:2 * P + E].copy(),
                state=b.emit_state.cpu().numpy()[:E].copy())


def _same(a, b):
    return all(np.array_equal(a[k], b[k]) for k in a)


def _poison(b):
    b.scalars.fill_(-3)
    b.emit_parent.fill_(-3)
    b.emit_off.fill_(-3)
    b.emit_data.fill_(0xEE)
    b.emit_cnt.fill_(-3)
    b.emit_state.fill_(0xEE)


def test_stream_step_in_a_graph():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_18703_amd as R
    from paper_2609_18703_amd import pipeline as PL

    s = W.config5(n_parents=3000, n_children=60_000, n_waves=12)
    P, N = s.n_parents, s.n_children
    total = int(s.wave_reports[-1].off[-1])
    arena = np.zeros(total + 1, np.uint8)
    for rep in s.wave_reports:
        arena[int(rep.off[0]):int(rep.off[-1])] = rep.data()

    # oracle: the emission of the last wave
    offs = O.expand(s.counts, tags=False)
    ost = O.Stream(offs)
    for q, rep in zip(s.waves, s.wave_reports):
        _, par, ordi, _ = O.batch(q, None, offs, s.batch_size)
        ost.report(par, ordi, rep.state, rep.off, arena)
        want = ost.emit()
    ost.close()

    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        ctx = R.Context()
        b = PL.StreamingBuffers(D.to_dev(s.counts), [D.to_dev(q.view(np.int32)) for q in s.waves],
                                [D.to_dev(rep.state) for rep in s.wave_reports],
                                [D.to_dev(rep.off) for rep in s.wave_reports], D.to_dev(arena), N,
                                s.batch_size, total)
        ctx.reserve(N, P, max(len(q) for q in s.waves))
        ctx.expand(b.counts, b.offsets)
        st = ctx.stream(b.offsets, N)

        def step():
            PL.streaming(ctx, b, st=st)

        _say("graph: eager steps", P, N, len(s.waves))
        step()
        step()
        ctx.check("eager")
        eager = _outputs(b, P)
        E = int(eager["scalars"][2])
        assert E == len(want["parent"]) and int(eager["scalars"][3]) == want["n_bytes"]
        assert np.array_equal(eager["parent"], want["parent"])
        assert np.array_equal(eager["off"], want["off"])
        assert np.array_equal(eager["data"], want["data"])
        assert np.array_equal(eager["ns"], want["n_success"]) and np.array_equal(eager["nf"], want["n_failed"])
        assert np.array_equal(eager["nk"], want["n_skipped"])
        assert np.array_equal(eager["state"], want["parent_state"])

        _say("graph: capture")
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            step()
        torch.cuda.synchronize()
        try:
            for r in range(3):
                _poison(b)
                g.replay()
                ctx.check(f"replay {r}")
                _say("graph: replay", r)
                assert _same(_outputs(b, P), eager), r
                _poison(b)
                step()                      # eager work between replays
                ctx.check(f"eager after replay {r}")
                assert _same(_outputs(b, P), eager), r
        finally:
            del g
            torch.cuda.synchronize()
            st.close()
            ctx.close()


_NESTED_INPUTS = ("counts1", "queue1", "counts2", "queue2", "leaf_state", "leaf_off", "leaf_data")


def _nested_outputs(b):
    torch.cuda.synchronize()
    return {k: v.cpu().numpy().copy() for k, v in vars(b).items()
            if isinstance(v, torch.Tensor) and k not in _NESTED_INPUTS}


def test_nested_step_in_a_graph():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_18703_amd as R
    from paper_2609_18703_amd import pipeline as PL

    n = W.config3(n_docs=300)
    r = n.reports
    data = r.data()
    want = O.nested(n.counts1, n.queue1, None, n.batch1, n.counts2, n.queue2, None, n.batch2,
                    r.state, r.off, data)
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        ctx = R.Context()
        b = PL.NestedBuffers(D.to_dev(n.counts1), D.to_dev(n.queue1.view(np.int32)), n.batch1,
                             D.to_dev(n.counts2), D.to_dev(n.queue2.view(np.int32)), n.batch2,
                             D.to_dev(r.state), D.to_dev(r.off), D.to_dev(data), len(n.queue1),
                             len(n.queue2), upper_in_place=True)
        ctx.reserve(b.N2, b.N1, b.N2)

        def step():
            PL.nested(ctx, b)

        _say("graph: nested eager steps", b.P1, b.N1, b.N2)
        step()
        step()
        ctx.check("eager")
        eager = _nested_outputs(b)
        N1, P1 = b.N1, b.P1
        low, up = want["low"], want["up"]
        assert np.array_equal(eager["offsets1"][:P1 + 1], want["offsets1"])
        assert np.array_equal(eager["offsets2"][:N1 + 1], want["offsets2"])
        assert np.array_equal(eager["mid_off"][:N1 + 1], low["out_off"])
        assert np.array_equal(eager["mid_data"][:int(low["out_off"][-1])], low["out_data"])
        assert np.array_equal(eager["top_off"][:P1 + 1], up["out_off"])
        assert np.array_equal(eager["top_state"][:P1], up["parent_state"])
        assert np.array_equal(eager["top_cnt"][:P1], up["n_success"])

        _say("graph: nested capture")
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            step()
        torch.cuda.synchronize()
        try:
            for k in range(3):
                for name in eager:
                    getattr(b, name).fill_(7)
                g.replay()
                ctx.check(f"nested replay {k}")
                _say("graph: nested replay", k)
                got = _nested_outputs(b)
                assert all(np.array_equal(got[x], eager[x]) for x in eager), k
                for name in eager:
                    getattr(b, name).fill_(7)
                step()
                ctx.check(f"nested eager after replay {k}")
                got = _nested_outputs(b)
                assert all(np.array_equal(got[x], eager[x]) for x in eager), k
        finally:
            del g
            torch.cuda.synchronize()
            ctx.close()
