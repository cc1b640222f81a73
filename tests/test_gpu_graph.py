"""A streaming step captured in one HIP graph.

The step is the streaming sequence of the library: expand, stream reset, then
per wave the stream's batch, report and emission (Sec. 1 and Sec. 4: a parent
proceeds once all its children are terminal, in parent order).  It is
captured on the context's stream with a torch CUDA graph.  Every replay, with
eager steps and synchronisations between replays, must leave the same outputs
as an eager step, and the last wave's emission must equal the oracle's.  The
outputs are overwritten before each replay, so a replay that writes nothing
fails.
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
