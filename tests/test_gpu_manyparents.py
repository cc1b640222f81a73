"""Parent-heavy shapes: millions of parents with zero to three children
each (a quarter of them empty), so that a scan tile covers thousands of
parents and the per-parent passes, not the per-child ones, carry the work.
The single-level chain and a ten-wave stream against the oracle, every
output in full."""
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


def test_single_level_six_million_parents(ctx):
    from paper_2609_18703_amd import pipeline as PL
    c = W.single_level("parent-heavy", 21, lambda r: r.integers(0, 4, 6_000_000),
                       lambda r, n: r.integers(0, 41, n), 0.04, 0.03, 256)
    _say("many parents: P =", c.n_parents, "N =", c.n_children)
    b = G.stage_single(c)
    ctx.reserve(c.n_children, c.n_parents, c.n_children)
    PL.single_level(ctx, b)
    ctx.check("parent-heavy single level")
    G.compare_single(b, G.oracle_single(c))


def test_stream_three_million_parents(ctx):
    from paper_2609_18703_amd import pipeline as PL
    s = W.streaming("parent-heavy streaming", 22, lambda r: r.integers(0, 4, 3_000_000),
                    lambda r, n: r.integers(0, 65, n), 10, 512)
    P = s.n_parents
    _say("many parents streaming: P =", P, "N =", s.n_children, "waves =", len(s.waves))
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
    host_arena = np.concatenate([rep.data() for rep in s.wave_reports]) if total else np.zeros(1, np.uint8)
    emitted = [0]

    def on_wave(w):
        q, rep = s.waves[w], s.wave_reports[w]
        _, par, ordi, _ = O.batch(q, None, offs, s.batch_size)
        ost.report(par, ordi, rep.state, rep.off, host_arena)
        want = ost.emit()
        sc = b.scalars.cpu().numpy()
        E, nb = int(sc[2]), int(sc[3])
        assert E == len(want["parent"]) and nb == want["n_bytes"], w
        assert np.array_equal(G.u32(b.emit_parent)[:E], want["parent"]), w
        assert np.array_equal(b.emit_off.cpu().numpy()[:E + 1], want["off"]), w
        assert np.array_equal(b.emit_cnt.cpu().numpy()[:E], want["n_success"]), w
        assert np.array_equal(b.emit_state.cpu().numpy()[:E], want["parent_state"]), w
        assert np.array_equal(b.emit_data[:nb].cpu().numpy(), want["data"]), w
        emitted[0] += E
        _say("  wave", w, "emitted", E)

    ctx.reserve(s.n_children, P, max(len(q) for q in s.waves))
    PL.streaming(ctx, b, on_wave)
    ctx.check("parent-heavy streaming")
    ost.close()
    assert emitted[0] == P
