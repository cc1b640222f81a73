"""GPU parity for F.filter and F.broadcast against the oracle."""
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
    yield c
    c.close()


STATES = np.array([0, 0, 0, 1, 2, 3], np.uint8)


@pytest.mark.parametrize("n", [1, 15, 16, 17, 4095, 100_003])
@pytest.mark.parametrize("shift", [0, 3])
@pytest.mark.parametrize("with_mask_state", [False, True])
def test_filter_matches_oracle(ctx, n, shift, with_mask_state):
    rng = np.random.default_rng(n + shift)
    xs = rng.choice(STATES, n)
    ms = rng.choice(STATES, n) if with_mask_state else None
    mv = (rng.random(n) < 0.5).astype(np.uint8)
    want = O.filter(xs, mv, ms)

    def dev(a):   # misaligned views take the bytewise path
        t = torch.zeros(n + 16, dtype=torch.uint8, device="cuda")
        t[shift:shift + n] = torch.from_numpy(a).cuda()
        return t[shift:shift + n]
    out = dev(np.zeros(n, np.uint8))
    _say("filter", n, shift, with_mask_state)
    ctx.filter(dev(xs), dev(mv), out, mask_state=None if ms is None else dev(ms))
    ctx.check("filter")
    assert np.array_equal(out.cpu().numpy(), want)


def test_filter_bad_state(ctx):
    xs = torch.tensor([0, 4, 0], dtype=torch.uint8, device="cuda")
    mv = torch.ones(3, dtype=torch.uint8, device="cuda")
    out = torch.zeros(3, dtype=torch.uint8, device="cuda")
    ctx.filter(xs, mv, out)
    assert ctx.status() == O.ESTATE
    ctx.check("after bad state")


@pytest.mark.parametrize("levels", [1, 2, 3])
def test_broadcast_matches_oracle(ctx, levels):
    rng = np.random.default_rng(levels)
    counts = [rng.integers(0, 6, 3000).astype(np.int32)]
    maps = []
    for _ in range(levels):
        offs, cp, _ = O.expand(counts[-1])
        maps.insert(0, cp)
        counts.append(rng.integers(0, 6, int(offs[-1])).astype(np.int32))
    n = len(maps[0])
    x = rng.choice(STATES, len(counts[0]))
    like = rng.choice(STATES, n)
    anc, st = O.broadcast(maps, x, like)
    d_anc = torch.zeros(max(n, 1), dtype=torch.int32, device="cuda")
    d_st = torch.zeros(max(n, 1), dtype=torch.uint8, device="cuda")
    _say("broadcast levels", levels, "n", n)
    ctx.broadcast([D.to_dev(m.view(np.int32)) for m in maps], D.to_dev(x), d_st, d_anc, D.to_dev(like))
    ctx.check("broadcast")
    assert np.array_equal(d_anc.cpu().numpy().view(np.uint32)[:n], anc)
    assert np.array_equal(d_st.cpu().numpy()[:n], st)


def test_broadcast_documents_to_regions(ctx):
    """Two levels at the documents workload's full size: each region gets its
    document's Item, with the propagation rule over the region's own state."""
    nw = W.config3()
    o1, p1, _ = O.expand(nw.counts1)
    o2, p2, _ = O.expand(nw.counts2)
    rng = np.random.default_rng(3)
    x = rng.choice(STATES, len(nw.counts1))
    anc, st = O.broadcast([p2, p1], x, nw.states)
    n = len(p2)
    d_anc = torch.zeros(n, dtype=torch.int32, device="cuda")
    d_st = torch.zeros(n, dtype=torch.uint8, device="cuda")
    _say("broadcast documents -> regions", n)
    ctx.broadcast([D.to_dev(p2.view(np.int32)), D.to_dev(p1.view(np.int32))], D.to_dev(x), d_st, d_anc,
                  D.to_dev(nw.states))
    ctx.check("broadcast documents")
    assert np.array_equal(d_anc.cpu().numpy().view(np.uint32), anc)
    assert np.array_equal(d_st.cpu().numpy(), st)


@pytest.mark.parametrize("like", [True, False])
def test_broadcast_eight_levels(ctx, like):
    """The deepest broadcast the library takes (8 composed maps), with and
    without the descendant's own state, and without the ancestor output."""
    rng = np.random.default_rng(8 + like)
    counts = [rng.integers(1, 4, 5).astype(np.int32)]
    maps = []
    for _ in range(8):
        offs, cp, _ = O.expand(counts[-1])
        maps.insert(0, cp)
        counts.append(rng.integers(0, 4, int(offs[-1])).astype(np.int32))
    n = len(maps[0])
    x = rng.choice(STATES, len(counts[0]))
    ls = rng.choice(STATES, n) if like else None
    anc, st = O.broadcast(maps, x, ls)
    d_st = torch.zeros(max(n, 1), dtype=torch.uint8, device="cuda")
    _say("broadcast 8 levels, n", n, "like", like)
    ctx.broadcast([D.to_dev(m.view(np.int32)) for m in maps], D.to_dev(x), d_st, None,
                  D.to_dev(ls) if like else None)
    ctx.check("broadcast 8 levels")
    assert np.array_equal(d_st.cpu().numpy()[:n], st)


def test_broadcast_errors(ctx):
    import paper_2609_18703_amd as R
    m = D.to_dev(np.array([0, 1, 1, 2], np.int32))
    x = D.to_dev(np.array([0, 0, 1], np.uint8))
    out = torch.zeros(4, dtype=torch.uint8, device="cuda")
    with pytest.raises(R.RoError) as e:                          # more than 8 levels, refused on the host
        ctx.broadcast([m] * 9, x, out)
    assert e.value.code == O.EINVAL
    ctx.broadcast([m], D.to_dev(np.array([0, 0], np.uint8)), out)    # ancestor 2 of 2 ancestors
    assert ctx.status() == O.ERANGE
    # an intermediate index past the next map's end is refused before it is read
    short = D.to_dev(np.array([0, 0], np.int32))
    ctx.broadcast([m, short], x, out)
    assert ctx.status() == O.ERANGE
    ctx.broadcast([m], x, out)
    ctx.check("after the range error")
    assert np.array_equal(out.cpu().numpy(), np.array([0, 0, 0, 1], np.uint8))
