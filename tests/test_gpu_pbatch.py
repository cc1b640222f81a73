"""GPU parity for parent-bound reservation against the oracle: every slot's
child, parent and ordinal and every batch boundary, bit-exact."""
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


def _run(ctx, queue, keep, offs, B, barrier=None, out_cap=None, batch_cap=None):
    Q = len(queue)
    cap = Q if out_cap is None else out_cap
    bcap = Q + 1 if batch_cap is None else batch_cap
    q = D.to_dev(np.ascontiguousarray(queue, np.uint32).view(np.int32)) if Q else \
        torch.zeros(1, dtype=torch.int32, device="cuda")
    k = None if keep is None else (D.to_dev(np.asarray(keep, np.uint8)) if Q else
                                   torch.zeros(1, dtype=torch.uint8, device="cuda"))
    bar = None if barrier is None else D.to_dev(np.asarray(barrier, np.uint8))
    oc = torch.full((max(cap, 1),), -1, dtype=torch.int32, device="cuda")
    op = torch.full((max(cap, 1),), -1, dtype=torch.int32, device="cuda")
    oo = torch.full((max(cap, 1),), -1, dtype=torch.int32, device="cuda")
    boff = torch.full((max(bcap, 1),), -1, dtype=torch.int64, device="cuda")
    sc = torch.full((2,), -1, dtype=torch.int64, device="cuda")
    ctx.batch_parent(q, k, D.to_dev(offs), B, boff[:bcap], oc, op, oo, sc[0:1], sc[1:2], q_len=Q, out_cap=cap,
                     barrier=bar)
    return oc, op, oo, boff, sc


def _check(ctx, queue, keep, offs, B, barrier=None, what=""):
    want = O.batch(queue, keep, offs, B, barrier=barrier, parent_bound=True)
    oc, op, oo, boff, sc = _run(ctx, queue, keep, offs, B, barrier)
    ctx.check(what)
    m, nb = (int(x) for x in sc.cpu().numpy())
    assert m == len(want[0]) and nb == len(want[3]), what
    u32 = lambda t: t.cpu().numpy().view(np.uint32)[:m]
    assert np.array_equal(u32(oc), want[0]), what
    assert np.array_equal(u32(op), want[1]), what
    assert np.array_equal(u32(oo), want[2]), what
    assert np.array_equal(boff.cpu().numpy()[:nb + 1], np.concatenate([[0], np.cumsum(want[3])])), what


@pytest.mark.parametrize("P,B,seed", [(1, 4, 0), (2, 3, 1), (7, 1, 2), (300, 16, 3), (513, 5, 4), (513, 512, 5),
                                      (5000, 64, 6), (70_000, 256, 7), (70_000, 1 << 30, 8)])
def test_pbatch_random(ctx, P, B, seed):
    rng = np.random.default_rng(seed)
    counts = rng.integers(0, 9, P).astype(np.int32)
    if P > 1:
        counts[rng.integers(0, P)] = 9000                   # one parent spans several sort tiles
    offs = O.expand(counts, tags=False)
    N = int(offs[-1])
    queue = rng.permutation(N).astype(np.uint32)
    keep = (rng.random(N) < 0.9).astype(np.uint8)
    _say("pbatch", P, B, seed, "N", N)
    _check(ctx, queue, keep, offs, B, what=f"P={P} B={B} keep")
    _check(ctx, queue, None, offs, B, what=f"P={P} B={B} all")
    bar = (rng.random(P) < 0.2).astype(np.uint8)
    _check(ctx, queue, keep, offs, B, barrier=bar, what=f"P={P} B={B} barrier")


def test_pbatch_partial_queue_and_edges(ctx):
    rng = np.random.default_rng(11)
    counts = rng.integers(0, 5, 2000).astype(np.int32)
    offs = O.expand(counts, tags=False)
    N = int(offs[-1])
    q = rng.choice(N, N // 3, replace=False).astype(np.uint32)     # a queue holding some children only
    _check(ctx, q, None, offs, 7, what="partial queue")
    _check(ctx, np.zeros(0, np.uint32), None, offs, 7, what="empty queue")
    _check(ctx, q, np.zeros(len(q), np.uint8), offs, 7, what="nothing ready")
    # canonical order: every parent's entries are already together
    _check(ctx, np.arange(N, dtype=np.uint32), None, offs, 3, what="canonical order")


def test_pbatch_errors(ctx):
    import paper_2609_18703_amd as R
    offs = O.expand(np.array([3, 2], np.int32), tags=False)
    q = np.array([4, 0, 1, 3, 2], np.uint32)
    _run(ctx, q, None, offs, 2, out_cap=3)
    assert ctx.status() == R.ECAP
    _run(ctx, q, None, offs, 2, batch_cap=3)                       # 4 batches need 5 offsets
    assert ctx.status() == R.ECAP
    _run(ctx, np.array([0, 9], np.uint32), None, offs, 2)
    assert ctx.status() == R.ERANGE
    _check(ctx, q, None, offs, 2, what="after errors")


def test_pbatch_zipf_full(ctx):
    """The 41M-child Zipf workload's ready queue (sealed children masked out),
    B = 256, in full."""
    c = W.config2()
    offs = O.expand(c.counts, tags=False)
    _say("pbatch zipf full: Q", len(c.queue))
    _check(ctx, c.queue, c.keep, offs, c.batch_size, what="zipf full")
