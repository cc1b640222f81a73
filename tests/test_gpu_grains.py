"""GPU parity for Grain phases and the generation fence against the oracle:
case by case, and in lockstep over random schedules with retries, stale
and repeated reports."""
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

import oracle as O  # noqa: E402
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


def _phases(g, n):
    """(phase, generation) of every child, through ro_grains_read."""
    ph = torch.full((max(n, 1),), -1, dtype=torch.int32, device="cuda")
    gn = torch.full((max(n, 1),), -1, dtype=torch.int32, device="cuda")
    g.read(ph, gn)
    return ph.cpu().numpy().view(np.uint32)[:n], gn.cpu().numpy().view(np.uint32)[:n]


def _i32(a):
    a = np.ascontiguousarray(a, np.uint32)
    return D.to_dev(a.view(np.int32)) if len(a) else torch.zeros(1, dtype=torch.int32, device="cuda")


def _commit(ctx, g, par, ordi, st, off, data, gen, offs):
    n = len(par)
    out = torch.full((max(n, 1),), 0xEE, dtype=torch.uint8, device="cuda")
    cnt = torch.full((4,), -1, dtype=torch.int64, device="cuda")
    g.commit(_i32(par), _i32(ordi), D.to_dev(np.asarray(st, np.uint8)) if n else torch.zeros(1, dtype=torch.uint8, device="cuda"),
             D.to_dev(np.asarray(off, np.int64)), D.to_dev(np.asarray(data, np.uint8)), _i32(gen), D.to_dev(offs),
             out, cnt, n=n)
    ctx.check("commit")
    return out.cpu().numpy()[:n], tuple(int(x) for x in cnt.cpu().numpy())


def test_fence_cases(ctx):
    offs = O.expand(np.array([3], np.int32), tags=False)
    og = O.Grains(3)
    g = ctx.grains(3)
    gen = torch.zeros(3, dtype=torch.int32, device="cuda")
    g.dispatch(_i32([0, 1, 2]), gen)
    assert list(og.dispatch([0, 1, 2])) == list(gen.cpu().numpy())
    par = np.zeros(5, np.uint32)
    ordi = np.array([0, 0, 0, 1, 1], np.uint32)
    st = np.array([0, 0, 0, 0, 1], np.uint8)
    off = np.array([0, 1, 1, 2, 3, 3], np.int64)
    data = np.array([5, 6, 7], np.uint8)
    gn = np.array([0, 0, 0, 7, 0], np.uint32)
    want = og.commit(par, ordi, st, off, data, gn, offs)
    got = _commit(ctx, g, par, ordi, st, off, data, gn, offs)
    assert np.array_equal(got[0], want[0]) and got[1] == want[1]
    ph, gg = _phases(g, 3)
    assert np.array_equal(ph, og.phase()) and np.array_equal(gg, og.gen())
    g.retry(_i32([2]))
    og.retry([2])
    g.dispatch(_i32([2]), gen)
    assert int(gen[0].item()) == og.dispatch([2])[0] == 1
    g.dispatch(_i32([0]))                              # sealed: not ready
    assert ctx.status() == O.ESTATE
    g.retry(_i32([1]))                                 # not in flight
    assert ctx.status() == O.ESTATE
    g.dispatch(_i32([2, 2]))                           # named twice (already in flight anyway)
    assert ctx.status() == O.ESTATE
    ctx.check("after phase errors")
    g.close(); og.close()


@pytest.mark.parametrize("seed,fence_left", [(0, 0), (1, 0), (2, 0), (3, 2)])
def test_fence_lockstep_random_schedule(ctx, seed, fence_left):
    rng = np.random.default_rng(seed)
    counts = rng.integers(0, 7, 5000).astype(np.int32)
    offs, cp, co = O.expand(counts)
    N = int(offs[-1])
    outcomes = rng.choice(np.array([0, 0, 0, 1, 2], np.uint8), N)
    lens = rng.integers(0, 40, N)
    payload = rng.integers(0, 256, int(lens.sum()) + 1, dtype=np.uint8)
    poff = np.concatenate([[0], np.cumsum(lens)])
    og = O.Grains(N)
    g = ctx.grains(N)
    ctx.debug_epochs(grains=g, fence_left=fence_left)     # with 2: the fence epoch wraps after the 2nd commit
    ready = list(rng.permutation(N))
    committed = np.zeros(N, bool)
    old = []
    rounds = 0
    acc_par, acc_ord, acc_st, acc_data = [], [], [], []
    B = 1500
    _say("fence lockstep", seed, "N", N)
    while not committed.all():
        batch = np.array(ready[:B], np.uint32)
        ready = ready[B:]
        want_gen = og.dispatch(batch)
        gen = torch.zeros(max(len(batch), 1), dtype=torch.int32, device="cuda")
        g.dispatch(_i32(batch), gen, n=len(batch))
        ctx.check("dispatch")
        assert np.array_equal(gen.cpu().numpy().view(np.uint32)[:len(batch)], want_gen)
        groups = []                                          # [(child, generation, state, bytes), ...]
        for c, gv in old:
            if rng.random() < 0.3:
                groups.append([(c, gv, outcomes[c], b"late")])             # stale attempt
        for c, gv in zip(batch, want_gen):
            if rng.random() < 0.25:
                old.append((c, gv))                                         # lost: retried below
                continue
            b = bytes(payload[poff[c]:poff[c + 1]]) if outcomes[c] == 0 else b""
            grp = [(c, gv, outcomes[c], b)]
            u = rng.random()
            if u < 0.1:
                grp.append((c, gv, outcomes[c], b))                         # identical repeat
            elif u < 0.15:
                grp.append((c, gv, outcomes[c], b + b"x"))                  # conflicting repeat
            groups.append(grp)
        reps = [r for i in rng.permutation(len(groups)) for r in groups[i]]
        par = np.array([cp[r[0]] for r in reps], np.uint32)
        ordi = np.array([co[r[0]] for r in reps], np.uint32)
        st = np.array([r[2] for r in reps], np.uint8)
        gn = np.array([r[1] for r in reps], np.uint32)
        off = np.concatenate([[0], np.cumsum([len(r[3]) for r in reps])]).astype(np.int64)
        data = np.frombuffer(b"".join(r[3] for r in reps) + b"\0", np.uint8)
        want = og.commit(par, ordi, st, off, data, gn, offs)
        got = _commit(ctx, g, par, ordi, st, off, data, gn, offs)
        assert np.array_equal(got[0], want[0]) and got[1] == want[1], rounds
        acc = want[0] != O.PENDING
        committed[offs[par[acc]] + ordi[acc]] = True
        acc_par.append(par[acc]); acc_ord.append(ordi[acc]); acc_st.append(st[acc])
        acc_data += [reps[i][3] for i in np.flatnonzero(acc)]
        lost = np.array([c for c in batch if not committed[c]], np.uint32)
        if len(lost):
            og.retry(lost)
            g.retry(_i32(lost), n=len(lost))
            ready += list(lost)
        ph, gg = _phases(g, N)
        assert np.array_equal(ph, og.phase()), rounds
        assert np.array_equal(gg, og.gen()), rounds
        rounds += 1
    # what the fence committed is one report per child with its fixed outcome
    par = np.concatenate(acc_par); ordi = np.concatenate(acc_ord); st = np.concatenate(acc_st)
    off = np.concatenate([[0], np.cumsum([len(b) for b in acc_data])]).astype(np.int64)
    data = np.frombuffer(b"".join(acc_data) + b"\0", np.uint8)
    got = O.gather(par, ordi, st, off, data, offs)
    clean = O.gather(cp, co, outcomes, np.concatenate([[0], np.cumsum(np.where(outcomes == 0, lens, 0))]).astype(np.int64),
                     np.concatenate([payload[poff[c]:poff[c + 1]] for c in range(N) if outcomes[c] == 0] + [np.zeros(1, np.uint8)]),
                     offs)
    for k in ("out_off", "n_success", "n_failed", "n_skipped", "parent_state", "out_data"):
        assert np.array_equal(got[k], clean[k]), k
    _say("  rounds", rounds)
    g.close(); og.close()


def test_fence_empty_calls_and_reset(ctx):
    offs = O.expand(np.array([2, 0, 1], np.int32), tags=False)
    og = O.Grains(3)
    g = ctx.grains(3)
    e = torch.zeros(1, dtype=torch.int32, device="cuda")
    g.dispatch(e, n=0)
    g.retry(e, n=0)
    got = _commit(ctx, g, [], [], [], [0], [0], [], offs)
    want = og.commit(np.zeros(0, np.uint32), np.zeros(0, np.uint32), np.zeros(0, np.uint8), np.zeros(1, np.int64),
                     np.zeros(1, np.uint8), np.zeros(0, np.uint32), offs)
    assert got[1] == want[1] == (0, 0, 0, 0)
    g.dispatch(_i32([0, 2]))
    g.reset()
    ph, gn = _phases(g, 3)
    assert np.array_equal(ph, np.full(3, O.READY, np.uint32))
    assert np.array_equal(gn, np.zeros(3, np.uint32))
    g.close(); og.close()


def test_fence_trace_full(ctx):
    """The fence trace over the full single-level Zipf workload, in the
    benchmark's calls: dispatch generations, the state each report commits,
    the four counts and every grain's phase and generation, all in full."""
    import workloads as W
    c = W.config2()
    f = W.fence_trace(c)
    N = c.n_children
    r0, r1 = f.rounds
    _say("fence full: N", N, "reports", r0.n, r1.n)
    offs = O.expand(c.counts, tags=False)
    od = D.to_dev(offs)
    g = ctx.grains(N)
    g.reset()
    og = O.Grains(N)
    gen = torch.empty(len(f.dispatch0), dtype=torch.int32, device="cuda")
    g.dispatch(D.to_dev(f.dispatch0.view(np.int32)), gen)
    assert np.array_equal(gen.cpu().numpy().view(np.uint32), og.dispatch(f.dispatch0))
    for k, r in enumerate(f.rounds):
        if k == 1:
            lost = D.to_dev(f.lost.view(np.int32))
            g.retry(lost)
            og.retry(f.lost)
            gen1 = torch.empty(max(len(f.lost), 1), dtype=torch.int32, device="cuda")
            g.dispatch(lost, gen1, n=len(f.lost))
            assert np.array_equal(gen1.cpu().numpy().view(np.uint32)[:len(f.lost)], og.dispatch(f.lost))
        data = D.reports_data_dev(r)
        out = torch.empty(r.n, dtype=torch.uint8, device="cuda")
        cnt = torch.zeros(4, dtype=torch.int64, device="cuda")
        g.commit(D.to_dev(r.parent.view(np.int32)), D.to_dev(r.ordinal.view(np.int32)), D.to_dev(r.state),
                 D.to_dev(r.off), data, D.to_dev(r.generation.view(np.int32)), od, out, cnt)
        ctx.check(f"fence commit {k}")
        del data
        _say("  oracle commit", k)
        want_out, want_cnt = og.commit(r.parent, r.ordinal, r.state, r.off, r.repeated_data(), r.generation, offs)
        assert np.array_equal(out.cpu().numpy(), want_out), k
        assert tuple(int(x) for x in cnt.cpu().numpy()) == tuple(int(x) for x in want_cnt), k
    ph, gg = _phases(g, N)
    assert np.array_equal(ph, og.phase())
    assert np.array_equal(gg, og.gen())
    g.close(); og.close()


def test_fence_many_long_repeats(ctx):
    """Every child reported three times in one call: first copy, identical
    repeat, and a repeat of the same length with one byte changed (first,
    middle or last); records up to 5,000 bytes, so a wave queues more
    comparisons than it holds and a record spans several chunk rounds."""
    rng = np.random.default_rng(9)
    counts = rng.integers(1, 5, 400).astype(np.int32)
    offs = O.expand(counts, tags=False)
    N = int(offs[-1])
    par = np.repeat(np.arange(400, dtype=np.uint32), counts)
    ordi = (np.arange(N) - np.repeat(offs[:-1], counts)).astype(np.uint32)
    lens = rng.integers(1, 5001, N)
    recs = [rng.integers(0, 256, int(n), dtype=np.uint8) for n in lens]
    reps = []
    for c in range(N):
        alt = recs[c].copy()
        alt[[0, len(alt) // 2, len(alt) - 1][c % 3]] ^= 0x5A
        reps += [(c, recs[c]), (c, recs[c].copy()), (c, alt)]
    order = np.concatenate([np.arange(0, 3 * N, 3), rng.permutation(np.concatenate([np.arange(1, 3 * N, 3),
                                                                                    np.arange(2, 3 * N, 3)]))])
    reps = [reps[i] for i in order]
    rp = par[[r[0] for r in reps]]
    ro_ = ordi[[r[0] for r in reps]]
    st = np.zeros(len(reps), np.uint8)
    gn = np.zeros(len(reps), np.uint32)
    off = np.concatenate([[0], np.cumsum([len(r[1]) for r in reps])]).astype(np.int64)
    data = np.concatenate([r[1] for r in reps])
    og = O.Grains(N)
    g = ctx.grains(N)
    og.dispatch(np.arange(N, dtype=np.uint32))
    g.dispatch(_i32(np.arange(N)))
    want = og.commit(rp, ro_, st, off, data, gn, offs)
    got = _commit(ctx, g, rp, ro_, st, off, data, gn, offs)
    assert want[1] == (N, 0, N, N)
    assert np.array_equal(got[0], want[0]) and got[1] == tuple(want[1])
    g.close(); og.close()
