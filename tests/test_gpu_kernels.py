"""GPU parity per entry point: HIP path vs the CPU oracle, bit-exact, on edge
shapes that span several tiles and ragged tails."""
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
    c.reserve(1 << 20, 1 << 18, 1 << 20)
    yield c
    c.close()


def _u32(t, n):
    return t.cpu().numpy().view(np.uint32)[:n]


COUNT_CASES = {
    "empty": np.zeros(0, np.int32),
    "all_zero": np.zeros(7, np.int32),
    "single": np.array([5], np.int32),
    "zeros_between": np.array([0, 3, 0, 0, 2, 0], np.int32),
    "tile_minus_1": np.ones(4095, np.int32),
    "tile": np.ones(4096, np.int32),
    "tile_plus_1": np.ones(4097, np.int32),
    "big_parent": np.array([2, 100_000, 0, 3], np.int32),
    "random_multi_tile": None,
    "long_empty_run": np.concatenate([[4], np.zeros(20_000, np.int32), [7]]).astype(np.int32),
}


def _counts(name):
    c = COUNT_CASES[name]
    if c is None:
        rng = np.random.default_rng(3)
        c = rng.integers(0, 6, 30_001).astype(np.int32)
        c[rng.random(len(c)) < 0.2] = 0
    return c


@pytest.mark.parametrize("name", list(COUNT_CASES))
def test_expand_matches_oracle(ctx, name):
    counts = _counts(name)
    _say("expand", name, len(counts))
    offs, par, ordi = O.expand(counts)
    N = int(offs[-1])
    d_off = torch.empty(len(counts) + 1, dtype=torch.int64, device="cuda")
    d_par = torch.full((max(N, 1),), -1, dtype=torch.int32, device="cuda")
    d_ord = torch.full((max(N, 1),), -1, dtype=torch.int32, device="cuda")
    ctx.expand(D.to_dev(counts) if len(counts) else torch.zeros(1, dtype=torch.int32, device="cuda")[:0],
               d_off, d_par, d_ord)
    ctx.check("expand")
    assert np.array_equal(d_off.cpu().numpy(), offs)
    assert np.array_equal(_u32(d_par, N), par)
    assert np.array_equal(_u32(d_ord, N), ordi)


def test_expand_errors(ctx):
    d_off = torch.empty(4, dtype=torch.int64, device="cuda")
    ctx.expand(D.to_dev(np.array([1, -2, 3], np.int32)), d_off)
    assert ctx.status() == O.EINVAL
    small = torch.empty(3, dtype=torch.int32, device="cuda")
    ctx.expand(D.to_dev(np.array([2, 2, 2], np.int32)), d_off, small, small.clone())
    assert ctx.status() == O.ECAP
    ctx.expand(D.to_dev(np.full(3, 2 ** 31 - 1, np.int32)), d_off)
    assert ctx.status() == O.EOVERFLOW
    ctx.check("after errors")


def _batch_case(ctx, counts, queue, keep, B):
    offs = O.expand(counts, tags=False)
    Q = len(queue)
    want = O.batch(queue, keep, offs, B)
    d_off = D.to_dev(offs)
    d_q = D.to_dev(queue.view(np.int32)) if Q else torch.zeros(1, dtype=torch.int32, device="cuda")
    d_k = None if keep is None else (D.to_dev(keep) if Q else torch.zeros(1, dtype=torch.uint8, device="cuda"))
    oc = torch.full((max(Q, 1),), -1, dtype=torch.int32, device="cuda")
    op = oc.clone()
    oo = oc.clone()
    sc = torch.full((2,), -1, dtype=torch.int64, device="cuda")
    ctx.batch(d_q, d_k, d_off, B, oc, op, oo, sc[0:1], sc[1:2], q_len=Q, out_cap=Q)
    ctx.check("batch")
    m = len(want[0])
    s = sc.cpu().numpy()
    assert s[0] == m and s[1] == len(want[3])
    assert np.array_equal(_u32(oc, m), want[0])
    assert np.array_equal(_u32(op, m), want[1])
    assert np.array_equal(_u32(oo, m), want[2])


@pytest.mark.parametrize("Q", [0, 1, 4095, 4096, 4097, 50_003])
@pytest.mark.parametrize("mask", ["none", "all0", "all1", "alt", "rand"])
def test_batch_matches_oracle(ctx, Q, mask):
    rng = np.random.default_rng(Q + len(mask))
    counts = rng.integers(0, 9, max(Q // 4, 1)).astype(np.int32)
    N = int(counts.sum())
    if N < Q:
        counts[0] += Q - N
        N = Q
    queue = rng.permutation(N)[:Q].astype(np.uint32)
    keep = {"none": None, "all0": np.zeros(Q, np.uint8), "all1": np.ones(Q, np.uint8),
            "alt": (np.arange(Q) % 2).astype(np.uint8),
            "rand": (rng.random(Q) < 0.7).astype(np.uint8)}[mask]
    for B in (1, 63, 64, 65, max(Q, 1)):
        _say("batch", Q, mask, B)
        _batch_case(ctx, counts, queue, keep, B)


def test_batch_unaligned_and_errors(ctx):
    rng = np.random.default_rng(9)
    counts = rng.integers(1, 5, 3000).astype(np.int32)
    N = int(counts.sum())
    queue = rng.permutation(N).astype(np.uint32)
    keep = (rng.random(N) < 0.5).astype(np.uint8)
    offs = O.expand(counts, tags=False)
    want = O.batch(queue[1:], keep[1:], offs, 7)
    # misaligned views (one element in) take the scalar load path
    d_q = D.to_dev(queue.view(np.int32))[1:]
    d_k = D.to_dev(keep)[1:]
    op = torch.empty(N, dtype=torch.int32, device="cuda")
    ctx.batch(d_q, d_k, D.to_dev(offs), 7, None, op, None, q_len=N - 1, out_cap=N)
    ctx.check("batch unaligned")
    assert np.array_equal(_u32(op, len(want[1])), want[1])
    bad = queue.copy()
    bad[5] = N + 3
    ctx.batch(D.to_dev(bad.view(np.int32)), None, D.to_dev(offs), 7, None, op, None, out_cap=N)
    assert ctx.status() == O.ERANGE
    ctx.batch(D.to_dev(queue.view(np.int32)), None, D.to_dev(offs), 7, None, op, None, out_cap=10)
    assert ctx.status() == O.ECAP
    # tag arrays that share memory with an input or with each other are
    # rejected on the host, before anything is enqueued
    from paper_2609_18703_amd.ro import RoError
    d_q = D.to_dev(queue.view(np.int32))
    d_offs = D.to_dev(offs)
    for args in ((None, d_q[N // 2:], None), (op, op, None), (None, op, op[N // 8:]),
                 (None, d_offs.view(torch.int32), None)):
        with pytest.raises(RoError) as e:
            ctx.batch(d_q, None, d_offs, 7, *args, out_cap=N // 4)
        assert e.value.code == O.EINVAL
    assert ctx.status() == O.OK


# ------------------------------------------------------------------ gather
LENS = np.array([0, 1, 15, 16, 17, 63, 64, 65, 4095, 4096], np.int64)


def _gather_case(ctx, counts, par, ordi, st, off, data, extra_lead=0):
    offs = O.expand(counts, tags=False)
    P = len(counts)
    n = len(par)
    want = O.gather(par, ordi, st, off, data, offs, child_dst=True)
    lead = torch.zeros(extra_lead + len(data) + 16, dtype=torch.uint8, device="cuda")
    lead[extra_lead:extra_lead + len(data)] = torch.from_numpy(data).cuda()
    d_data = lead[extra_lead:]
    tot = int(want["out_off"][-1])
    out_base = torch.full((tot + 64,), 0xAB, dtype=torch.uint8, device="cuda")
    shift = (extra_lead * 7) % 16
    out = out_base[shift:shift + max(tot, 1)]
    o_off = torch.empty(P + 1, dtype=torch.int64, device="cuda")
    ns = torch.empty(max(P, 1), dtype=torch.int32, device="cuda")
    nf, nk = ns.clone(), ns.clone()
    comp = torch.empty(max(P, 1), dtype=torch.uint8, device="cuda")
    pst = comp.clone()
    z32 = torch.zeros(1, dtype=torch.int32, device="cuda")
    d_par = D.to_dev(par.view(np.int32)) if n else z32
    d_ord = D.to_dev(ordi.view(np.int32)) if n else z32
    d_st = D.to_dev(st) if n else torch.zeros(1, dtype=torch.uint8, device="cuda")
    cdst = torch.full((int(offs[-1]) + 1,), -5, dtype=torch.int64, device="cuda")
    ctx.gather(d_par, d_ord, d_st, D.to_dev(off), d_data, D.to_dev(offs), o_off, out, ns, nf, nk,
               comp, pst, n=n, out_cap=tot, child_dst_off=cdst)
    ctx.check("gather")
    assert np.array_equal(o_off.cpu().numpy(), want["out_off"])
    assert np.array_equal(cdst.cpu().numpy(), want["child_dst_off"])
    assert np.array_equal(ns.cpu().numpy()[:P], want["n_success"])
    assert np.array_equal(nf.cpu().numpy()[:P], want["n_failed"])
    assert np.array_equal(nk.cpu().numpy()[:P], want["n_skipped"])
    assert np.array_equal(comp.cpu().numpy()[:P], want["complete"])
    assert np.array_equal(pst.cpu().numpy()[:P], want["parent_state"])
    got = out_base.cpu().numpy()
    assert np.array_equal(got[shift:shift + tot], want["out_data"])
    assert np.all(got[:shift] == 0xAB) and np.all(got[shift + tot:] == 0xAB)   # nothing outside


def _make_reports(rng, counts, p_report=1.0, states=(0, 0, 0, 1, 2), lens=LENS):
    par, ordi, st, ln = [], [], [], []
    for p, k in enumerate(counts):
        for o in range(k):
            if rng.random() >= p_report:
                continue
            par.append(p)
            ordi.append(o)
            st.append(rng.choice(states))
            ln.append(int(rng.choice(lens)))
    order = rng.permutation(len(par))
    par = np.array(par, np.uint32)[order]
    ordi = np.array(ordi, np.uint32)[order]
    st = np.array(st, np.uint8)[order]
    ln = np.array(ln, np.int64)[order]
    off = np.concatenate([[0], np.cumsum(ln)]).astype(np.int64)
    data = rng.integers(0, 256, int(off[-1]) + 1, dtype=np.uint8)
    return par, ordi, st, off, data


@pytest.mark.parametrize("case", ["small", "zeros", "multi_tile", "partial", "pending", "big_parent", "empty_runs"])
def test_gather_matches_oracle(ctx, case):
    rng = np.random.default_rng(len(case))
    if case == "empty_runs":
        # runs of thousands of empty parents: some 4,096-child scan tiles span
        # more parents than a tile holds children (their parent search runs
        # in global memory) and more than its LDS count slots
        counts = np.concatenate([rng.integers(1, 40, 300), np.zeros(7000), rng.integers(0, 3, 5000),
                                 np.zeros(12000), [5000], np.zeros(3000), rng.integers(0, 5, 2000),
                                 np.zeros(4500)]).astype(np.int32)
    elif case == "small":
        counts = np.array([3, 1, 4], np.int32)
    elif case == "zeros":
        counts = np.array([0, 2, 0, 0, 5, 0, 1, 0], np.int32)
    elif case == "multi_tile":
        counts = rng.integers(0, 7, 3000).astype(np.int32)
    elif case == "big_parent":
        counts = np.array([3, 9000, 0, 4], np.int32)
    else:
        counts = rng.integers(0, 9, 2000).astype(np.int32)
    p_rep = 0.8 if case == "partial" else 1.0
    states = (0, 0, 1, 2, 3) if case == "pending" else (0, 0, 0, 1, 2)
    lens = LENS if case != "big_parent" else np.array([0, 1, 3, 17, 40], np.int64)
    par, ordi, st, off, data = _make_reports(rng, counts, p_rep, states, lens)
    for lead in (0, 3):
        _say("gather", case, len(par), "lead", lead)
        _gather_case(ctx, counts, par, ordi, st, off, data, extra_lead=lead)


def test_gather_every_alignment(ctx):
    """Every (source, destination) byte alignment mod 16, with records of
    16..80 bytes so each one has interior chunks and two edges."""
    rng = np.random.default_rng(1)
    counts = np.full(64, 8, np.int32)
    for lead in range(16):
        par, ordi, st, off, data = _make_reports(rng, counts, 1.0, (0,),
                                                 np.arange(16, 81, dtype=np.int64))
        _gather_case(ctx, counts, par, ordi, st, off, data, extra_lead=lead)


def test_gather_errors(ctx):
    counts = np.array([2, 1], np.int32)
    offs = D.to_dev(O.expand(counts, tags=False))
    o_off = torch.empty(3, dtype=torch.int64, device="cuda")
    out = torch.empty(64, dtype=torch.uint8, device="cuda")
    data = torch.zeros(64, dtype=torch.uint8, device="cuda")

    def run(par, ordi, st, off, cap=64):
        ctx.gather(D.to_dev(np.array(par, np.int32)), D.to_dev(np.array(ordi, np.int32)),
                   D.to_dev(np.array(st, np.uint8)), D.to_dev(np.array(off, np.int64)), data, offs,
                   o_off, out, out_cap=cap)
        return ctx.status()

    assert run([0, 0], [0, 0], [0, 1], [0, 1, 1]) == O.EDUP
    assert run([2], [0], [0], [0, 1]) == O.ERANGE
    assert run([1], [1], [0], [0, 1]) == O.ERANGE
    assert run([0], [0], [4], [0, 1]) == O.ESTATE
    assert run([0, 0], [0, 1], [0, 0], [0, 3, 2]) == O.EINVAL
    assert run([0, 0, 1], [0, 1, 0], [0, 0, 0], [0, 30, 60, 90], cap=50) == O.ECAP
    assert run([0, 0, 1], [0, 1, 0], [0, 3, 0], [0, 4, 4, 9]) == O.OK
    # a clean call after the errors gives the oracle's answer
    _gather_case(ctx, counts, np.array([1, 0, 0], np.uint32), np.array([0, 1, 0], np.uint32),
                 np.array([0, 0, 1], np.uint8), np.array([0, 3, 5, 9], np.int64),
                 np.arange(10, dtype=np.uint8))


@pytest.mark.parametrize("case", ["short_runs", "empty_runs"])
def test_gather_in_place(ctx, case):
    """Output = the reports' own bytes.  With every surviving record already
    at its output position (reports in canonical order, non-surviving ones
    without bytes) nothing moves and the result is the oracle's; one failed
    report holding bytes shifts every later record, which is RO_EINVAL.  The
    runs of empty parents send some scan tiles to their global-memory parent
    search."""
    rng = np.random.default_rng(21 if case == "short_runs" else 22)
    if case == "short_runs":
        counts = rng.integers(0, 9, 5000).astype(np.int32)
    else:
        counts = np.concatenate([rng.integers(1, 30, 400), np.zeros(9000), rng.integers(0, 4, 3000),
                                 np.zeros(6000), [3000], rng.integers(0, 6, 1000)]).astype(np.int32)
    offs = O.expand(counts, tags=False)
    P, N = len(counts), int(offs[-1])
    par = np.repeat(np.arange(P), counts).astype(np.uint32)
    ordi = np.concatenate([np.arange(k) for k in counts]).astype(np.uint32)
    st = rng.choice(np.array([0, 0, 0, 0, 1, 2], np.uint8), N)
    lens = np.where(st == 0, rng.integers(0, 70, N), 0).astype(np.int64)
    bad = int(np.nonzero(st == 1)[0][N // 10 % max(1, int((st == 1).sum()))])   # a failed report
    for moved in (False, True):
        ln = lens.copy()
        if moved:
            ln[bad] = 5                      # failed, yet holding bytes
        off = np.concatenate([[0], np.cumsum(ln)]).astype(np.int64)
        data = rng.integers(0, 256, int(off[-1]) + 16, dtype=np.uint8)
        want = O.gather(par, ordi, st, off, data, offs)
        d_data = D.to_dev(data)
        o_off = torch.empty(P + 1, dtype=torch.int64, device="cuda")
        ns = torch.empty(P, dtype=torch.int32, device="cuda")
        nf, nk = ns.clone(), ns.clone()
        comp = torch.empty(P, dtype=torch.uint8, device="cuda")
        pst = comp.clone()
        _say("gather in place", case, N, "moved" if moved else "in place")
        ctx.gather(D.to_dev(par.view(np.int32)), D.to_dev(ordi.view(np.int32)), D.to_dev(st), D.to_dev(off),
                   d_data, D.to_dev(offs), o_off, d_data, ns, nf, nk, comp, pst, n=N, out_cap=d_data.numel())
        rc = ctx.status()
        if moved:
            assert rc == O.EINVAL
            continue
        assert rc == O.OK
        tot = int(want["out_off"][-1])
        assert tot == int(off[-1])
        assert np.array_equal(o_off.cpu().numpy(), want["out_off"])
        assert np.array_equal(ns.cpu().numpy(), want["n_success"])
        assert np.array_equal(nf.cpu().numpy(), want["n_failed"])
        assert np.array_equal(nk.cpu().numpy(), want["n_skipped"])
        assert np.array_equal(comp.cpu().numpy(), want["complete"])
        assert np.array_equal(pst.cpu().numpy(), want["parent_state"])
        got = d_data.cpu().numpy()
        assert np.array_equal(got[:tot], want["out_data"]) and np.array_equal(got, data)


def test_gather_repeated_calls_reuse_workspace(ctx):
    """Canonical slots of an earlier call never leak into a later one."""
    rng = np.random.default_rng(4)
    counts = rng.integers(1, 6, 1500).astype(np.int32)
    par, ordi, st, off, data = _make_reports(rng, counts)
    _gather_case(ctx, counts, par, ordi, st, off, data)
    # the same expansion with only some children reported
    keep = rng.random(len(par)) < 0.5
    ln = np.diff(off)[keep]
    off2 = np.concatenate([[0], np.cumsum(ln)]).astype(np.int64)
    data2 = np.concatenate([data[off[i]:off[i + 1]] for i in np.nonzero(keep)[0]] + [np.zeros(1, np.uint8)])
    _gather_case(ctx, counts, par[keep], ordi[keep], st[keep], off2, data2)
