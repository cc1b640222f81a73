"""GPU parity for group-failure containment (barriers in batch, gather and
streaming) against the oracle, including the paper's figure and the
failure-containment analog at full size."""
import json
import os
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

import oracle as O  # noqa: E402
import workloads as W  # noqa: E402
from workloads import device as D  # noqa: E402

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


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


def _i32(a):
    a = np.ascontiguousarray(a, np.uint32)
    return D.to_dev(a.view(np.int32)) if len(a) else torch.zeros(1, dtype=torch.int32, device="cuda")


def _u32(t, n):
    return t.cpu().numpy().view(np.uint32)[:n]


@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_batch_barrier_matches_oracle(ctx, seed):
    rng = np.random.default_rng(seed)
    counts = rng.integers(0, 7, 3000 + 500 * seed).astype(np.int32)
    offs = O.expand(counts, tags=False)
    N = int(offs[-1])
    q = rng.permutation(N).astype(np.uint32)
    keep = None if seed % 2 else (rng.random(N) < 0.8).astype(np.uint8)
    bar = (rng.random(len(counts)) < 0.3).astype(np.uint8)
    want = O.batch(q, keep, offs, 37, barrier=bar)
    oc = torch.full((N,), -1, dtype=torch.int32, device="cuda")
    op, oo = oc.clone(), oc.clone()
    sc = torch.zeros(2, dtype=torch.int64, device="cuda")
    _say("batch barrier", seed, N)
    ctx.batch(_i32(q), None if keep is None else D.to_dev(keep), D.to_dev(offs), 37, oc, op, oo, sc[0:1],
              sc[1:2], q_len=N, out_cap=N, barrier=D.to_dev(bar))
    ctx.check("batch barrier")
    m = len(want[0])
    assert int(sc[0].item()) == m and int(sc[1].item()) == len(want[3])
    assert np.array_equal(_u32(oc, m), want[0])
    assert np.array_equal(_u32(op, m), want[1]) and np.array_equal(_u32(oo, m), want[2])


def _gf_reports(rng, counts, p_gf):
    par, ordi, st, ln = [], [], [], []
    for p, k in enumerate(counts):
        for o in range(k):
            if rng.random() < 0.15:
                continue
            par.append(p)
            ordi.append(o)
            u = rng.random()
            st.append(W.GROUP_FAILED if u < p_gf else (W.FAILED if u < p_gf + 0.05 else
                                                        (W.SKIPPED if u < p_gf + 0.08 else W.SUCCESS)))
            ln.append(int(rng.choice([0, 1, 15, 16, 17, 100, 1000])))
    order = rng.permutation(len(par))
    par = np.array(par, np.uint32)[order]
    ordi = np.array(ordi, np.uint32)[order]
    st = np.array(st, np.uint8)[order]
    ln = np.array(ln, np.int64)[order]
    off = np.concatenate([[0], np.cumsum(ln)]).astype(np.int64)
    data = rng.integers(0, 256, int(off[-1]) + 1, dtype=np.uint8)
    return par, ordi, st, off, data


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_gather_group_failure_matches_oracle(ctx, seed):
    _gf_gather_case(ctx, seed)


def test_gather_across_canonical_epoch_wrap():
    """Six group-failure gathers on one context whose canonical epoch wraps
    after the second (test aid): every slot of an earlier call reads as
    unreported, before and after the wrap."""
    import paper_2609_18703_amd as R
    c = R.Context()
    try:
        c.debug_epochs(canon_left=3)
        for seed in range(6):
            _gf_gather_case(c, seed)
    finally:
        c.close()


def _gf_gather_case(ctx, seed):
    rng = np.random.default_rng(100 + seed)
    counts = rng.integers(0, 9, 4000).astype(np.int32)
    offs = O.expand(counts, tags=False)
    P = len(counts)
    par, ordi, st, off, data = _gf_reports(rng, counts, [0.02, 0.1, 0.3][seed % 3])
    bar_in = (rng.random(P) < 0.1).astype(np.uint8)
    want = O.gather(par, ordi, st, off, data, offs, barrier=bar_in, child_dst=True)
    tot = int(want["out_off"][-1])
    out = torch.zeros(tot + 16, dtype=torch.uint8, device="cuda")
    o_off = torch.empty(P + 1, dtype=torch.int64, device="cuda")
    cnt = torch.empty(3 * P, dtype=torch.int32, device="cuda")
    comp = torch.empty(P, dtype=torch.uint8, device="cuda")
    pst = comp.clone()
    bar = D.to_dev(bar_in)
    nrej = torch.full((1,), -1, dtype=torch.int64, device="cuda")
    cdst = torch.empty(int(offs[-1]) + 1, dtype=torch.int64, device="cuda")
    ctx.reserve(int(offs[-1]), P, len(par))             # not every child reports: reserve the expansion
    _say("gather group failure", seed, len(par), int((st == W.GROUP_FAILED).sum()))
    ctx.gather(_i32(par), _i32(ordi), D.to_dev(st), D.to_dev(off), D.to_dev(data), D.to_dev(offs), o_off, out,
               cnt[:P], cnt[P:2 * P], cnt[2 * P:], comp, pst, n=len(par), out_cap=tot, child_dst_off=cdst,
               barrier=bar, n_rejected=nrej)
    ctx.check("gather group failure")
    assert np.array_equal(o_off.cpu().numpy(), want["out_off"])
    c = cnt.cpu().numpy()
    assert np.array_equal(c[:P], want["n_success"]) and np.array_equal(c[P:2 * P], want["n_failed"])
    assert np.array_equal(c[2 * P:], want["n_skipped"])
    assert np.array_equal(comp.cpu().numpy(), want["complete"])
    assert np.array_equal(pst.cpu().numpy(), want["parent_state"])
    assert np.array_equal(bar.cpu().numpy(), want["barrier"])
    assert int(nrej.item()) == want["n_rejected"]
    assert np.array_equal(cdst.cpu().numpy(), want["child_dst_off"])
    assert np.array_equal(out.cpu().numpy()[:tot], want["out_data"])


def test_gather_group_failure_needs_barrier(ctx):
    offs = O.expand(np.array([2], np.int32), tags=False)
    o_off = torch.empty(2, dtype=torch.int64, device="cuda")
    ctx.gather(_i32([0, 0]), _i32([0, 1]), D.to_dev(np.array([W.GROUP_FAILED, 0], np.uint8)),
               D.to_dev(np.array([0, 0, 0], np.int64)), D.to_dev(np.zeros(1, np.uint8)), D.to_dev(offs), o_off,
               None, n=2, out_cap=0)
    assert ctx.status() == O.ESTATE
    ctx.check("after state error")


def test_stream_group_failure_figure(ctx):
    """Fig. recovery-protocol on the GPU stream: B2 rejected, B3 suppressed."""
    fx = json.load(open(os.path.join(GOLDEN, "failure_group.json")))
    names = {n: i for i, n in enumerate("ABC")}
    codes = {"SUCCESS": W.SUCCESS, "GROUP_FAILED": W.GROUP_FAILED}
    counts = np.array(fx["counts"], np.int32)
    offs = O.expand(counts, tags=False)
    d_offs = D.to_dev(offs)
    bar = torch.zeros(3, dtype=torch.uint8, device="cuda")
    st = ctx.stream(d_offs, int(offs[-1]), bar)
    arena = torch.zeros(16, dtype=torch.uint8, device="cuda")
    nrej = torch.zeros(1, dtype=torch.int64, device="cuda")
    ep = torch.zeros(3, dtype=torch.int32, device="cuda")
    eo = torch.zeros(4, dtype=torch.int64, device="cuda")
    ed = torch.zeros(16, dtype=torch.uint8, device="cuda")
    ec = torch.zeros(9, dtype=torch.int32, device="cuda")
    es = torch.zeros(3, dtype=torch.uint8, device="cuda")
    sc = torch.zeros(4, dtype=torch.int64, device="cuda")
    base = [0]

    def wave(reports):
        n = len(reports)
        vals = [16 * names[r[0]] + r[1] for r in reports]
        arena[base[0]:base[0] + n] = torch.tensor(vals, dtype=torch.uint8, device="cuda")
        off = D.to_dev(np.arange(base[0], base[0] + n + 1, dtype=np.int64))
        base[0] += n
        st.report(_i32([names[r[0]] for r in reports]), _i32([r[1] for r in reports]),
                  D.to_dev(np.array([codes[r[2]] for r in reports], np.uint8)), off, arena, n=n, n_rejected=nrej)
        st.emit(ep, eo, ed, ec[:3], ec[3:6], ec[6:], es, sc[0:1], sc[1:2], cap_parents=3, cap_bytes=16)
        ctx.check("figure wave")
        e = int(sc[0].item())
        return e

    ex = fx["expect"]
    assert wave(fx["wave1"]["reports"]) == 0
    queue = np.array([offs[names[p]] + o for p, o in fx["queue"]], np.uint32)
    oc = torch.zeros(5, dtype=torch.int32, device="cuda")
    ctx.batch(_i32(queue), None, d_offs, fx["reserve"], oc, None, None, sc[2:3], sc[3:4], barrier=bar)
    ctx.check("figure batch")
    assert int(sc[2].item()) == 5                        # nothing barred yet: all five are ready
    e = wave(fx["wave2"]["reports"])
    assert int(nrej.item()) == ex["wave2_rejected"]
    assert ["ABC"[p] for p in _u32(ep, e)] == ex["wave2_emitted"]
    eoff = eo.cpu().numpy()
    for j, p in enumerate(_u32(ep, e)):
        n = "ABC"[p]
        assert int(es[j].item()) == codes.get(ex["states"][n], W.FAILED)
        assert int(ec[j].item()) == ex["n_success"][n] and int(ec[3 + j].item()) == ex["n_failed"][n]
        assert list(ed.cpu().numpy()[eoff[j]:eoff[j + 1]]) == ex["bytes"][n]
    assert list(bar.cpu().numpy()) == [0, 1, 0]
    ctx.batch(_i32(queue[4:]), None, d_offs, fx["reserve"], oc, None, None, sc[2:3], sc[3:4], barrier=bar)
    ctx.check("figure batch after barrier")
    assert int(sc[2].item()) == len(ex["next_reservation"])
    st.close()


@pytest.mark.parametrize("gf_left", [0, 3])
def test_failure_trace_waves(ctx, gf_left):
    """The failure-containment analog at full size (1,885 documents, 45,507
    pages, 99 poisoned), wave by wave against the oracle: the reserved
    children, rejected reports, and every emission.  With gf_left the
    stream's group-failure epoch wraps after its third report (test aid)."""
    from failure_sched import oracle_waves
    t = W.failure_trace()
    offs, waves = oracle_waves(t)
    N, P = t.n_children, t.n_parents
    d_offs = D.to_dev(offs)
    bar = torch.zeros(P, dtype=torch.uint8, device="cuda")
    st = ctx.stream(d_offs, N, bar)
    ctx.debug_epochs(stream=st, gf_left=gf_left)
    total = int(waves[-1]["off"][-1])
    arena = torch.zeros(total + 16, dtype=torch.uint8, device="cuda")
    remaining = _i32(t.queue)
    oc = torch.empty(N, dtype=torch.int32, device="cuda")
    op, oo = oc.clone(), oc.clone()
    sc = torch.zeros(4, dtype=torch.int64, device="cuda")
    nrej = torch.zeros(1, dtype=torch.int64, device="cuda")
    ep = torch.empty(P, dtype=torch.int32, device="cuda")
    eo = torch.empty(P + 1, dtype=torch.int64, device="cuda")
    ed = torch.empty(total + 16, dtype=torch.uint8, device="cuda")
    ec = torch.empty(3 * P, dtype=torch.int32, device="cuda")
    es = torch.empty(P, dtype=torch.uint8, device="cuda")
    _say("failure trace:", len(waves), "waves")
    for w, ow in enumerate(waves):
        Q = len(ow["queue"])
        ctx.batch(remaining, None, d_offs, t.batch_size, oc, op, oo, sc[0:1], sc[1:2], q_len=Q, out_cap=Q,
                  barrier=bar)
        m = int(sc[0].item())
        assert m == len(ow["child"]) and np.array_equal(_u32(oc, m), ow["child"]), w
        d = len(ow["dispatched"])
        assert np.array_equal(_u32(op, d), ow["parent"]) and np.array_equal(_u32(oo, d), ow["ordinal"]), w
        lo, hi = int(ow["off"][0]), int(ow["off"][-1])
        if hi > lo:
            arena[lo:hi] = torch.from_numpy(ow["data"]).cuda()
        nrej.zero_()
        st.report(op, oo, D.to_dev(ow["state"]), D.to_dev(ow["off"]), arena, n=d, n_rejected=nrej)
        st.emit(ep, eo, ed, ec[:P], ec[P:2 * P], ec[2 * P:], es, sc[2:3], sc[3:4], cap_parents=P,
                cap_bytes=total + 16)
        ctx.check(f"trace wave {w}")
        assert int(nrej.item()) == ow["rejected"], w
        em = ow["emitted"]
        E = int(sc[2].item())
        assert E == len(em["parent"]) and int(sc[3].item()) == em["n_bytes"], w
        assert np.array_equal(_u32(ep, E), em["parent"]), w
        assert np.array_equal(eo.cpu().numpy()[:E + 1], em["off"]), w
        assert np.array_equal(ec.cpu().numpy()[:E], em["n_success"]), w
        assert np.array_equal(ec.cpu().numpy()[P:P + E], em["n_failed"]), w
        assert np.array_equal(es.cpu().numpy()[:E], em["parent_state"]), w
        assert np.array_equal(ed.cpu().numpy()[:em["n_bytes"]], em["data"]), w
        nxt = torch.empty(max(m - d, 1), dtype=torch.int32, device="cuda")
        if m > d:
            nxt.copy_(oc[d:m])
        remaining = nxt
        if w % 20 == 0:
            _say("  wave", w, "dispatched", d, "emitted", E)
    st.close()
    assert int(bar.sum().item()) == len(t.poisoned)
