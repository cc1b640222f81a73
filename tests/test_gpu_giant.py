"""Records longer than 2^31 bytes and slots and outputs past 2^32 bytes: the
gather and the streaming emission against the oracle.  Integer outputs are
compared with the oracle in full; the payload (4.9 GiB) is compared on the
device with the records written again by the generator's fill at the
oracle's slot positions.  Also the library's record-length limit: a record
of 2^32 bytes or more is RO_EOVERFLOW."""
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

import oracle as O  # noqa: E402
import workloads as W  # noqa: E402
from workloads import device as D  # noqa: E402

GiB = 1 << 30
S, F, K = W.SUCCESS, W.FAILED, W.SKIPPED

# Six parents, nine children in canonical order: (state, record length).
COUNTS = np.array([2, 1, 3, 0, 2, 1], np.int32)
SPEC = [(S, 5), (S, 3 * GiB + 7),                      # parent 0: a slot past 2^31 bytes
        (S, 1),                                        # parent 1 starts past 3 GiB
        (S, GiB + GiB // 4 + 3), (K, 0), (S, 13),      # parent 2 ends past 2^32
        (F, 11), (S, (600 << 20) + 1),                 # parent 4: a failed member
        (S, 17)]


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


def _reports(lead=3, seed=5):
    """Reports of every child in a random order, records laid out in report
    order after `lead` bytes; record r is splitmix64 of its (parent, ordinal)."""
    offs = np.concatenate([[0], np.cumsum(COUNTS, dtype=np.int64)])
    parent = np.repeat(np.arange(len(COUNTS), dtype=np.uint32), COUNTS)
    ordinal = (np.arange(len(SPEC)) - offs[parent]).astype(np.uint32)
    state = np.array([s for s, _ in SPEC], np.uint8)
    length = np.array([n for _, n in SPEC], np.int64)
    order = np.random.default_rng(seed).permutation(len(SPEC))
    off = np.concatenate([[lead], lead + np.cumsum(length[order])]).astype(np.int64)
    return offs, parent, ordinal, state, length, order, off


def _expected_dev(parent, ordinal, state, length):
    """The packed slots by definition: SUCCESS records in canonical order."""
    keep = np.flatnonzero(state == S)
    pos = np.concatenate([[0], np.cumsum(length[keep])]).astype(np.int64)
    out = torch.empty(int(pos[-1]), dtype=torch.uint8, device="cuda")
    D.fill_records_dev(D.to_dev(W.content_seed(parent[keep], ordinal[keep])), D.to_dev(pos), out)
    return out


def test_giant_records_gather_and_stream(ctx):
    offs, parent, ordinal, state, length, order, off = _reports()
    P, N = len(COUNTS), len(SPEC)
    data = torch.zeros(int(off[-1]) + 16, dtype=torch.uint8, device="cuda")
    D.fill_records_dev(D.to_dev(W.content_seed(parent[order], ordinal[order])), D.to_dev(off), data)
    d_par, d_ord = D.to_dev(parent[order].view(np.int32)), D.to_dev(ordinal[order].view(np.int32))
    d_st, d_off, d_offs = D.to_dev(state[order]), D.to_dev(off), D.to_dev(offs)

    want = O.gather(parent[order], ordinal[order], state[order], off, None, offs, with_data=False,
                    child_dst=True)
    exp = _expected_dev(parent, ordinal, state, length)
    tot = exp.numel()
    assert tot == int(want["out_off"][-1]) and tot > (1 << 32)

    _say("giant gather: total", tot)
    shift = 5                                   # a misaligned output base, sentinels around it
    base = torch.full((tot + 64,), 0xAB, dtype=torch.uint8, device="cuda")
    out = base[shift:shift + tot + 16]
    o_off = torch.empty(P + 1, dtype=torch.int64, device="cuda")
    cnt = torch.zeros(3 * P, dtype=torch.int32, device="cuda")
    comp = torch.zeros(P, dtype=torch.uint8, device="cuda")
    pst = torch.zeros(P, dtype=torch.uint8, device="cuda")
    cdst = torch.empty(N + 1, dtype=torch.int64, device="cuda")
    ctx.gather(d_par, d_ord, d_st, d_off, data, d_offs, o_off, out, cnt[:P], cnt[P:2 * P], cnt[2 * P:], comp,
               pst, child_dst_off=cdst, out_cap=tot)
    ctx.check("giant gather")
    assert np.array_equal(o_off.cpu().numpy(), want["out_off"])
    assert np.array_equal(cdst.cpu().numpy(), want["child_dst_off"])
    c = cnt.cpu().numpy()
    assert np.array_equal(c[:P], want["n_success"]) and np.array_equal(c[P:2 * P], want["n_failed"])
    assert np.array_equal(c[2 * P:], want["n_skipped"])
    assert np.array_equal(comp.cpu().numpy(), want["complete"])
    assert np.array_equal(pst.cpu().numpy(), want["parent_state"])
    assert torch.equal(out[:tot], exp)
    assert bool((base[:shift] == 0xAB).all()) and bool((base[shift + tot:] == 0xAB).all())
    del base, out

    _say("giant stream: one wave")
    ost = O.Stream(offs)
    ost.report(parent[order], ordinal[order], state[order], off, None)
    w = ost.emit(with_data=False)
    st = ctx.stream(d_offs, N)
    st.report(d_par, d_ord, d_st, d_off, data)
    ep = torch.empty(P, dtype=torch.int32, device="cuda")
    eo = torch.empty(P + 1, dtype=torch.int64, device="cuda")
    ed = torch.full((tot + 16,), 0xAB, dtype=torch.uint8, device="cuda")
    ec = torch.zeros(3 * P, dtype=torch.int32, device="cuda")
    es = torch.zeros(P, dtype=torch.uint8, device="cuda")
    sc = torch.zeros(2, dtype=torch.int64, device="cuda")
    st.emit(ep, eo, ed, ec[:P], ec[P:2 * P], ec[2 * P:], es, sc[0:1], sc[1:2])
    ctx.check("giant emit")
    e = int(sc[0].item())
    assert e == len(w["parent"]) == P and int(sc[1].item()) == w["n_bytes"] == tot
    assert np.array_equal(ep.cpu().numpy().view(np.uint32)[:e], w["parent"])
    assert np.array_equal(eo.cpu().numpy()[:e + 1], w["off"])
    c = ec.cpu().numpy()
    assert np.array_equal(c[:e], w["n_success"]) and np.array_equal(c[P:P + e], w["n_failed"])
    assert np.array_equal(c[2 * P:2 * P + e], w["n_skipped"])
    assert np.array_equal(es.cpu().numpy()[:e], w["parent_state"])
    assert torch.equal(ed[:tot], exp) and bool((ed[tot:] == 0xAB).all())
    st.close()


def test_record_of_2_32_bytes_is_overflow(ctx):
    """A slot stores a record's length in 32 bits, so a SUCCESS record of 2^32
    bytes or more is refused with RO_EOVERFLOW by the gather and by a stream
    report (a documented limit of the library; the paper sets none, so there
    is no oracle side).  The record is allocated in full: even a kernel that
    read it would stay in bounds."""
    counts = np.array([1, 1], np.int32)
    offs = np.array([0, 1, 2], np.int64)
    par = D.to_dev(np.array([1, 0], np.int32))
    ordi = D.to_dev(np.zeros(2, np.int32))
    st = D.to_dev(np.array([S, S], np.uint8))
    off = D.to_dev(np.array([0, 7, 7 + (1 << 32)], np.int64))
    _say("overflow: record of", 1 << 32, "bytes")
    data = torch.zeros(7 + (1 << 32) + 16, dtype=torch.uint8, device="cuda")
    o_off = torch.empty(len(counts) + 1, dtype=torch.int64, device="cuda")
    out = torch.empty(64, dtype=torch.uint8, device="cuda")
    ctx.gather(par, ordi, st, off, data, D.to_dev(offs), o_off, out)
    assert ctx.status() == O.EOVERFLOW
    s = ctx.stream(D.to_dev(offs), 2)
    s.report(par, ordi, st, off, data)
    assert ctx.status() == O.EOVERFLOW
    s.close()
    ctx.check("after overflow")
