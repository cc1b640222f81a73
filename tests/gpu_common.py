"""Helpers shared by the GPU tests: staging workloads and reading results."""
import numpy as np
import torch

import oracle as O
import workloads as W
from workloads import device as D
from paper_2609_18703_amd import pipeline as PL


def u32(t):
    return t.cpu().numpy().view(np.uint32)


def np_of(t, n=None):
    a = t.cpu().numpy()
    return a if n is None else a[:n]


def stage_single(c, want_data=True):
    """Device buffers for a SingleLevel workload."""
    r = c.reports
    data = D.reports_data_dev(r) if want_data else torch.zeros(1, dtype=torch.uint8, device="cuda")
    b = PL.SingleLevelBuffers(
        D.to_dev(c.counts), D.to_dev(c.queue.view(np.int32)), D.to_dev(c.keep), D.to_dev(c.sealed_ids.view(np.int32)),
        D.to_dev(r.state), D.to_dev(r.off), data, c.n_children, c.n_dispatched, c.batch_size,
        want_data=want_data)
    return b


def oracle_single(c, data=None, with_data=True):
    """Oracle chain for a SingleLevel workload: the same four steps."""
    r = c.reports
    offs, cp, co = O.expand(c.counts)
    b1 = O.batch(c.queue, c.keep, offs, c.batch_size)
    b2 = O.batch(c.sealed_ids, None, offs, c.batch_size)
    par = np.concatenate([b1[1], b2[1]])
    ordi = np.concatenate([b1[2], b2[2]])
    if with_data and data is None:
        data = r.data()
    g = O.gather(par, ordi, r.state, r.off, data, offs, with_data=with_data)
    return dict(offsets=offs, child_parent=cp, child_ordinal=co, b1=b1, b2=b2, rep_parent=par,
                rep_ordinal=ordi, g=g)


def compare_single(b, want, with_data=True):
    N, M = b.N, b.M
    P = b.counts.numel()
    assert np.array_equal(np_of(b.offsets, P + 1), want["offsets"])
    assert np.array_equal(u32(b.child_parent)[:N], want["child_parent"])
    assert np.array_equal(u32(b.child_ordinal)[:N], want["child_ordinal"])
    assert np.array_equal(u32(b.rep_parent)[:N], want["rep_parent"])
    assert np.array_equal(u32(b.rep_ordinal)[:N], want["rep_ordinal"])
    sc = np_of(b.scalars)
    assert sc[0] == len(want["b1"][0]) and sc[1] == len(want["b1"][3])
    if N > M:
        assert sc[2] == len(want["b2"][0]) and sc[3] == len(want["b2"][3])
    g = want["g"]
    assert np.array_equal(np_of(b.out_off, P + 1), g["out_off"])
    assert np.array_equal(np_of(b.n_success, P), g["n_success"])
    assert np.array_equal(np_of(b.n_failed, P), g["n_failed"])
    assert np.array_equal(np_of(b.n_skipped, P), g["n_skipped"])
    assert np.array_equal(np_of(b.complete, P), g["complete"])
    assert np.array_equal(np_of(b.parent_state, P), g["parent_state"])
    if with_data:
        tot = int(g["out_off"][-1])
        assert np.array_equal(np_of(b.out_data, tot), g["out_data"])
