"""ctypes wrapper around the C oracle in ``oracle.c`` plus the plain two-level
composition (test infrastructure only).

The nested pipeline is the composition the paper's multi-grain program
implies (Sec. 2/3: each ``F.expand`` is matched by an ``F.reduce``; Sec. 4,
Reduce rule): the lower gather's parent slots become the upper level's child
reports, keyed by the level-1 children's own (parent, ordinal) lineage and
carrying the lower parent's derived state.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

__all__ = ["build", "lib", "OracleError", "expand", "batch", "gather", "nested", "Stream", "filter", "broadcast",
           "Grains", "WAITING", "READY", "IN_FLIGHT", "SEALED",
           "OK", "EINVAL", "ERANGE", "EDUP", "ECAP", "EOVERFLOW", "ESTATE",
           "SUCCESS", "FAILED", "SKIPPED", "PENDING", "GROUP_FAILED"]

OK, EINVAL, ERANGE, EDUP, ECAP, EOVERFLOW, ESTATE = 0, -1, -2, -3, -4, -5, -6
SUCCESS, FAILED, SKIPPED, PENDING, GROUP_FAILED = 0, 1, 2, 3, 4

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")


class OracleError(RuntimeError):
    def __init__(self, code, what):
        super().__init__(f"{what}: oracle error {code}")
        self.code = code


def build(extra_flags=(), out=None):
    """Compile oracle.c into a shared library (gcc, -O2)."""
    out = out or _LIB
    cmd = ["gcc", "-O2", "-std=c99", "-shared", "-fPIC", *extra_flags, "-o", out, _SRC]
    subprocess.run(cmd, check=True)
    return out


_lib = None


def _load(path):
    L = C.CDLL(path)
    P = C.c_void_p
    i64 = C.c_int64
    L.oracle_expand.argtypes = [P, i64, P, P, P, i64]
    L.oracle_batch.argtypes = [P, P, i64, P, i64, C.c_int32, P, P, P, i64, P, P, P, P]
    L.oracle_batch_parent.argtypes = [P, P, i64, P, i64, C.c_int32, P, P, P, i64, P, P, P, P]
    L.oracle_gather.argtypes = [P, P, P, P, P, i64, P, i64, P, P, i64, P, P, P, P, P, P, P, P]
    L.oracle_stream_create.argtypes = [P, i64]
    L.oracle_stream_create.restype = P
    L.oracle_stream_destroy.argtypes = [P]
    L.oracle_stream_report.argtypes = [P, P, P, P, P, P, i64, P]
    L.oracle_filter.argtypes = [P, P, P, i64, P]
    L.oracle_broadcast.argtypes = [P, C.c_int32, i64, P, i64, P, P, P]
    L.oracle_grains_create.argtypes = [i64]
    L.oracle_grains_create.restype = P
    L.oracle_grains_destroy.argtypes = [P]
    L.oracle_grains_dispatch.argtypes = [P, P, i64, P]
    L.oracle_grains_retry.argtypes = [P, P, i64]
    L.oracle_grains_commit.argtypes = [P, P, P, P, P, P, P, i64, P, i64, P, P]
    L.oracle_grains_phase.argtypes = [P]
    L.oracle_grains_phase.restype = C.POINTER(C.c_uint8)
    L.oracle_grains_gen.argtypes = [P]
    L.oracle_grains_gen.restype = C.POINTER(C.c_uint32)
    for f in ("oracle_grains_dispatch", "oracle_grains_retry", "oracle_grains_commit"):
        getattr(L, f).restype = C.c_int
    L.oracle_stream_barrier.argtypes = [P]
    L.oracle_stream_barrier.restype = C.POINTER(C.c_uint8)
    L.oracle_stream_emit.argtypes = [P, P, P, P, i64, i64, P, P, P, P, P, P]
    for f in ("oracle_expand", "oracle_batch", "oracle_batch_parent", "oracle_gather", "oracle_stream_report",
              "oracle_stream_emit", "oracle_filter", "oracle_broadcast"):
        getattr(L, f).restype = C.c_int
    return L


def lib(path=None):
    """The loaded oracle library (built on first use if missing)."""
    global _lib
    if path is not None:
        return _load(path)
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        _lib = _load(_LIB)
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _check(rc, what):
    if rc != OK:
        raise OracleError(rc, what)


def expand(counts, tags=True, L=None):
    L = L or lib()
    counts = np.ascontiguousarray(counts, dtype=np.int32)
    P = len(counts)
    offsets = np.zeros(P + 1, dtype=np.int64)
    if not tags:
        _check(L.oracle_expand(_p(counts), P, _p(offsets), None, None, 0), "expand")
        return offsets
    # the count total is read back only to size the tag arrays
    n = int(counts.astype(np.int64).sum()) if P else 0
    n = max(n, 0)
    parent = np.zeros(max(n, 1), dtype=np.uint32)
    ordinal = np.zeros(max(n, 1), dtype=np.uint32)
    _check(L.oracle_expand(_p(counts), P, _p(offsets), _p(parent), _p(ordinal), n), "expand")
    return offsets, parent[:n], ordinal[:n]


def batch(queue, keep, offsets, batch_size, barrier=None, L=None, parent_bound=False):
    """FIFO batches: returns (child, parent, ordinal, batch_sizes).  With a
    barrier (uint8 per parent), children of barred parents are dropped.
    Elastic reservations by default; parent_bound=True takes up to B siblings
    of the first ready parent per reservation."""
    L = L or lib()
    queue = np.ascontiguousarray(queue, dtype=np.uint32)
    keep = None if keep is None else np.ascontiguousarray(keep, dtype=np.uint8)
    offsets = np.ascontiguousarray(offsets, dtype=np.int64)
    Q = len(queue)
    cap = max(Q, 1)
    child = np.zeros(cap, np.uint32)
    parent = np.zeros(cap, np.uint32)
    ordinal = np.zeros(cap, np.uint32)
    sizes = np.zeros(cap, np.int64)
    n_out = np.zeros(1, np.int64)
    n_b = np.zeros(1, np.int64)
    barrier = None if barrier is None else np.ascontiguousarray(barrier, dtype=np.uint8)
    fn = L.oracle_batch_parent if parent_bound else L.oracle_batch
    _check(fn(_p(queue), _p(keep), Q, _p(offsets), len(offsets) - 1, int(batch_size),
              _p(child), _p(parent), _p(ordinal), Q, _p(n_out), _p(n_b), _p(sizes), _p(barrier)),
           "batch")
    m, nb = int(n_out[0]), int(n_b[0])
    return child[:m], parent[:m], ordinal[:m], sizes[:nb]


def gather(parent, ordinal, state, off, data, offsets, with_data=True, child_dst=False, barrier=None,
           L=None):
    """Ordered gather; returns a dict of per-parent outputs (and, with
    child_dst, every child's output start position, N+1 entries).  With a
    barrier (uint8 per parent, the Call's group-failure state before this
    call) the result also holds the updated barrier and the number of
    rejected reports."""
    L = L or lib()
    parent = np.ascontiguousarray(parent, dtype=np.uint32)
    ordinal = np.ascontiguousarray(ordinal, dtype=np.uint32)
    state = np.ascontiguousarray(state, dtype=np.uint8)
    off = np.ascontiguousarray(off, dtype=np.int64)
    offsets = np.ascontiguousarray(offsets, dtype=np.int64)
    n = len(parent)
    P = len(offsets) - 1
    data = None if data is None else np.ascontiguousarray(data, dtype=np.uint8)
    cap = int(off[-1] - off[0]) if n else 0
    out_data = np.zeros(max(cap, 1), np.uint8) if with_data else None
    out_off = np.zeros(P + 1, np.int64)
    ns = np.zeros(max(P, 1), np.int32)
    nf = np.zeros(max(P, 1), np.int32)
    nk = np.zeros(max(P, 1), np.int32)
    comp = np.zeros(max(P, 1), np.uint8)
    pst = np.zeros(max(P, 1), np.uint8)
    cdst = np.zeros(int(offsets[-1]) + 1, np.int64) if child_dst else None
    bar = None if barrier is None else np.array(barrier, dtype=np.uint8, copy=True)
    nrej = np.zeros(1, np.int64)
    _check(L.oracle_gather(_p(parent), _p(ordinal), _p(state), _p(off),
                           _p(data) if with_data else None, n, _p(offsets), P,
                           _p(out_off), _p(out_data), cap, _p(ns), _p(nf), _p(nk),
                           _p(comp), _p(pst), _p(cdst) if child_dst else None, _p(bar), _p(nrej)),
           "gather")
    res = dict(out_off=out_off, n_success=ns[:P], n_failed=nf[:P], n_skipped=nk[:P],
               complete=comp[:P], parent_state=pst[:P])
    if child_dst:
        res["child_dst_off"] = cdst
    if barrier is not None:
        res["barrier"] = bar
        res["n_rejected"] = int(nrej[0])
    if with_data:
        res["out_data"] = out_data[:int(out_off[-1])]
    return res


def nested(counts1, queue1, keep1, batch1, counts2, queue2, keep2, batch2,
           region_state, region_off, region_data, L=None, with_data=True):
    """Two-level composition: expand(top->mid), batch(mid), expand(mid->leaf),
    batch(leaf), gather(leaf->mid), gather(mid->top).

    ``region_state``/``region_off``/``region_data`` are the leaf reports in
    leaf dispatch order (the order of the leaf batches); their tags come from
    the leaf batch.  The mid-level reports are the mid slots in canonical mid
    order, tagged with the mid children's own lineage keys.
    """
    L = L or lib()
    off1, par1, ord1 = expand(counts1, L=L)
    b1 = batch(queue1, keep1, off1, batch1, L=L)
    off2, par2, ord2 = expand(counts2, L=L)
    b2 = batch(queue2, keep2, off2, batch2, L=L)
    low = gather(b2[1], b2[2], region_state, region_off, region_data, off2,
                 with_data=with_data, L=L)
    up = gather(par1, ord1, low["parent_state"], low["out_off"],
                low.get("out_data"), off1, with_data=with_data, L=L)
    return dict(offsets1=off1, parent1=par1, ordinal1=ord1, batch1=b1,
                offsets2=off2, parent2=par2, ordinal2=ord2, batch2=b2,
                low=low, up=up)


def filter(x_state, mask, mask_state=None, L=None):
    """F.filter: output state per item (SKIPPED where a present mask is false)."""
    L = L or lib()
    x_state = np.ascontiguousarray(x_state, dtype=np.uint8)
    mask = np.ascontiguousarray(mask, dtype=np.uint8)
    ms = None if mask_state is None else np.ascontiguousarray(mask_state, dtype=np.uint8)
    out = np.zeros(max(len(x_state), 1), np.uint8)
    _check(L.oracle_filter(_p(x_state), _p(ms), _p(mask), len(x_state), _p(out)), "filter")
    return out[:len(x_state)]


def broadcast(maps, x_state, like_state=None, L=None):
    """F.broadcast: (ancestor index, output state) per descendant; maps[0]
    is the descendant level's child->parent array, maps[1] the next, ..."""
    L = L or lib()
    maps = [np.ascontiguousarray(m, dtype=np.uint32) for m in maps]
    n = len(maps[0])
    x_state = np.ascontiguousarray(x_state, dtype=np.uint8)
    ls = None if like_state is None else np.ascontiguousarray(like_state, dtype=np.uint8)
    arr = (C.c_void_p * len(maps))(*[m.ctypes.data for m in maps])
    anc = np.zeros(max(n, 1), np.uint32)
    out = np.zeros(max(n, 1), np.uint8)
    _check(L.oracle_broadcast(C.cast(arr, C.c_void_p), len(maps), n, _p(x_state), len(x_state), _p(ls),
                              _p(anc), _p(out)), "broadcast")
    return anc[:n], out[:n]


WAITING, READY, IN_FLIGHT, SEALED = 0, 1, 2, 3


class Grains:
    """Grain phases and generations of one Call's children (oracle side)."""

    def __init__(self, n, L=None):
        self.L = L or lib()
        self.n = int(n)
        self.h = self.L.oracle_grains_create(self.n)
        if not self.h:
            raise OracleError(EINVAL, "grains_create")

    def dispatch(self, child):
        child = np.ascontiguousarray(child, dtype=np.uint32)
        gen = np.zeros(max(len(child), 1), np.uint32)
        _check(self.L.oracle_grains_dispatch(self.h, _p(child), len(child), _p(gen)), "grains_dispatch")
        return gen[:len(child)]

    def retry(self, child):
        child = np.ascontiguousarray(child, dtype=np.uint32)
        _check(self.L.oracle_grains_retry(self.h, _p(child), len(child)), "grains_retry")

    def commit(self, parent, ordinal, state, off, data, gen, offsets):
        """Returns (state_out, (accepted, stale, duplicate, conflict))."""
        parent = np.ascontiguousarray(parent, dtype=np.uint32)
        ordinal = np.ascontiguousarray(ordinal, dtype=np.uint32)
        state = np.ascontiguousarray(state, dtype=np.uint8)
        off = np.ascontiguousarray(off, dtype=np.int64)
        data = None if data is None else np.ascontiguousarray(data, dtype=np.uint8)
        gen = np.ascontiguousarray(gen, dtype=np.uint32)
        offsets = np.ascontiguousarray(offsets, dtype=np.int64)
        out = np.zeros(max(len(parent), 1), np.uint8)
        counts = np.zeros(4, np.int64)
        _check(self.L.oracle_grains_commit(self.h, _p(parent), _p(ordinal), _p(state), _p(off), _p(data), _p(gen),
                                           len(parent), _p(offsets), len(offsets) - 1, _p(out), _p(counts)),
               "grains_commit")
        return out[:len(parent)], tuple(int(x) for x in counts)

    def phase(self):
        return np.ctypeslib.as_array(self.L.oracle_grains_phase(self.h), shape=(max(self.n, 1),))[:self.n].copy()

    def gen(self):
        return np.ctypeslib.as_array(self.L.oracle_grains_gen(self.h), shape=(max(self.n, 1),))[:self.n].copy()

    def close(self):
        if self.h:
            self.L.oracle_grains_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Stream:
    """Streaming gather over one expansion (oracle side)."""

    def __init__(self, offsets, L=None):
        self.L = L or lib()
        self.offsets = np.ascontiguousarray(offsets, dtype=np.int64)
        self.h = self.L.oracle_stream_create(_p(self.offsets), len(self.offsets) - 1)
        if not self.h:
            raise OracleError(EINVAL, "stream_create")
        self._keep = []          # byte buffers must outlive their parents' emission

    def report(self, parent, ordinal, state, off, data):
        parent = np.ascontiguousarray(parent, dtype=np.uint32)
        ordinal = np.ascontiguousarray(ordinal, dtype=np.uint32)
        state = np.ascontiguousarray(state, dtype=np.uint8)
        off = np.ascontiguousarray(off, dtype=np.int64)
        data = None if data is None else np.ascontiguousarray(data, dtype=np.uint8)
        self._keep.append((parent, ordinal, state, off, data))
        nrej = np.zeros(1, np.int64)
        _check(self.L.oracle_stream_report(self.h, _p(parent), _p(ordinal), _p(state), _p(off),
                                           _p(data), len(parent), _p(nrej)), "stream_report")
        return int(nrej[0])

    def barrier(self):
        """Copy of the stream's group-failure barrier (uint8 per parent)."""
        P = len(self.offsets) - 1
        ptr = self.L.oracle_stream_barrier(self.h)
        return np.ctypeslib.as_array(ptr, shape=(max(P, 1),))[:P].copy()

    def emit(self, cap_parents=None, cap_bytes=None, with_data=True):
        P = len(self.offsets) - 1
        cap_parents = P if cap_parents is None else cap_parents
        if cap_bytes is None:
            cap_bytes = sum(int(k[3][-1] - k[3][0]) for k in self._keep)
        ep = np.zeros(max(cap_parents, 1), np.uint32)
        eo = np.zeros(cap_parents + 1, np.int64)
        ed = np.zeros(max(cap_bytes, 1), np.uint8) if with_data else None
        ns = np.zeros(max(cap_parents, 1), np.int32)
        nf = np.zeros(max(cap_parents, 1), np.int32)
        nk = np.zeros(max(cap_parents, 1), np.int32)
        st = np.zeros(max(cap_parents, 1), np.uint8)
        ne = np.zeros(1, np.int64)
        nb = np.zeros(1, np.int64)
        _check(self.L.oracle_stream_emit(self.h, _p(ep), _p(eo), _p(ed), cap_parents, cap_bytes,
                                         _p(ns), _p(nf), _p(nk), _p(st), _p(ne), _p(nb)),
               "stream_emit")
        e, b = int(ne[0]), int(nb[0])
        res = dict(parent=ep[:e], off=eo[:e + 1], n_success=ns[:e], n_failed=nf[:e],
                   n_skipped=nk[:e], parent_state=st[:e], n_bytes=b)
        if with_data:
            res["data"] = ed[:b].copy()
        return res

    def close(self):
        if self.h:
            self.L.oracle_stream_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
