"""Python binding of the ``ro`` C ABI (argument marshalling only).

Every array argument is a torch tensor on the GPU; the binding passes its
data pointer and size to ``libro.so`` and the torch current stream to the
context.  Nothing here computes any step of the path.  If the library is
missing, loading fails loudly: there is no fallback.
"""
from __future__ import annotations

import ctypes as C
import os
import weakref

__all__ = ["RoError", "load", "Context", "Stream", "Grains", "expand_noalloc", "EXPAND_NOALLOC_MAX_PARENTS",
           "KERNELS", "OK", "EINVAL", "ERANGE", "EDUP", "ECAP",
           "EOVERFLOW", "ESTATE", "EHIP", "SUCCESS", "FAILED", "SKIPPED", "PENDING", "GROUP_FAILED",
           "LIB_PATH"]

OK, EINVAL, ERANGE, EDUP, ECAP, EOVERFLOW, ESTATE, EHIP = 0, -1, -2, -3, -4, -5, -6, -7
SUCCESS, FAILED, SKIPPED, PENDING, GROUP_FAILED = 0, 1, 2, 3, 4

# kernel kinds reported by Context.trace_read, in the C enum's order
KERNELS = ["expand_scan", "expand_tags", "batch_samples", "batch", "gather_scatter", "gather_scan",
           "gather_finalize", "gather_copy", "gather_reset", "stream_report", "stream_select",
           "stream_scan", "stream_copy", "stream_finish", "misc", "filter", "broadcast", "grains",
           "fence_first", "fence_decide", "pbatch_sort", "pbatch"]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libro.so")


class RoError(RuntimeError):
    def __init__(self, code, what):
        super().__init__(f"{what}: ro error {code}")
        self.code = code


class ReportsT(C.Structure):
    _fields_ = [("parent", C.c_void_p), ("ordinal", C.c_void_p), ("state", C.c_void_p),
                ("off", C.c_void_p), ("data", C.c_void_p), ("n", C.c_int64)]


class GatherOutT(C.Structure):
    _fields_ = [("out_off", C.c_void_p), ("out_data", C.c_void_p), ("out_cap", C.c_int64),
                ("n_success", C.c_void_p), ("n_failed", C.c_void_p), ("n_skipped", C.c_void_p),
                ("complete", C.c_void_p), ("parent_state", C.c_void_p), ("child_dst_off", C.c_void_p),
                ("barrier", C.c_void_p), ("n_rejected", C.c_void_p)]


_lib = None


def load(path=None):
    """Load libro.so (raises if it has not been built)."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    path = path or LIB_PATH
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with paper_2609_18703_amd/build.py")
    L = C.CDLL(path)
    P, i64, i32 = C.c_void_p, C.c_int64, C.c_int32
    pp = C.POINTER(C.c_void_p)
    L.ro_ctx_create.argtypes = [pp, P]
    L.ro_ctx_set_stream.argtypes = [P, P]
    L.ro_ctx_reserve.argtypes = [P, i64, i64, i64]
    L.ro_ctx_status.argtypes = [P]
    L.ro_ctx_destroy.argtypes = [P]
    L.ro_expand.argtypes = [P, P, i64, P, P, P, i64]
    L.ro_expand_noalloc.argtypes = [P, P, i64, P, P, P, i64, P]
    L.ro_batch.argtypes = [P, P, P, i64, P, i64, i32, P, P, P, i64, P, P, P]
    L.ro_batch_parent.argtypes = [P, P, P, i64, P, i64, i32, P, P, P, i64, P, i64, P, P, P]
    L.ro_gather.argtypes = [P, C.POINTER(ReportsT), P, i64, C.POINTER(GatherOutT)]
    L.ro_stream_create.argtypes = [P, P, i64, i64, P, pp]
    L.ro_stream_batch.argtypes = [P, P, P, P, i64, i32, P, P, P, i64, P, P]
    L.ro_debug_epochs.argtypes = [P, P, P, i64, i64, i64, i64]
    L.ro_stream_report.argtypes = [P, P, C.POINTER(ReportsT), P]
    L.ro_stream_emit.argtypes = [P, P, P, P, P, i64, i64, P, P, P, P, P, P]
    L.ro_stream_reset.argtypes = [P, P]
    L.ro_filter.argtypes = [P, P, P, P, i64, P]
    L.ro_grains_create.argtypes = [P, i64, pp]
    L.ro_grains_reset.argtypes = [P, P]
    L.ro_grains_destroy.argtypes = [P]
    L.ro_grains_read.argtypes = [P, P, P, P]
    L.ro_grains_dispatch.argtypes = [P, P, P, i64, P]
    L.ro_grains_retry.argtypes = [P, P, P, i64]
    L.ro_grains_commit.argtypes = [P, P, C.POINTER(ReportsT), P, P, i64, P, P]
    L.ro_broadcast.argtypes = [P, P, P, i32, i64, P, i64, P, P, P]
    L.ro_stream_destroy.argtypes = [P]
    L.ro_ctx_trace.argtypes = [P, C.c_int]
    L.ro_ctx_trace_read.argtypes = [P, P, P, i32]
    for name in ("ro_ctx_trace", "ro_ctx_trace_read", "ro_ctx_create", "ro_ctx_set_stream", "ro_ctx_reserve",
                 "ro_ctx_status", "ro_ctx_destroy", "ro_expand", "ro_expand_noalloc", "ro_batch", "ro_batch_parent", "ro_gather",
                 "ro_stream_create", "ro_stream_batch", "ro_stream_report", "ro_stream_emit", "ro_stream_reset", "ro_stream_destroy", "ro_filter",
                 "ro_broadcast", "ro_grains_create", "ro_grains_reset", "ro_grains_destroy", "ro_grains_read",
                 "ro_grains_dispatch", "ro_grains_retry", "ro_grains_commit", "ro_debug_epochs"):
        getattr(L, name).restype = C.c_int
    if path == LIB_PATH:
        _lib = L
    return L


def _ptr(t, item=None, n=0, name="array"):
    """Device pointer of tensor t (None passes through).  The C side sees only
    the pointer, so the element size (`item` bytes) and the length (at least
    `n` elements) the call will use are checked here."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"ro {name} must live in GPU memory")
    if not t.is_contiguous():
        raise ValueError(f"ro {name} must be contiguous")
    if item is not None and t.element_size() != item:
        raise TypeError(f"ro {name} needs {item}-byte elements, got {t.dtype}")
    if t.numel() < n:
        raise ValueError(f"ro {name} needs at least {n} elements, has {t.numel()}")
    return C.c_void_p(t.data_ptr())


def _check(rc, what):
    if rc != OK:
        raise RoError(rc, what)


# the largest expansion ro_expand_noalloc takes (its fixed device workspace)
EXPAND_NOALLOC_MAX_PARENTS = 1 << 24


def expand_noalloc(counts, offsets, child_parent=None, child_ordinal=None, status=None, n_parents=None):
    """ro_expand_noalloc on torch's current stream: ro_expand without a
    context and without any device allocation.  ``status`` (optional, one
    int32 on the GPU) receives the device-detected status of the call."""
    import torch
    L = load()
    cap = 0
    if child_parent is not None or child_ordinal is not None:
        cap = min(t.numel() for t in (child_parent, child_ordinal) if t is not None)
    P = counts.numel() if n_parents is None else int(n_parents)
    stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    _check(L.ro_expand_noalloc(stream, _ptr(counts, 4, P, "counts"), P, _ptr(offsets, 8, P + 1, "offsets"),
                               _ptr(child_parent, 4, 0, "child_parent"), _ptr(child_ordinal, 4, 0, "child_ordinal"),
                               cap, _ptr(status, 4, 1, "status")), "ro_expand_noalloc")


def _reports(parent, ordinal, state, off, data, n=None):
    n = parent.numel() if n is None else int(n)
    return ReportsT(_ptr(parent, 4, n, "report parents"), _ptr(ordinal, 4, n, "report ordinals"),
                    _ptr(state, 1, n, "report states"), _ptr(off, 8, n + 1, "report offsets"),
                    _ptr(data, 1, 0, "report bytes"), n)


def _queue_args(queue, keep, q_len):
    q_len = int(q_len)
    return _ptr(queue, 4, q_len, "queue"), _ptr(keep, 1, q_len, "keep"), q_len


def _tag_args(out_child, out_parent, out_ordinal, out_cap):
    out_cap = int(out_cap)
    return (_ptr(out_child, 4, out_cap, "out_child"), _ptr(out_parent, 4, out_cap, "out_parent"),
            _ptr(out_ordinal, 4, out_cap, "out_ordinal"), out_cap)


class Context:
    """An ro context bound to a HIP stream (torch's current stream by default)."""

    def __init__(self, stream=None):
        import torch
        self.L = load()
        if stream is None:
            stream = torch.cuda.current_stream()
        self._stream = stream
        h = C.c_void_p()
        _check(self.L.ro_ctx_create(C.byref(h), C.c_void_p(stream.cuda_stream)), "ro_ctx_create")
        self.h = h
        self._owned = weakref.WeakSet()     # grain sets and streams: destroyed before the context

    def reserve(self, max_children, max_parents, max_queue=0):
        _check(self.L.ro_ctx_reserve(self.h, int(max_children), int(max_parents), int(max_queue)),
               "ro_ctx_reserve")

    def status(self):
        return self.L.ro_ctx_status(self.h)

    def check(self, what="device"):
        _check(self.status(), what)

    def debug_epochs(self, stream=None, grains=None, canon_left=0, run_left=0, gf_left=0, fence_left=0):
        """Test aid: bring epoch wrap-arounds within a few calls (ro_debug_epochs)."""
        _check(self.L.ro_debug_epochs(self.h, stream.h if stream is not None else None,
                                      grains.h if grains is not None else None, int(canon_left), int(run_left),
                                      int(gf_left), int(fence_left)), "ro_debug_epochs")

    def set_stream(self, stream):
        """Re-bind the context to another torch stream (waits for the old one)."""
        _check(self.L.ro_ctx_set_stream(self.h, C.c_void_p(stream.cuda_stream)), "ro_ctx_set_stream")
        self._stream = stream

    def trace(self, enable=True):
        """Bracket every kernel this context launches with HIP events."""
        _check(self.L.ro_ctx_trace(self.h, 1 if enable else 0), "ro_ctx_trace")

    def trace_read(self):
        """{kernel: (launches, total_ms)} since the last read (waits for the stream)."""
        n = len(KERNELS)
        launches = (C.c_int64 * n)()
        ms = (C.c_double * n)()
        _check(self.L.ro_ctx_trace_read(self.h, C.cast(launches, C.c_void_p), C.cast(ms, C.c_void_p), n),
               "ro_ctx_trace_read")
        return {k: (int(launches[i]), float(ms[i])) for i, k in enumerate(KERNELS) if launches[i]}

    def expand(self, counts, offsets, child_parent=None, child_ordinal=None):
        cap = 0
        if child_parent is not None or child_ordinal is not None:
            cap = min(t.numel() for t in (child_parent, child_ordinal) if t is not None)
        P = counts.numel()
        _check(self.L.ro_expand(self.h, _ptr(counts, 4, P, "counts"), P, _ptr(offsets, 8, P + 1, "offsets"),
                                _ptr(child_parent, 4, 0, "child_parent"), _ptr(child_ordinal, 4, 0, "child_ordinal"),
                                cap), "ro_expand")

    def batch(self, queue, keep, offsets, batch_size, out_child=None, out_parent=None,
              out_ordinal=None, n_out=None, n_batches=None, q_len=None, out_cap=None, barrier=None):
        q_len = queue.numel() if q_len is None else q_len
        if out_cap is None:
            outs = [t.numel() for t in (out_child, out_parent, out_ordinal) if t is not None]
            out_cap = min(outs) if outs else q_len
        P = offsets.numel() - 1
        _check(self.L.ro_batch(self.h, *_queue_args(queue, keep, q_len), _ptr(offsets, 8, 1, "offsets"), P,
                               int(batch_size), *_tag_args(out_child, out_parent, out_ordinal, out_cap),
                               _ptr(n_out, 8, 1, "n_out"), _ptr(n_batches, 8, 1, "n_batches"),
                               _ptr(barrier, 1, P, "barrier")),
               "ro_batch")

    def batch_parent(self, queue, keep, offsets, batch_size, batch_off, out_child=None, out_parent=None,
                     out_ordinal=None, n_out=None, n_batches=None, q_len=None, out_cap=None, barrier=None):
        """Parent-bound reservations; batch j is slots [batch_off[j], batch_off[j+1])."""
        q_len = queue.numel() if q_len is None else q_len
        if out_cap is None:
            outs = [t.numel() for t in (out_child, out_parent, out_ordinal) if t is not None]
            out_cap = min(outs) if outs else q_len
        P = offsets.numel() - 1
        _check(self.L.ro_batch_parent(self.h, *_queue_args(queue, keep, q_len), _ptr(offsets, 8, 1, "offsets"), P,
                                      int(batch_size), *_tag_args(out_child, out_parent, out_ordinal, out_cap),
                                      _ptr(batch_off, 8, 1, "batch_off"), batch_off.numel(),
                                      _ptr(n_out, 8, 1, "n_out"), _ptr(n_batches, 8, 1, "n_batches"),
                                      _ptr(barrier, 1, P, "barrier")),
               "ro_batch_parent")

    def gather(self, parent, ordinal, state, off, data, offsets, out_off, out_data=None,
               n_success=None, n_failed=None, n_skipped=None, complete=None, parent_state=None,
               n=None, out_cap=None, child_dst_off=None, barrier=None, n_rejected=None):
        rep = _reports(parent, ordinal, state, off, data, n)
        if out_cap is None:
            out_cap = out_data.numel() if out_data is not None else 0
        P = offsets.numel() - 1
        out = GatherOutT(_ptr(out_off, 8, P + 1, "out_off"), _ptr(out_data, 1, int(out_cap), "out_data"),
                         int(out_cap), _ptr(n_success, 4, P, "n_success"), _ptr(n_failed, 4, P, "n_failed"),
                         _ptr(n_skipped, 4, P, "n_skipped"), _ptr(complete, 1, P, "complete"),
                         _ptr(parent_state, 1, P, "parent_state"), _ptr(child_dst_off, 8, 1, "child_dst_off"),
                         _ptr(barrier, 1, P, "barrier"), _ptr(n_rejected, 8, 1, "n_rejected"))
        _check(self.L.ro_gather(self.h, C.byref(rep), _ptr(offsets, 8, 1, "offsets"), P, C.byref(out)),
               "ro_gather")

    def filter(self, x_state, mask, out_state, mask_state=None, n=None):
        n = x_state.numel() if n is None else int(n)
        _check(self.L.ro_filter(self.h, _ptr(x_state, 1, n, "x_state"), _ptr(mask_state, 1, n, "mask_state"),
                                _ptr(mask, 1, n, "mask"), n, _ptr(out_state, 1, n, "out_state")),
               "ro_filter")

    def broadcast(self, maps, x_state, out_state, out_ancestor=None, like_state=None, n=None):
        """maps: device tensors, the descendant level's child->parent first."""
        n = maps[0].numel() if n is None else int(n)
        _ptr(maps[0], 4, n, "maps[0]")
        arr = (C.c_void_p * len(maps))(*[_ptr(m, 4, 0, "map").value for m in maps])
        lens = (C.c_int64 * len(maps))(*[m.numel() for m in maps])
        _check(self.L.ro_broadcast(self.h, C.cast(arr, C.c_void_p), C.cast(lens, C.c_void_p), len(maps), n,
                                   _ptr(x_state, 1, 0, "x_state"),
                                   x_state.numel(), _ptr(like_state, 1, n, "like_state"),
                                   _ptr(out_ancestor, 4, n, "out_ancestor"), _ptr(out_state, 1, n, "out_state")),
               "ro_broadcast")

    def grains(self, n_children):
        g = Grains(self, n_children)
        self._owned.add(g)
        return g

    def stream(self, offsets, n_children, barrier=None):
        st = Stream(self, offsets, n_children, barrier)
        self._owned.add(st)
        return st

    def close(self):
        if getattr(self, "h", None):
            for o in list(getattr(self, "_owned", ())):
                o.close()
            self.L.ro_ctx_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Grains:
    """Grain phases and generations of one Call's children (device side)."""

    def __init__(self, ctx, n_children):
        self.ctx = ctx
        self.n = int(n_children)
        h = C.c_void_p()
        _check(ctx.L.ro_grains_create(ctx.h, self.n, C.byref(h)), "ro_grains_create")
        self.h = h

    def reset(self):
        _check(self.ctx.L.ro_grains_reset(self.ctx.h, self.h), "ro_grains_reset")

    def read(self, phase=None, generation=None):
        """Write every child's phase and generation into int32 device tensors
        of n_children entries (either may be None)."""
        _check(self.ctx.L.ro_grains_read(self.ctx.h, self.h, _ptr(phase, 4, self.n, "phase"),
                                         _ptr(generation, 4, self.n, "generation")), "ro_grains_read")

    def dispatch(self, child, out_generation=None, n=None):
        n = child.numel() if n is None else int(n)
        _check(self.ctx.L.ro_grains_dispatch(self.ctx.h, self.h, _ptr(child, 4, n, "child"), n,
                                             _ptr(out_generation, 4, n, "out_generation")),
               "ro_grains_dispatch")

    def retry(self, child, n=None):
        n = child.numel() if n is None else int(n)
        _check(self.ctx.L.ro_grains_retry(self.ctx.h, self.h, _ptr(child, 4, n, "child"), n), "ro_grains_retry")

    def commit(self, parent, ordinal, state, off, data, generation, offsets, state_out, counts=None, n=None):
        rep = _reports(parent, ordinal, state, off, data, n)
        _check(self.ctx.L.ro_grains_commit(self.ctx.h, self.h, C.byref(rep), _ptr(generation, 4, rep.n, "generation"),
                                           _ptr(offsets, 8, 1, "offsets"), offsets.numel() - 1,
                                           _ptr(state_out, 1, rep.n, "state_out"), _ptr(counts, 8, 4, "counts")),
               "ro_grains_commit")

    def close(self):
        if getattr(self, "h", None):
            self.ctx.L.ro_grains_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Stream:
    """Streaming gather over one expansion."""

    def __init__(self, ctx, offsets, n_children, barrier=None):
        self.ctx = ctx
        self.offsets = offsets
        self.barrier = barrier          # kept alive: the library holds it by reference
        h = C.c_void_p()
        P = offsets.numel() - 1
        _check(ctx.L.ro_stream_create(ctx.h, _ptr(offsets, 8, 1, "offsets"), P, int(n_children),
                                      _ptr(barrier, 1, P, "barrier"), C.byref(h)), "ro_stream_create")
        self.h = h

    def batch(self, queue, keep, batch_size, out_child=None, out_parent=None, out_ordinal=None, n_out=None,
              n_batches=None, q_len=None, out_cap=None):
        """FIFO batches of one wave (ro_batch over this stream's expansion and barrier)."""
        q_len = queue.numel() if q_len is None else q_len
        if out_cap is None:
            outs = [t.numel() for t in (out_child, out_parent, out_ordinal) if t is not None]
            out_cap = min(outs) if outs else q_len
        _check(self.ctx.L.ro_stream_batch(self.ctx.h, self.h, *_queue_args(queue, keep, q_len), int(batch_size),
                                          *_tag_args(out_child, out_parent, out_ordinal, out_cap),
                                          _ptr(n_out, 8, 1, "n_out"), _ptr(n_batches, 8, 1, "n_batches")),
               "ro_stream_batch")

    def report(self, parent, ordinal, state, off, data, n=None, n_rejected=None):
        rep = _reports(parent, ordinal, state, off, data, n)
        _check(self.ctx.L.ro_stream_report(self.ctx.h, self.h, C.byref(rep), _ptr(n_rejected, 8, 1, "n_rejected")),
               "ro_stream_report")

    def emit(self, emit_parent, emit_off, emit_data, n_success=None, n_failed=None, n_skipped=None,
             parent_state=None, n_emitted=None, n_bytes=None, cap_parents=None, cap_bytes=None):
        if cap_parents is None:
            cap_parents = emit_off.numel() - 1
        if cap_bytes is None:
            cap_bytes = emit_data.numel() if emit_data is not None else 0
        cp, cb = int(cap_parents), int(cap_bytes)
        _check(self.ctx.L.ro_stream_emit(self.ctx.h, self.h, _ptr(emit_parent, 4, cp, "emit_parent"),
                                         _ptr(emit_off, 8, cp + 1, "emit_off"), _ptr(emit_data, 1, cb, "emit_data"),
                                         cp, cb, _ptr(n_success, 4, cp, "n_success"),
                                         _ptr(n_failed, 4, cp, "n_failed"), _ptr(n_skipped, 4, cp, "n_skipped"),
                                         _ptr(parent_state, 1, cp, "parent_state"),
                                         _ptr(n_emitted, 8, 1, "n_emitted"), _ptr(n_bytes, 8, 1, "n_bytes")),
               "ro_stream_emit")

    def reset(self):
        """Forget every report and emission (stream-ordered; keeps the allocation)."""
        _check(self.ctx.L.ro_stream_reset(self.ctx.h, self.h), "ro_stream_reset")

    def close(self):
        if getattr(self, "h", None):
            self.ctx.L.ro_stream_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
