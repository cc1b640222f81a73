"""Chains of ro calls for one expansion level and for two nested levels.

These functions only sequence C-ABI calls on device tensors the caller owns;
every step runs in the HIP library.

Single level (a batch of one Call over the children of one expansion):
  1. ro_expand  counts -> offsets, per-child (parent, ordinal)
  2. ro_batch   ready queue with the dispatch mask -> report tags of the
                dispatched children, in FIFO order, slots [0, M)
  3. ro_batch   the list of children that turned terminal without dispatch
                (sealed before reaching the queue head) -> their report tags,
                slots [M, N)
  4. ro_gather  reports -> parent slots, counts, completion

Nested (two expansions, RayOrch's multi-grain program shape): the lower
gather's slots and derived states are the upper level's child reports, keyed
by the level-1 children's own lineage (parent, ordinal).
"""
from __future__ import annotations

import torch

__all__ = ["SingleLevelBuffers", "single_level", "NestedBuffers", "nested", "StreamingBuffers",
           "streaming"]


def _empty(n, dtype):
    return torch.empty(max(int(n), 1), dtype=dtype, device="cuda")


class SingleLevelBuffers:
    """Device inputs and outputs of one single-level pipeline."""

    def __init__(self, counts, queue, keep, sealed_ids, rep_state, rep_off, data, n_children,
                 n_dispatched, batch_size, out_cap=None, want_data=True):
        P = counts.numel()
        N = int(n_children)
        self.counts, self.queue, self.keep, self.sealed_ids = counts, queue, keep, sealed_ids
        self.rep_state, self.rep_off, self.data = rep_state, rep_off, data
        self.N, self.M, self.B = N, int(n_dispatched), int(batch_size)
        self.offsets = _empty(P + 1, torch.int64)
        self.child_parent = _empty(N, torch.int32)
        self.child_ordinal = _empty(N, torch.int32)
        self.rep_parent = _empty(N, torch.int32)
        self.rep_ordinal = _empty(N, torch.int32)
        self.scalars = torch.zeros(4, dtype=torch.int64, device="cuda")   # M, nb, N-M, nb'
        self.out_off = _empty(P + 1, torch.int64)
        if out_cap is None:
            out_cap = int(rep_off[-1].item() - rep_off[0].item()) if N else 0
        self.out_cap = int(out_cap)
        self.out_data = _empty(self.out_cap, torch.uint8) if want_data else None
        self.n_success = _empty(P, torch.int32)
        self.n_failed = _empty(P, torch.int32)
        self.n_skipped = _empty(P, torch.int32)
        self.complete = _empty(P, torch.uint8)
        self.parent_state = _empty(P, torch.uint8)


def single_level(ctx, b: SingleLevelBuffers):
    """Enqueue the four calls of one level on ctx's stream."""
    N, M = b.N, b.M
    ctx.expand(b.counts, b.offsets, b.child_parent, b.child_ordinal)
    ctx.batch(b.queue, b.keep, b.offsets, b.B, None, b.rep_parent, b.rep_ordinal,
              b.scalars[0:1], b.scalars[1:2], out_cap=M)
    if N > M:
        ctx.batch(b.sealed_ids, None, b.offsets, b.B, None, b.rep_parent[M:], b.rep_ordinal[M:],
                  b.scalars[2:3], b.scalars[3:4], q_len=N - M, out_cap=N - M)
    ctx.gather(b.rep_parent, b.rep_ordinal, b.rep_state, b.rep_off, b.data, b.offsets, b.out_off,
               b.out_data, b.n_success, b.n_failed, b.n_skipped, b.complete, b.parent_state, n=N,
               out_cap=b.out_cap)


class NestedBuffers:
    """Device inputs and outputs of a two-level pipeline (top -> mid -> leaf).

    With ``upper_in_place`` the top level's bytes are the mid level's buffer
    itself: valid when every mid slot survives (no failed leaf), since each
    top slot then is the run of its mid slots as they already lie.  The upper
    gather checks this on the device and copies nothing (RO_EINVAL if a mid
    slot would have to move).
    """

    def __init__(self, counts1, queue1, batch1, counts2, queue2, batch2, leaf_state, leaf_off,
                 leaf_data, n_mid, n_leaf, want_data=True, upper_in_place=False):
        P1 = counts1.numel()
        self.P1, self.N1, self.N2 = P1, int(n_mid), int(n_leaf)
        self.counts1, self.queue1, self.B1 = counts1, queue1, int(batch1)
        self.counts2, self.queue2, self.B2 = counts2, queue2, int(batch2)
        self.leaf_state, self.leaf_off, self.leaf_data = leaf_state, leaf_off, leaf_data
        N1, N2 = self.N1, self.N2
        self.offsets1 = _empty(P1 + 1, torch.int64)
        self.mid_parent = _empty(N1, torch.int32)
        self.mid_ordinal = _empty(N1, torch.int32)
        self.b1_parent = _empty(N1, torch.int32)
        self.b1_ordinal = _empty(N1, torch.int32)
        self.offsets2 = _empty(N1 + 1, torch.int64)
        self.leaf_parent = _empty(N2, torch.int32)
        self.leaf_ordinal = _empty(N2, torch.int32)
        self.b2_parent = _empty(N2, torch.int32)
        self.b2_ordinal = _empty(N2, torch.int32)
        self.scalars = torch.zeros(4, dtype=torch.int64, device="cuda")
        cap = int(leaf_off[-1].item() - leaf_off[0].item()) if N2 else 0
        self.mid_off = _empty(N1 + 1, torch.int64)
        self.mid_data = _empty(cap, torch.uint8) if want_data else None
        self.mid_cnt = _empty(3 * N1, torch.int32)
        self.mid_complete = _empty(N1, torch.uint8)
        self.mid_state = _empty(N1, torch.uint8)
        self.top_off = _empty(P1 + 1, torch.int64)
        if not want_data:
            self.top_data = None
        elif upper_in_place:
            self.top_data = self.mid_data
        else:
            self.top_data = _empty(cap, torch.uint8)
        self.top_cnt = _empty(3 * P1, torch.int32)
        self.top_complete = _empty(P1, torch.uint8)
        self.top_state = _empty(P1, torch.uint8)
        self.cap = cap


def nested(ctx, b: NestedBuffers):
    """expand(top) -> batch(mid) -> expand(mid) -> batch(leaf) -> gather(leaf->mid) -> gather(mid->top)."""
    N1, N2 = b.N1, b.N2
    ctx.expand(b.counts1, b.offsets1, b.mid_parent, b.mid_ordinal)
    ctx.batch(b.queue1, None, b.offsets1, b.B1, None, b.b1_parent, b.b1_ordinal,
              b.scalars[0:1], b.scalars[1:2], out_cap=N1)
    ctx.expand(b.counts2, b.offsets2, b.leaf_parent, b.leaf_ordinal)
    ctx.batch(b.queue2, None, b.offsets2, b.B2, None, b.b2_parent, b.b2_ordinal,
              b.scalars[2:3], b.scalars[3:4], out_cap=N2)
    ctx.gather(b.b2_parent, b.b2_ordinal, b.leaf_state, b.leaf_off, b.leaf_data, b.offsets2,
               b.mid_off, b.mid_data, b.mid_cnt[:N1], b.mid_cnt[N1:2 * N1], b.mid_cnt[2 * N1:],
               b.mid_complete, b.mid_state, n=N2, out_cap=b.cap)
    ctx.gather(b.mid_parent, b.mid_ordinal, b.mid_state, b.mid_off, b.mid_data, b.offsets1,
               b.top_off, b.top_data, b.top_cnt[:b.P1], b.top_cnt[b.P1:2 * b.P1], b.top_cnt[2 * b.P1:],
               b.top_complete, b.top_state, n=N1, out_cap=b.cap)


class StreamingBuffers:
    """Device inputs and per-wave outputs of a streaming run over one expansion.

    ``queues[w]`` are the children that turn terminal in wave w (in ready
    order), ``states[w]`` / ``offs[w]`` their reports; every wave's bytes live
    in one arena (``data``) that outlives the run.
    """

    def __init__(self, counts, queues, states, offs, data, n_children, batch_size, emit_cap_bytes):
        P = counts.numel()
        self.P, self.N, self.B = P, int(n_children), int(batch_size)
        self.counts, self.queues, self.states, self.offs, self.data = counts, queues, states, offs, data
        self.offsets = _empty(P + 1, torch.int64)
        wmax = max((q.numel() for q in queues), default=1)
        self.tag_parent = _empty(wmax, torch.int32)
        self.tag_ordinal = _empty(wmax, torch.int32)
        self.scalars = torch.zeros(4, dtype=torch.int64, device="cuda")   # M, nb, emitted, bytes
        self.emit_parent = _empty(P, torch.int32)
        self.emit_off = _empty(P + 1, torch.int64)
        self.emit_cap = int(emit_cap_bytes)
        self.emit_data = _empty(self.emit_cap, torch.uint8)
        self.emit_cnt = _empty(3 * P, torch.int32)
        self.emit_state = _empty(P, torch.uint8)


def streaming(ctx, b: StreamingBuffers, on_wave=None, st=None):
    """expand once; per wave: the stream's batch -> stream report -> stream emit.

    ``on_wave(w)`` (optional) runs after each wave's emission is enqueued, to
    consume that wave's outputs before the next wave overwrites them.  ``st``
    (optional) is a stream created earlier over ``b.offsets``: it is reset and
    reused instead of creating one for this run.
    """
    P = b.P
    ctx.expand(b.counts, b.offsets)
    own = st is None
    if own:
        st = ctx.stream(b.offsets, b.N)
    else:
        st.reset()
    try:
        for w, q in enumerate(b.queues):
            n = q.numel()
            st.batch(q, None, b.B, None, b.tag_parent, b.tag_ordinal, b.scalars[0:1], b.scalars[1:2], q_len=n,
                     out_cap=n)
            st.report(b.tag_parent, b.tag_ordinal, b.states[w], b.offs[w], b.data, n=n)
            st.emit(b.emit_parent, b.emit_off, b.emit_data, b.emit_cnt[:P], b.emit_cnt[P:2 * P],
                    b.emit_cnt[2 * P:], b.emit_state, b.scalars[2:3], b.scalars[3:4],
                    cap_parents=P, cap_bytes=b.emit_cap)
            if on_wave is not None:
                on_wave(w)
    finally:
        if own:
            st.close()
