"""Wave schedule of the group-failure trace (test driver).

Each wave reserves up to `wave` entries (actors x batch) from the head of
the Call's ready queue, after the barrier has dropped the queued siblings of
barred parents; the reserved children report (group failure at the poisoned
first pages, success elsewhere), the reports commit in batch order, and the
complete or barred parents are emitted.  What is left of the queue carries
over to the next wave.
"""
import numpy as np

import oracle as O
import workloads as W


def wave_reports(t, disp, par, ordi, base):
    """Reports of the dispatched children, in batch order, with their bytes."""
    st = t.states[disp].astype(np.uint8)
    ln = np.where(st == W.SUCCESS, t.lengths[disp], 0).astype(np.int64)
    off = base + np.concatenate([[0], np.cumsum(ln)]).astype(np.int64)
    ok = st == W.SUCCESS
    data = W.record_bytes(W.content_seed(par[ok], ordi[ok]), ln[ok])
    return st, off, data


def oracle_waves(t):
    """Run the schedule on the oracle; per wave: dispatched children, tags,
    report states and offsets, the number of suppressed queue entries, the
    number of rejected reports, and the emission."""
    offs = O.expand(t.counts, tags=False)
    st = O.Stream(offs)
    remaining = t.queue.copy()
    base = 0
    arena = []
    out = []
    while len(remaining):
        child, par, ordi, _ = O.batch(remaining, None, offs, t.batch_size, barrier=st.barrier())
        d = min(t.wave, len(child))
        states, off, data = wave_reports(t, child[:d], par[:d], ordi[:d], base)
        arena.append(data)
        whole = np.concatenate(arena) if arena else np.zeros(0, np.uint8)
        rej = st.report(par[:d], ordi[:d], states, off, whole)
        em = st.emit()
        out.append(dict(queue=remaining, child=child, dispatched=child[:d], parent=par[:d], ordinal=ordi[:d],
                        state=states,
                        off=off, data=data, suppressed=len(remaining) - len(child), rejected=rej, emitted=em))
        base = int(off[-1])
        remaining = child[d:]
    st.close()
    return offs, out
