"""Pure-Python brute force for tiny inputs (test infrastructure only).

A second, independent formulation of the same definitions as ``oracle.c``
(Sec. 4 of the paper: Eq. flat-facts, the Reduce rule, FIFO Ready Queues with
elastic and parent-bound reservation).  Where the C oracle scans offsets and sorts reports,
this one enumerates the (parent, ordinal) pairs and looks every child up by a
linear search over all reports, so the two share no algorithm.
"""
from __future__ import annotations

SUCCESS, FAILED, SKIPPED, PENDING = 0, 1, 2, 3


class BruteError(RuntimeError):
    def __init__(self, code):
        super().__init__(f"brute error {code}")
        self.code = code


def children(counts):
    """All child keys (p, o) with o < k_p, in lexicographic order."""
    keys = []
    for p, k in enumerate(counts):
        if k < 0:
            raise BruteError(-1)
        keys.extend((p, o) for o in range(k))
    return keys


def expand(counts):
    keys = children(counts)
    offsets = [sum(1 for (p, _) in keys if p < q) for q in range(len(counts) + 1)]
    return offsets, [p for p, _ in keys], [o for _, o in keys]


def batch(queue, keep, counts, B):
    """Literal queue simulation; returns the list of batches of child ids."""
    keys = children(counts)
    ready = [c for i, c in enumerate(queue) if keep is None or keep[i]]
    for c in ready:
        if c >= len(keys):
            raise BruteError(-2)
    batches = []
    while ready:
        batches.append(ready[:B])
        ready = ready[B:]
    return batches, keys


def batch_parent(queue, keep, counts, B):
    """Literal parent-bound reservations on a list: the head's parent takes
    its first (at most B) entries found scanning the queue from the head, and
    the queue is rebuilt without them.  Returns the list of batches of child
    ids."""
    keys = children(counts)
    ready = [c for i, c in enumerate(queue) if keep is None or keep[i]]
    for c in ready:
        if c >= len(keys):
            raise BruteError(-2)
    batches = []
    while ready:
        p = keys[ready[0]][0]
        take = [c for c in ready if keys[c][0] == p][:B]
        batches.append(take)
        ready = [c for c in ready if c not in take]
    return batches, keys


def gather(reports, counts):
    """reports: list of (parent, ordinal, state, bytes).  Returns per-parent
    tuples (n_success, n_failed, n_skipped, complete, state, bytes)."""
    for (p, o, s, _) in reports:
        if s > PENDING:
            raise BruteError(-6)
        if s == PENDING:
            continue
        if p >= len(counts) or o >= counts[p]:
            raise BruteError(-2)
    out = []
    for p, k in enumerate(counts):
        ns = nf = nk = 0
        slot = b""
        for o in range(k):
            hits = [r for r in reports if r[2] != PENDING and r[0] == p and r[1] == o]
            if len(hits) > 1:
                raise BruteError(-3)
            if not hits:
                continue
            _, _, s, b = hits[0]
            if s == SUCCESS:
                ns += 1
                slot += bytes(b)
            elif s == FAILED:
                nf += 1
            else:
                nk += 1
        done = ns + nf + nk == k
        state = PENDING if not done else (FAILED if nf else SUCCESS)
        out.append((ns, nf, nk, int(done), state, slot))
    return out


def stream(waves, counts):
    """waves: list of report lists.  Returns per-wave lists of emitted
    (parent, n_success, n_failed, n_skipped, state, bytes)."""
    seen = set()
    got = {}
    emitted = set()
    result = []
    for wave in waves:
        for (p, o, s, b) in wave:
            if s == PENDING:
                continue
            if p >= len(counts) or o >= counts[p] or s > PENDING:
                raise BruteError(-2)
            if (p, o) in seen:
                raise BruteError(-3)
            seen.add((p, o))
            got[(p, o)] = (s, bytes(b))
        em = []
        for p, k in enumerate(counts):
            if p in emitted:
                continue
            if all((p, o) in got for o in range(k)):
                sts = [got[(p, o)][0] for o in range(k)]
                data = b"".join(got[(p, o)][1] for o in range(k) if got[(p, o)][0] == SUCCESS)
                nf = sts.count(FAILED)
                em.append((p, sts.count(SUCCESS), nf, sts.count(SKIPPED),
                           FAILED if nf else SUCCESS, data))
                emitted.add(p)
        result.append(em)
    return result
