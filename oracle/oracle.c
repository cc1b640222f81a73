/*
 * CPU oracle for expand / FIFO batch / ordered gather / streaming emission.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU
 * baseline leg of the benchmark load this file's library.  It shares no code,
 * header, table or helper with the HIP library: it is the plain definition of
 * what the lineage-controlled dataflow computes, written slowly and obviously,
 * single threaded, so that a reader can check it against the paper by eye.
 *
 * Sources (RayOrch, arXiv 2609.18703):
 *   - Sec. 4 "Lineage State and Parent Completion", Eq. (flat-facts): every
 *     object publishes exactly one terminal fact; an Expansion is the ordered
 *     child set of one parent; an empty successful Expansion is terminal;
 *     each child carries its parent's immutable zero-based ordinal.
 *   - same section, publication rules: facts are irreversible and conflicting
 *     publications are rejected (a second report for one child is an error).
 *   - same section, Reduce rule: a parent Item is emitted only once its
 *     Expansion and every member outcome are resolved; dropped members are
 *     excluded, failed/suppressed members suppress the parent, present values
 *     are emitted in ordinal order, zero survivors give a present empty list.
 *   - Sec. 4 "Scheduling Ready Grains": one FIFO Ready Queue per Call holds
 *     ready Grains in enqueue order; elastic reservation removes at most B
 *     entries from its head and may mix parents; parent-bound reservation
 *     takes up to B siblings of the first ready parent and leaves the rest
 *     of the queue in order.
 *   - Sec. 4 input propagation and Table "primitives": F.filter keeps or
 *     drops an Item in its own Domain, F.broadcast makes an ancestor's Item
 *     available in a descendant Domain, both under the precedence failed /
 *     suppressed, then unresolved, then dropped, then ready.
 *   - Sec. 4, Eq. (grain-phase) and Eq. (generation-fence): a report commits
 *     only while its Grain is in flight at the report's generation; a retry
 *     returns the Grain to READY at the next generation.
 *   - Sec. 4 "Commit, Failure, and Recovery": a typed GroupFailure puts a
 *     suppression barrier on one (Call, parent): queued siblings are
 *     suppressed before dispatch, in-flight siblings may finish but cannot
 *     commit, siblings committed before it stay as they are.
 *
 * Readings where the paper is silent (all listed in the design notes):
 *   state SUCCESS = Present, FAILED = Failed (and Suppressed passed up from a
 *   lower level), SKIPPED = Dropped, PENDING = no report yet; bytes of a
 *   non-SUCCESS report are never copied; a parent with a failed member keeps
 *   its packed surviving bytes and is flagged FAILED; an incomplete parent is
 *   PENDING with the bytes seen so far packed in ordinal order.  Group
 *   failures: reports commit in the order given (one call or wave after
 *   another); a GROUP_FAILED report commits as a failed member and bars its
 *   parent, so every later report of that parent is rejected (not committed,
 *   not counted, its bytes never copied); a barred parent is complete and
 *   FAILED, its slot keeps the bytes committed before the barrier; a barred
 *   parent's queued children are dropped by the batch.  GROUP_FAILED needs a
 *   barrier array (one per Call); without one it is a bad state.
 *
 * Parity status: every function here is pinned by the CPU test suite (worked
 * examples from the paper's figures, brute-force enumeration on tiny inputs,
 * closed forms and invariants).  No function is "parity unpinned".
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { OR_OK = 0, OR_EINVAL = -1, OR_ERANGE = -2, OR_EDUP = -3, OR_ECAP = -4,
       OR_EOVERFLOW = -5, OR_ESTATE = -6 };
enum { ST_SUCCESS = 0, ST_FAILED = 1, ST_SKIPPED = 2, ST_PENDING = 3, ST_GROUP_FAILED = 4 };

/* ------------------------------------------------------------------------ */
/* F.expand: child counts -> Expansion offsets and per-child lineage keys.   */
/* ------------------------------------------------------------------------ */
/* offsets[0] = 0, offsets[p+1] = offsets[p] + counts[p]: parent p's ordered
 * child set is the canonical id range [offsets[p], offsets[p+1]).  Child
 * number o of parent p gets the key (p, o). */
int oracle_expand(const int32_t *counts, int64_t n_parents, int64_t *offsets,
                  uint32_t *child_parent, uint32_t *child_ordinal, int64_t child_cap)
{
    if (n_parents < 0 || offsets == NULL || (n_parents > 0 && counts == NULL))
        return OR_EINVAL;
    offsets[0] = 0;
    for (int64_t p = 0; p < n_parents; ++p) {
        if (counts[p] < 0)
            return OR_EINVAL;
        offsets[p + 1] = offsets[p] + (int64_t)counts[p];
    }
    int64_t n = offsets[n_parents];
    if (n >= ((int64_t)1 << 32))
        return OR_EOVERFLOW;
    if (child_parent != NULL || child_ordinal != NULL) {
        if (n > child_cap)
            return OR_ECAP;
        int64_t c = 0;
        for (int64_t p = 0; p < n_parents; ++p) {
            for (int64_t o = 0; o < counts[p]; ++o) {
                if (child_parent)  child_parent[c] = (uint32_t)p;
                if (child_ordinal) child_ordinal[c] = (uint32_t)o;
                ++c;
            }
        }
    }
    return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* FIFO Ready Queue + elastic reservation of at most B entries.              */
/* ------------------------------------------------------------------------ */
typedef struct {
    uint32_t *slot;
    int64_t head, tail;          /* pop at head, push at tail */
} fifo_t;

static void fifo_push(fifo_t *q, uint32_t v) { q->slot[q->tail++] = v; }
static int fifo_empty(const fifo_t *q) { return q->head == q->tail; }
static uint32_t fifo_pop(fifo_t *q) { return q->slot[q->head++]; }

/* Every ready entry i with keep[i] != 0 (all entries if keep == NULL) is
 * appended to the queue in order; then reservations repeatedly take at most
 * B entries from the head until the queue is empty.  Batch j is written to
 * slots [j*B, j*B + size_j) of the outputs; batch_size_out (optional) gets
 * size_j.  The (parent, ordinal) tags of child c come from the same per-parent
 * enumeration as oracle_expand.  With a barrier array, an entry whose parent
 * is barred is suppressed before dispatch: it never enters the queue. */
int oracle_batch(const uint32_t *queue, const uint8_t *keep, int64_t q_len,
                 const int64_t *offsets, int64_t n_parents, int32_t batch_size,
                 uint32_t *out_child, uint32_t *out_parent, uint32_t *out_ordinal,
                 int64_t out_cap, int64_t *n_out, int64_t *n_batches,
                 int64_t *batch_size_out, const uint8_t *barrier)
{
    if (q_len < 0 || n_parents < 0 || batch_size <= 0 || offsets == NULL ||
        (q_len > 0 && queue == NULL))
        return OR_EINVAL;
    int64_t n = offsets[n_parents];
    uint32_t *par = (uint32_t *)malloc(sizeof(uint32_t) * (size_t)(n > 0 ? n : 1));
    uint32_t *ord = (uint32_t *)malloc(sizeof(uint32_t) * (size_t)(n > 0 ? n : 1));
    fifo_t q;
    q.slot = (uint32_t *)malloc(sizeof(uint32_t) * (size_t)(q_len > 0 ? q_len : 1));
    q.head = q.tail = 0;
    int rc = OR_OK;
    if (!par || !ord || !q.slot) { rc = OR_EINVAL; goto done; }
    for (int64_t p = 0; p < n_parents; ++p)
        for (int64_t c = offsets[p]; c < offsets[p + 1]; ++c) {
            par[c] = (uint32_t)p;
            ord[c] = (uint32_t)(c - offsets[p]);
        }
    for (int64_t i = 0; i < q_len; ++i) {
        if (keep != NULL && keep[i] == 0)
            continue;
        if ((int64_t)queue[i] >= n) { rc = OR_ERANGE; goto done; }
        if (barrier != NULL && barrier[par[queue[i]]])
            continue;                         /* suppressed: never dispatched */
        fifo_push(&q, queue[i]);
    }
    if (q.tail > out_cap) { rc = OR_ECAP; goto done; }
    int64_t slot = 0, nb = 0;
    while (!fifo_empty(&q)) {
        /* one elastic reservation: at most B entries, parents may mix */
        int64_t taken = 0;
        while (taken < batch_size && !fifo_empty(&q)) {
            uint32_t c = fifo_pop(&q);
            if (out_child)   out_child[slot] = c;
            if (out_parent)  out_parent[slot] = par[c];
            if (out_ordinal) out_ordinal[slot] = ord[c];
            ++slot;
            ++taken;
        }
        if (batch_size_out) batch_size_out[nb] = taken;
        ++nb;
    }
    if (n_out) *n_out = slot;
    if (n_batches) *n_batches = nb;
done:
    free(par);
    free(ord);
    free(q.slot);
    return rc;
}

/* ------------------------------------------------------------------------ */
/* FIFO Ready Queue + parent-bound reservation.                              */
/* ------------------------------------------------------------------------ */
/* Sec. 4 "Scheduling Ready Grains": a parent-bound reservation takes up to B
 * siblings of the first ready parent, and every entry it leaves keeps its
 * place in the queue.  The queue is filled as in oracle_batch (kept entries
 * in order, barred parents' entries suppressed).  Each reservation looks at
 * the head, the earliest entry still queued; its parent is the first ready
 * parent; the reservation takes that parent's queued entries in queue order,
 * at most B of them, and marks them gone.  Each parent keeps the list of its
 * queued entries in queue order, so finding the siblings does not rescan the
 * queue.  Outputs as in oracle_batch, except that batch j starts where batch
 * j - 1 ends (sizes vary; batch_size_out gives them). */
int oracle_batch_parent(const uint32_t *queue, const uint8_t *keep, int64_t q_len,
                        const int64_t *offsets, int64_t n_parents, int32_t batch_size,
                        uint32_t *out_child, uint32_t *out_parent, uint32_t *out_ordinal,
                        int64_t out_cap, int64_t *n_out, int64_t *n_batches,
                        int64_t *batch_size_out, const uint8_t *barrier)
{
    if (q_len < 0 || n_parents < 0 || batch_size <= 0 || offsets == NULL ||
        (q_len > 0 && queue == NULL))
        return OR_EINVAL;
    int64_t n = offsets[n_parents];
    size_t m = (size_t)(q_len > 0 ? q_len : 1);
    size_t np = (size_t)(n_parents > 0 ? n_parents : 1);
    uint32_t *par = (uint32_t *)malloc(sizeof(uint32_t) * (size_t)(n > 0 ? n : 1));
    uint32_t *ord = (uint32_t *)malloc(sizeof(uint32_t) * (size_t)(n > 0 ? n : 1));
    uint32_t *qc = (uint32_t *)malloc(sizeof(uint32_t) * m);      /* queued children, in order */
    int64_t *next = (int64_t *)malloc(sizeof(int64_t) * m);       /* next queued sibling */
    uint8_t *gone = (uint8_t *)calloc(m, 1);
    int64_t *first = (int64_t *)malloc(sizeof(int64_t) * np);     /* parent's earliest queued entry */
    int64_t *last = (int64_t *)malloc(sizeof(int64_t) * np);
    int rc = OR_OK;
    if (!par || !ord || !qc || !next || !gone || !first || !last) { rc = OR_EINVAL; goto done; }
    for (int64_t p = 0; p < n_parents; ++p) {
        first[p] = last[p] = -1;
        for (int64_t c = offsets[p]; c < offsets[p + 1]; ++c) {
            par[c] = (uint32_t)p;
            ord[c] = (uint32_t)(c - offsets[p]);
        }
    }
    int64_t len = 0;
    for (int64_t i = 0; i < q_len; ++i) {
        if (keep != NULL && keep[i] == 0)
            continue;
        if ((int64_t)queue[i] >= n) { rc = OR_ERANGE; goto done; }
        uint32_t p = par[queue[i]];
        if (barrier != NULL && barrier[p])
            continue;                         /* suppressed: never dispatched */
        qc[len] = queue[i];
        next[len] = -1;
        if (last[p] < 0) first[p] = len; else next[last[p]] = len;
        last[p] = len;
        ++len;
    }
    if (len > out_cap) { rc = OR_ECAP; goto done; }
    int64_t slot = 0, nb = 0, head = 0;
    for (;;) {
        while (head < len && gone[head]) ++head;
        if (head == len) break;
        /* one parent-bound reservation: the head's parent, at most B siblings */
        uint32_t p = par[qc[head]];
        int64_t taken = 0;
        while (taken < batch_size && first[p] >= 0) {
            int64_t e = first[p];
            uint32_t c = qc[e];
            gone[e] = 1;
            first[p] = next[e];
            if (out_child)   out_child[slot] = c;
            if (out_parent)  out_parent[slot] = p;
            if (out_ordinal) out_ordinal[slot] = ord[c];
            ++slot;
            ++taken;
        }
        if (batch_size_out) batch_size_out[nb] = taken;
        ++nb;
    }
    if (n_out) *n_out = slot;
    if (n_batches) *n_batches = nb;
done:
    free(par); free(ord); free(qc); free(next); free(gone); free(first); free(last);
    return rc;
}

/* ------------------------------------------------------------------------ */
/* F.reduce: ordered gather of child reports into parent slots.              */
/* ------------------------------------------------------------------------ */
typedef struct {
    uint32_t parent, ordinal;
    int64_t index;               /* report position: makes the sort stable */
} key_t;

static int key_cmp(const void *a, const void *b)
{
    const key_t *x = (const key_t *)a, *y = (const key_t *)b;
    if (x->parent != y->parent) return x->parent < y->parent ? -1 : 1;
    if (x->ordinal != y->ordinal) return x->ordinal < y->ordinal ? -1 : 1;
    if (x->index != y->index) return x->index < y->index ? -1 : 1;
    return 0;
}

/* Reports r_i = (parent, ordinal, state, bytes data[off[i], off[i+1])) in any
 * order.  Outputs per parent p: counts of SUCCESS/FAILED/SKIPPED reports,
 * complete = all k_p children have a terminal report, parent_state, and the
 * slot out_data[out_off[p], out_off[p+1]) holding the SUCCESS bytes in
 * ordinal order.  out_data may be NULL (metadata only).  child_dst (NULL or
 * [N+1]) receives, for every child in canonical order, the output position
 * where its bytes start (its bytes, if any, end where the next child's
 * start; child_dst[N] = total).  barrier (NULL or [P], read and updated) is
 * the Call's group-failure barrier; n_rejected (optional) counts the reports
 * it rejected. */
int oracle_gather(const uint32_t *rep_parent, const uint32_t *rep_ordinal,
                  const uint8_t *rep_state, const int64_t *rep_off,
                  const uint8_t *data, int64_t n_reports,
                  const int64_t *offsets, int64_t n_parents,
                  int64_t *out_off, uint8_t *out_data, int64_t out_cap,
                  int32_t *n_success, int32_t *n_failed, int32_t *n_skipped,
                  uint8_t *complete, uint8_t *parent_state, int64_t *child_dst,
                  uint8_t *barrier, int64_t *n_rejected)
{
    if (n_reports < 0 || n_parents < 0 || offsets == NULL || out_off == NULL)
        return OR_EINVAL;
    if (n_reports > 0 && (rep_parent == NULL || rep_ordinal == NULL ||
                          rep_state == NULL || rep_off == NULL))
        return OR_EINVAL;
    if (n_reports > 0 && rep_off[0] < 0)
        return OR_EINVAL;
    /* 1. validate every report */
    int64_t n_valid = 0;
    for (int64_t i = 0; i < n_reports; ++i) {
        if (rep_off[i + 1] < rep_off[i])
            return OR_EINVAL;
        if (rep_state[i] > ST_GROUP_FAILED || (rep_state[i] == ST_GROUP_FAILED && barrier == NULL))
            return OR_ESTATE;
        if (rep_state[i] == ST_PENDING)
            continue;                         /* no report for this slot */
        uint32_t p = rep_parent[i];
        if ((int64_t)p >= n_parents)
            return OR_ERANGE;
        if ((int64_t)rep_ordinal[i] >= offsets[p + 1] - offsets[p])
            return OR_ERANGE;
        ++n_valid;
    }
    /* 1b. commit in report order: a report of a barred parent is rejected; a
     *     group failure commits as a failed member and bars its parent */
    uint8_t *accepted = (uint8_t *)calloc((size_t)(n_reports > 0 ? n_reports : 1), 1);
    if (!accepted)
        return OR_EINVAL;
    int64_t rejected = 0;
    for (int64_t i = 0; i < n_reports; ++i) {
        if (rep_state[i] == ST_PENDING)
            continue;
        uint32_t p = rep_parent[i];
        if (barrier != NULL && barrier[p]) {
            ++rejected;
            continue;
        }
        accepted[i] = 1;
        if (rep_state[i] == ST_GROUP_FAILED)
            barrier[p] = 1;
    }
    if (n_rejected) *n_rejected = rejected;
    /* 2. stable sort of the accepted report indices by (parent, ordinal) */
    key_t *keys = (key_t *)malloc(sizeof(key_t) * (size_t)(n_valid > 0 ? n_valid : 1));
    if (!keys) {
        free(accepted);
        return OR_EINVAL;
    }
    int64_t m = 0;
    for (int64_t i = 0; i < n_reports; ++i) {
        if (!accepted[i])
            continue;
        keys[m].parent = rep_parent[i];
        keys[m].ordinal = rep_ordinal[i];
        keys[m].index = i;
        ++m;
    }
    qsort(keys, (size_t)m, sizeof(key_t), key_cmp);
    for (int64_t j = 1; j < m; ++j) {
        if (keys[j].parent == keys[j - 1].parent && keys[j].ordinal == keys[j - 1].ordinal) {
            free(keys);
            free(accepted);
            return OR_EDUP;                   /* conflicting second fact */
        }
    }
    /* 3. total surviving bytes, checked against the output capacity */
    int64_t total = 0;
    for (int64_t j = 0; j < m; ++j) {
        int64_t i = keys[j].index;
        if (rep_state[i] == ST_SUCCESS)
            total += rep_off[i + 1] - rep_off[i];
    }
    if (out_data != NULL && total > out_cap) {
        free(keys);
        free(accepted);
        return OR_ECAP;
    }
    /* 4. per parent, ascending: counts, completion, state, and the bytes of
     *    its children in ordinal order (a child without a SUCCESS report
     *    adds none) */
    int64_t j = 0, pos = 0;
    for (int64_t p = 0; p < n_parents; ++p) {
        int32_t ns = 0, nf = 0, nk = 0;
        int64_t k = offsets[p + 1] - offsets[p];
        out_off[p] = pos;
        for (int64_t o = 0; o < k; ++o) {
            if (child_dst) child_dst[offsets[p] + o] = pos;
            if (j < m && (int64_t)keys[j].parent == p && (int64_t)keys[j].ordinal == o) {
                int64_t i = keys[j].index;
                if (rep_state[i] == ST_SUCCESS) {
                    int64_t len = rep_off[i + 1] - rep_off[i];
                    if (out_data != NULL && len > 0)
                        memcpy(out_data + pos, data + rep_off[i], (size_t)len);
                    pos += len;
                    ++ns;
                } else if (rep_state[i] == ST_FAILED || rep_state[i] == ST_GROUP_FAILED) {
                    ++nf;
                } else {
                    ++nk;
                }
                ++j;
            }
        }
        /* a barred parent's uncommitted children are suppressed: it is done */
        int barred = barrier != NULL && barrier[p];
        int done = barred || ((int64_t)ns + nf + nk == k);
        if (n_success) n_success[p] = ns;
        if (n_failed)  n_failed[p] = nf;
        if (n_skipped) n_skipped[p] = nk;
        if (complete)  complete[p] = (uint8_t)done;
        if (parent_state)
            parent_state[p] = !done ? ST_PENDING : ((barred || nf > 0) ? ST_FAILED : ST_SUCCESS);
    }
    out_off[n_parents] = pos;
    if (child_dst) child_dst[offsets[n_parents]] = pos;
    free(keys);
    free(accepted);
    return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* Streaming: reports arrive in waves; complete parents are emitted in       */
/* ascending parent order at the end of each wave, exactly once.             */
/* ------------------------------------------------------------------------ */
typedef struct {
    int64_t n_parents, n_children;
    int64_t *offsets;            /* own copy */
    uint8_t *seen;               /* per child: a terminal report was accepted */
    uint8_t *state;              /* per child */
    const uint8_t **src;         /* per child: first byte of its SUCCESS record */
    int64_t *len;                /* per child: SUCCESS record length, else 0 */
    int32_t *cnt[3];             /* per parent: SUCCESS / FAILED / SKIPPED */
    uint8_t *emitted;            /* per parent */
    uint8_t *barrier;            /* per parent: group failure seen (the stream is one Call) */
} oracle_stream;

void oracle_stream_destroy(oracle_stream *s)
{
    if (!s) return;
    free(s->offsets); free(s->seen); free(s->state); free((void *)s->src); free(s->len);
    for (int t = 0; t < 3; ++t) free(s->cnt[t]);
    free(s->emitted);
    free(s->barrier);
    free(s);
}

oracle_stream *oracle_stream_create(const int64_t *offsets, int64_t n_parents)
{
    if (n_parents < 0 || offsets == NULL)
        return NULL;
    oracle_stream *s = (oracle_stream *)calloc(1, sizeof(oracle_stream));
    if (!s) return NULL;
    int64_t n = offsets[n_parents];
    size_t np = (size_t)(n_parents + 1), nc = (size_t)(n > 0 ? n : 1);
    s->n_parents = n_parents;
    s->n_children = n;
    s->offsets = (int64_t *)malloc(sizeof(int64_t) * np);
    s->seen = (uint8_t *)calloc(nc, 1);
    s->state = (uint8_t *)calloc(nc, 1);
    s->src = (const uint8_t **)calloc(nc, sizeof(uint8_t *));
    s->len = (int64_t *)calloc(nc, sizeof(int64_t));
    for (int t = 0; t < 3; ++t) s->cnt[t] = (int32_t *)calloc(np, sizeof(int32_t));
    s->emitted = (uint8_t *)calloc(np, 1);
    s->barrier = (uint8_t *)calloc(np, 1);
    if (!s->offsets || !s->seen || !s->state || !s->src || !s->len ||
        !s->cnt[0] || !s->cnt[1] || !s->cnt[2] || !s->emitted || !s->barrier) {
        oracle_stream_destroy(s);
        return NULL;
    }
    memcpy(s->offsets, offsets, sizeof(int64_t) * np);
    return s;
}

/* The stream's group-failure barrier (read it to drop the suppressed
 * siblings of the next wave's queue). */
const uint8_t *oracle_stream_barrier(const oracle_stream *s) { return s ? s->barrier : NULL; }

/* Record one wave of reports, committed in the order given.  A child
 * reported in an earlier wave, or twice in this one, is a conflicting
 * publication.  A report of a barred parent is rejected; a GROUP_FAILED
 * report commits as a failed member and bars its parent.  The bytes stay in
 * the caller's buffer until the parent is emitted. */
int oracle_stream_report(oracle_stream *s, const uint32_t *rep_parent,
                         const uint32_t *rep_ordinal, const uint8_t *rep_state,
                         const int64_t *rep_off, const uint8_t *data, int64_t n_reports,
                         int64_t *n_rejected)
{
    if (!s || n_reports < 0)
        return OR_EINVAL;
    if (n_reports > 0 && (!rep_parent || !rep_ordinal || !rep_state || !rep_off))
        return OR_EINVAL;
    if (n_reports > 0 && rep_off[0] < 0)
        return OR_EINVAL;
    for (int64_t i = 0; i < n_reports; ++i) {      /* validate first */
        if (rep_off[i + 1] < rep_off[i]) return OR_EINVAL;
        if (rep_state[i] > ST_GROUP_FAILED) return OR_ESTATE;
        if (rep_state[i] == ST_PENDING) continue;
        uint32_t p = rep_parent[i];
        if ((int64_t)p >= s->n_parents) return OR_ERANGE;
        if ((int64_t)rep_ordinal[i] >= s->offsets[p + 1] - s->offsets[p]) return OR_ERANGE;
    }
    int64_t rejected = 0;
    for (int64_t i = 0; i < n_reports; ++i) {
        if (rep_state[i] == ST_PENDING) continue;
        uint32_t p = rep_parent[i];
        if (s->barrier[p]) {                           /* cannot commit */
            ++rejected;
            continue;
        }
        int64_t c = s->offsets[p] + rep_ordinal[i];
        if (s->seen[c])
            return OR_EDUP;
        int st = rep_state[i] == ST_GROUP_FAILED ? ST_FAILED : rep_state[i];
        s->seen[c] = 1;
        s->state[c] = (uint8_t)st;
        s->src[c] = data != NULL ? data + rep_off[i] : NULL;   /* NULL: metadata only */
        s->len[c] = st == ST_SUCCESS ? rep_off[i + 1] - rep_off[i] : 0;
        s->cnt[st][p] += 1;
        if (rep_state[i] == ST_GROUP_FAILED)
            s->barrier[p] = 1;
    }
    if (n_rejected) *n_rejected = rejected;
    return OR_OK;
}

/* Emit every parent that is complete now (or barred) and was not emitted
 * before, in ascending parent order: its id, its slot offset inside
 * emit_data, its counts, its derived state and its SUCCESS bytes in ordinal
 * order. */
int oracle_stream_emit(oracle_stream *s, uint32_t *emit_parent, int64_t *emit_off,
                       uint8_t *emit_data, int64_t cap_parents, int64_t cap_bytes,
                       int32_t *n_success, int32_t *n_failed, int32_t *n_skipped,
                       uint8_t *parent_state, int64_t *n_emitted, int64_t *n_bytes)
{
    if (!s || !emit_off)
        return OR_EINVAL;
    int64_t e = 0, pos = 0;
    /* first pass: sizes, checked against the capacities */
    for (int64_t p = 0; p < s->n_parents; ++p) {
        int64_t k = s->offsets[p + 1] - s->offsets[p];
        if (s->emitted[p] || (!s->barrier[p] && (int64_t)s->cnt[0][p] + s->cnt[1][p] + s->cnt[2][p] != k))
            continue;
        ++e;
        for (int64_t c = s->offsets[p]; c < s->offsets[p + 1]; ++c)
            pos += s->len[c];
    }
    if (e > cap_parents || (emit_data != NULL && pos > cap_bytes))
        return OR_ECAP;
    e = 0;
    pos = 0;
    for (int64_t p = 0; p < s->n_parents; ++p) {
        int64_t k = s->offsets[p + 1] - s->offsets[p];
        if (s->emitted[p] || (!s->barrier[p] && (int64_t)s->cnt[0][p] + s->cnt[1][p] + s->cnt[2][p] != k))
            continue;
        if (emit_parent) emit_parent[e] = (uint32_t)p;
        emit_off[e] = pos;
        for (int64_t c = s->offsets[p]; c < s->offsets[p + 1]; ++c) {
            if (emit_data != NULL && s->len[c] > 0)
                memcpy(emit_data + pos, s->src[c], (size_t)s->len[c]);
            pos += s->len[c];
        }
        if (n_success) n_success[e] = s->cnt[0][p];
        if (n_failed)  n_failed[e] = s->cnt[1][p];
        if (n_skipped) n_skipped[e] = s->cnt[2][p];
        if (parent_state) parent_state[e] = (s->barrier[p] || s->cnt[1][p] > 0) ? ST_FAILED : ST_SUCCESS;
        s->emitted[p] = 1;
        ++e;
    }
    emit_off[e] = pos;
    if (n_emitted) *n_emitted = e;
    if (n_bytes) *n_bytes = pos;
    return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* F.filter and F.broadcast, with the input propagation rule.                */
/* ------------------------------------------------------------------------ */
/* Sec. 4, input propagation: a failed or suppressed input suppresses the
 * output; otherwise an unresolved input makes it wait; otherwise a dropped
 * required input drops it; otherwise the output is ready.  In states:
 * FAILED before PENDING before SKIPPED before SUCCESS. */
static int propagate(int a, int b)
{
    if (a == ST_FAILED || b == ST_FAILED) return ST_FAILED;
    if (a == ST_PENDING || b == ST_PENDING) return ST_PENDING;
    if (a == ST_SKIPPED || b == ST_SKIPPED) return ST_SKIPPED;
    return ST_SUCCESS;
}

/* F.filter(x, mask) (Table "primitives"): same Domain; the output passes x
 * when the mask is true and is dropped when it is false, after the
 * propagation rule over both inputs.  mask_state may be NULL (mask present). */
int oracle_filter(const uint8_t *x_state, const uint8_t *mask_state, const uint8_t *mask, int64_t n,
                  uint8_t *out_state)
{
    if (n < 0 || (n > 0 && (!x_state || !mask || !out_state)))
        return OR_EINVAL;
    for (int64_t i = 0; i < n; ++i) {
        int ms = mask_state ? mask_state[i] : ST_SUCCESS;
        if (x_state[i] > ST_PENDING || ms > ST_PENDING)
            return OR_ESTATE;
        int s = propagate(x_state[i], ms);
        if (s == ST_SUCCESS && mask[i] == 0)
            s = ST_SKIPPED;
        out_state[i] = (uint8_t)s;
    }
    return OR_OK;
}

/* F.broadcast(x, like=y) (Table "primitives"): ancestor x made available in
 * y's Domain.  maps[0] takes a descendant to its parent, maps[1] that parent
 * to its own parent, and so on for `levels` levels; the last index is the
 * ancestor.  The output state follows the propagation rule over x at the
 * ancestor and y (like_state, NULL = present). */
int oracle_broadcast(const uint32_t *const *maps, int32_t levels, int64_t n, const uint8_t *x_state,
                     int64_t n_ancestors, const uint8_t *like_state, uint32_t *out_ancestor,
                     uint8_t *out_state)
{
    if (n < 0 || levels < 1 || (n > 0 && (!maps || !x_state || !out_ancestor || !out_state)))
        return OR_EINVAL;
    for (int64_t d = 0; d < n; ++d) {
        uint32_t a = (uint32_t)d;
        for (int32_t l = 0; l < levels; ++l)
            a = maps[l][a];
        if ((int64_t)a >= n_ancestors)
            return OR_ERANGE;
        int ls = like_state ? like_state[d] : ST_SUCCESS;
        if (x_state[a] > ST_PENDING || ls > ST_PENDING)
            return OR_ESTATE;
        out_ancestor[d] = a;
        out_state[d] = (uint8_t)propagate(x_state[a], ls);
    }
    return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* Grain phases and the generation fence.                                    */
/* ------------------------------------------------------------------------ */
/* Sec. 4, Eq. (grain-phase): WAITING -> READY -> IN-FLIGHT -> SEALED, and a
 * retry takes IN-FLIGHT back to READY; Eq. (generation-fence): a report
 * commits only if its Grain is in flight and the report's generation is the
 * Grain's current one; publication rules: a repeat of a committed fact is
 * idempotent, a conflicting one is rejected.  One Grain per child of an
 * expansion, all READY at generation 0 to start with. */
enum { PH_WAITING = 0, PH_READY = 1, PH_IN_FLIGHT = 2, PH_SEALED = 3 };

typedef struct {
    int64_t n;
    uint8_t *phase;
    uint32_t *gen;
    int64_t *winner;             /* per child: report index accepted in the current commit call, or -1 */
} oracle_grains;

void oracle_grains_destroy(oracle_grains *g)
{
    if (!g) return;
    free(g->phase); free(g->gen); free(g->winner);
    free(g);
}

oracle_grains *oracle_grains_create(int64_t n)
{
    if (n < 0) return NULL;
    oracle_grains *g = (oracle_grains *)calloc(1, sizeof(oracle_grains));
    if (!g) return NULL;
    size_t m = (size_t)(n > 0 ? n : 1);
    g->n = n;
    g->phase = (uint8_t *)malloc(m);
    g->gen = (uint32_t *)calloc(m, sizeof(uint32_t));
    g->winner = (int64_t *)malloc(m * sizeof(int64_t));
    if (!g->phase || !g->gen || !g->winner) { oracle_grains_destroy(g); return NULL; }
    for (int64_t c = 0; c < n; ++c) { g->phase[c] = PH_READY; g->winner[c] = -1; }
    return g;
}

const uint8_t *oracle_grains_phase(const oracle_grains *g) { return g ? g->phase : NULL; }
const uint32_t *oracle_grains_gen(const oracle_grains *g) { return g ? g->gen : NULL; }

/* Reserve: READY -> IN-FLIGHT; out_gen[i] = the generation the attempt runs
 * at.  A child that is not READY is a bad state. */
int oracle_grains_dispatch(oracle_grains *g, const uint32_t *child, int64_t n, uint32_t *out_gen)
{
    if (!g || n < 0 || (n > 0 && !child)) return OR_EINVAL;
    for (int64_t i = 0; i < n; ++i) {
        uint32_t c = child[i];
        if ((int64_t)c >= g->n) return OR_ERANGE;
        if (g->phase[c] != PH_READY) return OR_ESTATE;
        g->phase[c] = PH_IN_FLIGHT;
        if (out_gen) out_gen[i] = g->gen[c];
    }
    return OR_OK;
}

/* Retry: IN-FLIGHT -> READY at the next generation. */
int oracle_grains_retry(oracle_grains *g, const uint32_t *child, int64_t n)
{
    if (!g || n < 0 || (n > 0 && !child)) return OR_EINVAL;
    for (int64_t i = 0; i < n; ++i) {
        uint32_t c = child[i];
        if ((int64_t)c >= g->n) return OR_ERANGE;
        if (g->phase[c] != PH_IN_FLIGHT) return OR_ESTATE;
        g->phase[c] = PH_READY;
        g->gen[c] += 1;
    }
    return OR_OK;
}

/* Commit one call's reports in order.  The first report of an in-flight
 * Grain at its current generation is accepted and seals it; a later report
 * of the same call at that generation repeats the accepted one: a duplicate
 * if its state and bytes are the same, a conflict otherwise; any other
 * report is stale.  state_out[i] is the report's state if accepted, PENDING
 * otherwise (so a gather ignores it).  counts[0..3] = accepted, stale,
 * duplicate, conflict. */
int oracle_grains_commit(oracle_grains *g, const uint32_t *rep_parent, const uint32_t *rep_ordinal,
                         const uint8_t *rep_state, const int64_t *rep_off, const uint8_t *data,
                         const uint32_t *rep_gen, int64_t n, const int64_t *offsets, int64_t n_parents,
                         uint8_t *state_out, int64_t *counts)
{
    if (!g || n < 0 || !offsets || (n > 0 && (!rep_parent || !rep_ordinal || !rep_state || !rep_off || !rep_gen ||
                                              !state_out)))
        return OR_EINVAL;
    for (int64_t i = 0; i < n; ++i) {
        if (rep_off[i + 1] < rep_off[i]) return OR_EINVAL;
        if (rep_state[i] > ST_GROUP_FAILED) return OR_ESTATE;
        if (rep_state[i] == ST_PENDING) continue;
        uint32_t p = rep_parent[i];
        if ((int64_t)p >= n_parents) return OR_ERANGE;
        if ((int64_t)rep_ordinal[i] >= offsets[p + 1] - offsets[p]) return OR_ERANGE;
        if (offsets[p] + rep_ordinal[i] >= g->n) return OR_ERANGE;
    }
    int64_t acc = 0, stale = 0, dup = 0, conf = 0;
    for (int64_t i = 0; i < n; ++i) {
        state_out[i] = ST_PENDING;
        if (rep_state[i] == ST_PENDING) continue;
        int64_t c = offsets[rep_parent[i]] + rep_ordinal[i];
        if (g->phase[c] == PH_IN_FLIGHT && rep_gen[i] == g->gen[c]) {
            g->phase[c] = PH_SEALED;
            g->winner[c] = i;
            state_out[i] = rep_state[i];
            ++acc;
        } else if (g->winner[c] >= 0 && rep_gen[i] == g->gen[c]) {
            int64_t w = g->winner[c];
            int same = rep_state[w] == rep_state[i];
            if (same && rep_state[i] == ST_SUCCESS) {
                int64_t lw = rep_off[w + 1] - rep_off[w], li = rep_off[i + 1] - rep_off[i];
                same = lw == li && (lw == 0 || data == NULL ||
                                    memcmp(data + rep_off[w], data + rep_off[i], (size_t)lw) == 0);
            }
            if (same) ++dup; else ++conf;
        } else {
            ++stale;
        }
    }
    for (int64_t i = 0; i < n; ++i)          /* winners are per call */
        if (rep_state[i] != ST_PENDING) g->winner[offsets[rep_parent[i]] + rep_ordinal[i]] = -1;
    if (counts) { counts[0] = acc; counts[1] = stale; counts[2] = dup; counts[3] = conf; }
    return OR_OK;
}
