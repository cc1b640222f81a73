/*
 * ro.h -- C ABI of the lineage-controlled expand / batch / gather core for
 * AMD Instinct MI355X (gfx950).
 *
 * The operations follow RayOrch (arXiv 2609.18703):
 *   - ro_expand  : F.expand (Table "primitives"; Sec. 4 "Lineage State and
 *                  Parent Completion"): one Expansion per parent, an ordered
 *                  child set whose members carry (parent, immutable ordinal).
 *   - ro_batch   : per-Call FIFO Ready Queue with elastic reservation
 *                  (Sec. 4 "Scheduling Ready Grains"): at most B entries
 *                  leave the head of the queue per reservation, parents may mix.
 *   - ro_gather  : F.reduce and the Reduce rule (Sec. 4): a parent resolves
 *                  once every member is terminal; dropped members are
 *                  excluded, failed members suppress the parent, present
 *                  values are concatenated in ordinal order, zero survivors
 *                  give an empty list.  Conflicting second reports are
 *                  rejected (publication rules, same section).
 *   - ro_stream_*: the same gather fed wave by wave; a parent is emitted as
 *                  soon as all of its children are terminal (Sec. 1 and 4:
 *                  completed parents proceed while others still produce),
 *                  in ascending parent order, exactly once.
 *   - ro_batch_parent: parent-bound reservation (Sec. 4 "Scheduling Ready
 *                  Grains"): up to B siblings of the first ready parent.
 *   - ro_filter, ro_broadcast: F.filter and F.broadcast (Table
 *                  "primitives") under the input propagation precedence.
 *   - ro_grains_*: Grain phases and the generation fence (Sec. 4, Eq.
 *                  grain-phase and Eq. generation-fence).
 *
 * Conventions shared by every entry point:
 *   * Memory.  Every array argument is DEVICE memory owned by the caller
 *     (e.g. a torch tensor's data pointer).  The library keeps no caller
 *     pointer past the call, except a stream's offsets and the report bytes of
 *     parents not yet emitted (see ro_stream_report).
 *   * Ordering.  Every call enqueues its kernels on the context's HIP stream
 *     and returns at once.  Nothing synchronises except ro_ctx_status, the
 *     create/destroy calls, and a call that has to grow a workspace
 *     (hipMalloc): ro_ctx_reserve, a gather or batch beyond the reservation,
 *     the first ro_batch_parent of a larger queue, the first
 *     ro_grains_commit of a larger call.  Outputs are ready once the
 *     context's stream has drained: read them with work ordered after it
 *     (a copy on the same stream, or after ro_ctx_status or a stream
 *     synchronisation); a copy on another stream, including the null stream
 *     when the context's stream is non-blocking, is not ordered with it.
 *   * Errors.  Errors found on the host (NULL where an array is required, a
 *     negative size, batch_size <= 0, a failing HIP call) are returned
 *     immediately and nothing is enqueued.  Errors that depend on device data
 *     are written to the context's error word, first error wins, and are
 *     returned (and cleared) by ro_ctx_status.  After any error the outputs of
 *     that call are unspecified; a gather or stream emission that follows a
 *     recorded error copies no bytes until the error is cleared.
 *   * Sizes.  Child ids are uint32, so an expansion may hold at most
 *     2^32 - 1 children (RO_EOVERFLOW otherwise).  Byte offsets are int64;
 *     one record may hold at most 2^32 - 1 bytes (a slot keeps its length in
 *     32 bits; a longer SUCCESS record is RO_EOVERFLOW).
 *   * Terminal states are uint8: RO_SUCCESS (Present), RO_FAILED (Failed, or
 *     Suppressed handed up from a lower level), RO_SKIPPED (Dropped) and
 *     RO_PENDING (no report yet).  A report may also carry RO_GROUP_FAILED,
 *     a typed group failure (Sec. 4 "Commit, Failure, and Recovery"): it
 *     commits as a failed member and bars its parent for the rest of the
 *     Call.  Barriers live in a caller-owned uint8 array per Call, one byte
 *     per parent; reports commit in the order given, call after call, so a
 *     later report of a barred parent is rejected (not committed, not
 *     counted, its bytes never copied), reports committed earlier stay, and
 *     ro_batch drops the barred parent's queued children before dispatch.
 *     A barred parent is complete and RO_FAILED.  RO_GROUP_FAILED without a
 *     barrier array is RO_ESTATE.
 *
 * A context is bound to one stream and is not thread safe.
 */
#ifndef RO_H
#define RO_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    RO_OK = 0,
    RO_EINVAL = -1,     /* bad argument, negative count, decreasing byte offsets      */
    RO_ERANGE = -2,     /* parent >= P, ordinal >= k_p, or queued child id >= N        */
    RO_EDUP = -3,       /* a child reported twice (within a call or across waves)      */
    RO_ECAP = -4,       /* an output or the reserved workspace is too small            */
    RO_EOVERFLOW = -5,  /* N >= 2^32 children, a record of 2^32 bytes or more, or
                           byte totals beyond 2^45                                     */
    RO_ESTATE = -6,     /* a state byte > RO_PENDING (RO_GROUP_FAILED is valid only
                           where a barrier array is given), or a Grain not in the
                           phase an operation needs                                    */
    RO_EHIP = -7        /* a HIP runtime call failed                                   */
};

enum { RO_SUCCESS = 0, RO_FAILED = 1, RO_SKIPPED = 2, RO_PENDING = 3, RO_GROUP_FAILED = 4 };

typedef struct ro_ctx ro_ctx;

/* Create a context on the current HIP device, bound to `hip_stream`
 * (a hipStream_t; NULL means the null stream).  Returns RO_OK or RO_EHIP. */
int ro_ctx_create(ro_ctx **out, void *hip_stream);

/* Re-bind the context to another stream of the same device. */
int ro_ctx_set_stream(ro_ctx *ctx, void *hip_stream);

/* Pre-size the device workspace for expansions of up to `max_children`
 * children and `max_parents` parents, and queues of up to `max_queue`
 * entries, so that later expand / batch / gather / stream calls never
 * allocate (ro_batch_parent and the Grain commit keep workspaces of their
 * own, sized on first use).  Calls whose host-known sizes
 * (parents, queue length, report count) exceed the reservation grow it
 * (hipMalloc, which synchronises).  An expansion whose child count, known
 * only on the device, exceeds the reservation fails with RO_ECAP. */
int ro_ctx_reserve(ro_ctx *ctx, int64_t max_children, int64_t max_parents, int64_t max_queue);

/* Wait for the context's stream, then return and clear the first error the
 * device recorded (RO_OK if none). */
int ro_ctx_status(ro_ctx *ctx);

/* Free the context's workspace.  Waits for its stream first.  Destroy the
 * context's Grain sets and streams before the context: their destroy calls
 * wait on its stream. */
int ro_ctx_destroy(ro_ctx *ctx);

/* Per-kernel timing (measurement aid).  While enabled, every kernel the
 * context launches is bracketed by two HIP events on the context's stream.
 * ro_ctx_trace_read waits for the stream, adds up the elapsed time per
 * kernel kind since the last read into launches[k] / total_ms[k] for
 * k < n (indices below), and clears the record.  RO_K_GATHER_RESET is no
 * longer launched (a gather clears its counters in its finalize kernel); it
 * keeps its place so that the indices after it do not change. */
enum {
    RO_K_EXPAND_SCAN = 0, RO_K_EXPAND_TAGS, RO_K_BATCH_SAMPLES, RO_K_BATCH,
    RO_K_GATHER_SCATTER, RO_K_GATHER_SCAN, RO_K_GATHER_FINALIZE, RO_K_GATHER_COPY,
    RO_K_GATHER_RESET, RO_K_STREAM_REPORT, RO_K_STREAM_SELECT, RO_K_STREAM_SCAN,
    RO_K_STREAM_COPY, RO_K_STREAM_FINISH, RO_K_MISC, RO_K_FILTER, RO_K_BROADCAST,
    RO_K_GRAINS, RO_K_FENCE_FIRST, RO_K_FENCE_DECIDE, RO_K_PBATCH_SORT, RO_K_PBATCH, RO_K_COUNT
};
int ro_ctx_trace(ro_ctx *ctx, int enable);
int ro_ctx_trace_read(ro_ctx *ctx, int64_t *launches, double *total_ms, int32_t n);

/* F.expand.  counts[P] (int32, >= 0) -> offsets[P+1] (int64 exclusive scan,
 * offsets[P] = N): parent p's ordered children are the canonical ids
 * [offsets[p], offsets[p+1]).  If child_parent / child_ordinal are not NULL,
 * child c also gets its key (p, c - offsets[p]); both need room for N
 * entries, N <= child_cap (RO_ECAP otherwise).  A negative count is
 * RO_EINVAL; N >= 2^32 is RO_EOVERFLOW. */
int ro_expand(ro_ctx *ctx, const int32_t *counts, int64_t n_parents, int64_t *offsets,
              uint32_t *child_parent, uint32_t *child_ordinal, int64_t child_cap);

/* ro_expand for callers that cannot allocate device memory: code under
 * stream capture, tight serving loops, harnesses that forbid hipMalloc.  It
 * takes no context and calls no allocating routine: the scan's workspace
 * (control words and look-back descriptors, about 33 KB) is one fixed
 * device array per GPU, set up on the first call on that GPU (the calling
 * thread's current device) and held until the process ends.  Same inputs,
 * outputs and results as ro_expand, on the HIP stream hip_stream (NULL = the
 * null stream).  At most 2^24 parents: larger n_parents returns RO_ECAP at
 * once.  Host-detectable errors return at once (RO_EINVAL); the
 * device-detected status (RO_OK, or RO_EINVAL / RO_ECAP / RO_EOVERFLOW as
 * for ro_expand) is written, stream-ordered, to the device int32
 * *status_dev at the end of the call (status_dev may be NULL).  Every call
 * on one GPU shares that GPU's workspace: calls that overlap on one GPU (on
 * different streams or host threads) race and must not be issued. */
int ro_expand_noalloc(void *hip_stream, const int32_t *counts, int64_t n_parents, int64_t *offsets,
                      uint32_t *child_parent, uint32_t *child_ordinal, int64_t child_cap, int32_t *status_dev);

/* FIFO Ready Queue + elastic reservation.  queue[q_len] holds canonical
 * child ids in enqueue order; entry i is ready iff keep == NULL or
 * keep[i] != 0.  Ready entries are compacted in queue order into slots
 * [0, M); reservation j is slots [j*B, min((j+1)*B, M)).  Each slot gets the
 * child id (out_child), its parent (out_parent) and its ordinal
 * (out_ordinal); any of the three may be NULL.  M must be <= out_cap
 * (RO_ECAP).  A ready id >= N (N = offsets[n_parents]) is RO_ERANGE.  M and
 * ceil(M/B) are written to the device scalars *n_out_dev and *n_batches_dev
 * (either may be NULL).  With a group-failure barrier ([n_parents], may be
 * NULL), an entry whose parent is barred is not ready: it is suppressed
 * before dispatch and takes no slot.  The tag arrays (out_cap entries each)
 * must not share memory with the queue, the mask, the offsets, the barrier
 * or one another (RO_EINVAL, checked on the host). */
int ro_batch(ro_ctx *ctx, const uint32_t *queue, const uint8_t *keep, int64_t q_len,
             const int64_t *offsets, int64_t n_parents, int32_t batch_size,
             uint32_t *out_child, uint32_t *out_parent, uint32_t *out_ordinal, int64_t out_cap,
             int64_t *n_out_dev, int64_t *n_batches_dev, const uint8_t *barrier);

/* FIFO Ready Queue + parent-bound reservation (Sec. 4 "Scheduling Ready
 * Grains"): each reservation takes up to B siblings of the first ready
 * parent, the parent of the earliest entry still queued, and every other
 * entry keeps its place.  Ready entries, ids, tags, barrier and errors as in
 * ro_batch (batch_off, too, may share no memory with the inputs or tag
 * arrays); reservations run until the queue is empty.  Reservation j is
 * slots [batch_off[j], batch_off[j+1]) (int64, device; batch_off[n_batches]
 * = M), so it needs n_batches + 1 <= batch_cap (RO_ECAP; n_batches <= M).
 * M and n_batches go to *n_out_dev and *n_batches_dev (either may be
 * NULL).  Workspace: about 36 bytes per queue entry and 8 per parent, held
 * by the context and grown on demand. */
int ro_batch_parent(ro_ctx *ctx, const uint32_t *queue, const uint8_t *keep, int64_t q_len,
                    const int64_t *offsets, int64_t n_parents, int32_t batch_size, uint32_t *out_child,
                    uint32_t *out_parent, uint32_t *out_ordinal, int64_t out_cap, int64_t *batch_off,
                    int64_t batch_cap, int64_t *n_out_dev, int64_t *n_batches_dev, const uint8_t *barrier);

/* One terminal report per child, in any order.  Report i is the child
 * (parent[i], ordinal[i]) with state[i]; its value is the byte range
 * data[off[i], off[i+1]) (Arrow-style offsets, off nondecreasing, off[0]
 * >= 0, RO_EINVAL otherwise).  Only RO_SUCCESS bytes are ever read.  A
 * report with state RO_PENDING is ignored. */
typedef struct ro_reports {
    const uint32_t *parent;
    const uint32_t *ordinal;
    const uint8_t *state;
    const int64_t *off;       /* [n + 1] */
    const uint8_t *data;
    int64_t n;
} ro_reports;

/* Per-parent outputs of a gather ([P] arrays unless noted). */
typedef struct ro_gather_out {
    int64_t *out_off;         /* [P + 1] slot p = out_data[out_off[p], out_off[p+1])   */
    uint8_t *out_data;        /* the packed slots; needs out_off[P] <= out_cap bytes    */
    int64_t out_cap;
    int32_t *n_success;       /* reports per state (may be NULL)                         */
    int32_t *n_failed;
    int32_t *n_skipped;
    uint8_t *complete;        /* 1 iff all k_p children have a terminal report (NULL ok) */
    uint8_t *parent_state;    /* RO_PENDING if incomplete, else RO_FAILED if any member
                                 failed, else RO_SUCCESS (NULL ok)                        */
    int64_t *child_dst_off;   /* [N + 1] or NULL: output position of every child in
                                 canonical order; child c's bytes (none unless it has a
                                 SUCCESS report) are [child_dst_off[c],
                                 child_dst_off[c+1]), child_dst_off[N] = out_off[P]     */
    uint8_t *barrier;         /* [P] or NULL: the Call's group-failure barrier, read and
                                 updated (a parent barred by this call's reports is set) */
    int64_t *n_rejected;      /* device scalar or NULL: reports rejected by a barrier    */
} ro_gather_out;

/* F.reduce: ordered gather of reports into parent slots.  Slot p holds the
 * bytes of parent p's RO_SUCCESS reports in ordinal order; an incomplete
 * parent's slot holds the ones received so far; a parent with a failed
 * member keeps its surviving bytes and is flagged RO_FAILED; a parent with
 * no children is complete and RO_SUCCESS with an empty slot.  Errors:
 * RO_ERANGE, RO_ESTATE, RO_EINVAL (offsets), RO_EDUP (two reports for one
 * child), RO_ECAP (bytes > out_cap, or N above the reservation).
 * out_data must not overlap the report bytes, with one exception: it may be
 * the reports' own data pointer when every copied record already sits at
 * its output position, as in the upper level of a nested gather whose lower
 * slots all survive (Sec. 4: a parent's value is its members' values in
 * order, so the lower slots already are the upper ones).  Nothing is then
 * copied; a record that would have to move is RO_EINVAL. */
int ro_gather(ro_ctx *ctx, const ro_reports *reports, const int64_t *offsets, int64_t n_parents,
              const ro_gather_out *out);

/* F.filter (Table "primitives"; Sec. 4 input propagation): for n Items of
 * one Domain, out_state[i] derives from x_state[i] and the mask's state
 * mask_state[i] (NULL = all present) by the propagation precedence (a
 * FAILED input gives FAILED, else a PENDING one PENDING, else a SKIPPED one
 * SKIPPED, else SUCCESS); a SUCCESS output whose mask[i] is 0 is dropped
 * (SKIPPED).  The value of a passing Item is x's own record, so no bytes
 * move.  A state above RO_PENDING is RO_ESTATE. */
int ro_filter(ro_ctx *ctx, const uint8_t *x_state, const uint8_t *mask_state, const uint8_t *mask, int64_t n,
              uint8_t *out_state);

/* F.broadcast (Table "primitives"): make the ancestor Item x available in
 * a descendant Domain of n Items.  maps[0] is the descendant level's
 * child -> parent array (as ro_expand's child_parent), maps[1] the level
 * above, ..., `levels` arrays in all (1..8); the last index reached is the
 * ancestor (out_ancestor[d], may be NULL).  map_len[l] is the number of
 * entries of maps[l] (map_len[0] >= n, RO_EINVAL otherwise); an index that
 * falls outside the next map, or an ancestor >= n_ancestors, is RO_ERANGE
 * (checked before it is used).  out_state[d] combines x_state[ancestor]
 * with like_state[d] (the descendant's own state, NULL = present) by the
 * same precedence as ro_filter.  `maps` and `map_len` are host arrays; the
 * maps themselves are in device memory. */
int ro_broadcast(ro_ctx *ctx, const uint32_t *const *maps, const int64_t *map_len, int32_t levels, int64_t n,
                 const uint8_t *x_state, int64_t n_ancestors, const uint8_t *like_state, uint32_t *out_ancestor,
                 uint8_t *out_state);

/* Grain phases and the generation fence (Sec. 4, Eq. grain-phase and Eq.
 * generation-fence).  One Grain per child of an expansion: READY at
 * generation 0 when created or reset; reservation moves it to IN-FLIGHT, a
 * retry back to READY at the next generation, an accepted report seals it.
 * The state lives in device memory allocated here (16 bytes per child). */
enum { RO_WAITING = 0, RO_READY = 1, RO_IN_FLIGHT = 2, RO_SEALED = 3 };
typedef struct ro_grains ro_grains;
int ro_grains_create(ro_ctx *ctx, int64_t n_children, ro_grains **out);
int ro_grains_reset(ro_ctx *ctx, ro_grains *g);
/* Waits for the owning context's stream, then frees the Grain state (the
 * context must still exist). */
int ro_grains_destroy(ro_grains *g);

/* Write every child's phase (RO_READY, RO_IN_FLIGHT or RO_SEALED) and
 * generation into the device arrays phase[n_children] and
 * generation[n_children] (uint32; either may be NULL), on the context's
 * stream.  For inspection: the library keeps its own layout. */
int ro_grains_read(ro_ctx *ctx, ro_grains *g, uint32_t *phase, uint32_t *generation);

/* Reserve child[0..n): READY -> IN-FLIGHT; out_generation[i] (may be NULL)
 * is the generation the attempt runs at, which its report must carry.  A
 * child that is not READY (or named twice) is RO_ESTATE. */
int ro_grains_dispatch(ro_ctx *ctx, ro_grains *g, const uint32_t *child, int64_t n, uint32_t *out_generation);

/* Retry child[0..n): IN-FLIGHT -> READY at the next generation (a lost or
 * failed physical attempt; Grain identity is unchanged).  A child not in
 * flight is RO_ESTATE. */
int ro_grains_retry(ro_ctx *ctx, ro_grains *g, const uint32_t *child, int64_t n);

/* Commit one call's reports through the fence, in report order: the first
 * report of an in-flight Grain at its current generation (generation[i]) is
 * accepted and seals the Grain; a later report of this call at that
 * generation repeats it and is a duplicate (same state and bytes, dropped as
 * idempotent) or a conflict (rejected); every other report is stale.
 * state_out[i] is the report's state if accepted and RO_PENDING otherwise,
 * so a following ro_gather / ro_stream_report with these states commits
 * exactly the accepted reports.  counts_dev[0..3] (device, may be NULL) =
 * accepted, stale, duplicate, conflict.  Validation as in ro_gather. */
int ro_grains_commit(ro_ctx *ctx, ro_grains *g, const ro_reports *reports, const uint32_t *generation,
                     const int64_t *offsets, int64_t n_parents, uint8_t *state_out, int64_t *counts_dev);

/* Streaming gather over one expansion (offsets[P+1] on the device, kept by
 * reference until ro_stream_destroy).  The stream's own state lives in
 * device memory allocated here (about 36 bytes per child and 42 per parent).
 * A stream is one Call: `barrier` ([P], zeroed by the caller, may be NULL)
 * is its group-failure barrier, kept by reference; pass the same array to
 * ro_batch for each wave so that barred parents' queued children are
 * dropped. */
typedef struct ro_stream ro_stream;
int ro_stream_create(ro_ctx *ctx, const int64_t *offsets, int64_t n_parents, int64_t n_children,
                     uint8_t *barrier, ro_stream **out);

/* ro_batch for one wave of the stream's Call: the same compaction, tags and
 * errors, over the stream's expansion and with its barrier, but every
 * entry's parent comes from a child -> parent map the stream built when it
 * was created (one load instead of a search of the offsets). */
int ro_stream_batch(ro_ctx *ctx, ro_stream *s, const uint32_t *queue, const uint8_t *keep, int64_t q_len,
                    int32_t batch_size, uint32_t *out_child, uint32_t *out_parent, uint32_t *out_ordinal,
                    int64_t out_cap, int64_t *n_out_dev, int64_t *n_batches_dev);

/* Record one wave of reports (same validation as ro_gather; a child already
 * reported in an earlier wave is RO_EDUP).  Reports commit in the order
 * given, after every earlier wave: one of a barred parent is rejected and
 * added to *n_rejected_dev (device scalar, may be NULL).  The report bytes
 * are read when their parent is emitted, so `data` must stay valid until
 * then. */
int ro_stream_report(ro_ctx *ctx, ro_stream *s, const ro_reports *wave, int64_t *n_rejected_dev);

/* Emit every parent that is complete now (a barred parent is complete) and
 * was not emitted before, in ascending parent order: emit_parent[e], its slot
 * emit_data[emit_off[e], emit_off[e+1]), its counts and its state.  Needs
 * room for cap_parents parents (emit_off: cap_parents + 1) and cap_bytes
 * bytes (RO_ECAP).  The number of parents and bytes go to the device
 * scalars *n_emitted_dev / *n_bytes_dev (either may be NULL).  Parents
 * without children are emitted by the first call. */
int ro_stream_emit(ro_ctx *ctx, ro_stream *s, uint32_t *emit_parent, int64_t *emit_off,
                   uint8_t *emit_data, int64_t cap_parents, int64_t cap_bytes,
                   int32_t *n_success, int32_t *n_failed, int32_t *n_skipped,
                   uint8_t *parent_state, int64_t *n_emitted_dev, int64_t *n_bytes_dev);

/* Start the stream over for a new run on the same expansion (same offsets
 * buffer, same P and N; the offsets may be rewritten in between): every
 * report, count, emission and barrier is forgotten, the allocation is kept.
 * Stream-ordered like the other calls, allocates nothing and enqueues no
 * memset node.  A new Call over a parent batch of the same shape (Sec. 4,
 * per-Call queue) then reuses the state instead of creating it again.
 * RO_EINVAL if s belongs to another context. */
int ro_stream_reset(ro_ctx *ctx, ro_stream *s);

/* Waits for the owning context's stream, then frees the stream state (the
 * context must still exist). */
int ro_stream_destroy(ro_stream *s);

#ifdef __cplusplus
}
#endif

#endif /* RO_H */
