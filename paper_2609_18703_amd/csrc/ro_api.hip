// Host side of the C ABI: contexts, workspace, argument checks, launches.
#include <stdlib.h>
#include <string.h>

#include <vector>

#include "ro_internal.h"
#include "ro_testing.h"

using namespace ro;

namespace ro {

// Events bracketing every traced launch; recycled after each read.
struct Tracer {
    struct Rec {
        int kind;
        hipEvent_t e0, e1;
    };
    bool on = false;
    std::vector<hipEvent_t> pool;   // all events ever created
    size_t used = 0;                // events handed out since the last read
    std::vector<Rec> recs;
    hipEvent_t next_event()
    {
        if (used == pool.size()) {
            hipEvent_t e = nullptr;
            if (hipEventCreate(&e) != hipSuccess) return nullptr;
            pool.push_back(e);
        }
        return pool[used++];
    }
};

void trace_begin(const Launch &L, int kernel)
{
    Tracer *t = L.tracer;
    if (!t || !t->on) return;
    hipEvent_t e = t->next_event();
    if (e && hipEventRecord(e, L.stream) != hipSuccess) e = nullptr;
    t->recs.push_back({kernel, e, nullptr});
}

void trace_end(const Launch &L, int kernel)
{
    (void)kernel;
    Tracer *t = L.tracer;
    if (!t || !t->on || t->recs.empty()) return;
    hipEvent_t e = t->next_event();
    if (e && hipEventRecord(e, L.stream) != hipSuccess) e = nullptr;
    t->recs.back().e1 = e;
}

}  // namespace ro

struct ro_ctx {
    hipStream_t stream;
    int device;
    int num_cus;
    Ctl *ctl;
    uint64_t *desc;
    int64_t desc_cap;
    Canon *canon;
    int64_t canon_cap;
    int64_t *sub_base;
    int64_t sub_cap;
    uint32_t *cmap;           // coarse child -> parent map used by ro_batch
    int64_t cmap_cap;
    int32_t *cnt;             // [3 * cnt_cap] counters used when the caller passes none
    uint64_t *gkey;           // [cnt_cap] first group failure per parent (gather)
    int64_t cnt_cap;
    int64_t gathers;          // canonical epoch of the next gather (1..2^30-1)
    PbWs pb;                  // parent-bound reservation workspace
    int64_t pb_cap, pb_pcap;  // its queue entries and parents
    void *pb_block;
    Tracer *tracer;
};

struct ro_grains {
    ro_ctx *ctx;
    int64_t n;
    Grain *g;                 // [max(n, 1)] phase, generation and fence key per child
    uint32_t epoch;           // of the current commit call
    uint32_t *tag;            // [tag_cap] per report: epoch of the call in which it met another
    int64_t tag_cap;
};

struct ro_stream {
    ro_ctx *ctx;
    StreamState st;
    void *block;              // one device allocation for all stream state
};

namespace {

int hip_fail(hipError_t e) { return e == hipSuccess ? RO_OK : RO_EHIP; }

// Byte ranges [a, a + na) and [b, b + nb) share a byte (NULL or empty: never).
bool overlap(const void *a, int64_t na, const void *b, int64_t nb)
{
    if (!a || !b || na <= 0 || nb <= 0) return false;
    const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
    return x < y + (uintptr_t)nb && y < x + (uintptr_t)na;
}

// The batch kernels read the queue, mask, offsets and barrier and write the
// tag arrays through restrict-qualified pointers: a tag array that shares
// memory with any of those, or with another tag array, is rejected.
bool batch_outputs_alias(const uint32_t *queue, const uint8_t *keep, int64_t q_len, const int64_t *offsets,
                         int64_t P, const uint8_t *barrier, uint32_t *const outs[3], int64_t out_cap,
                         const void *extra, int64_t extra_bytes)
{
    for (int i = 0; i < 3; ++i) {
        const int64_t nb = out_cap * 4;
        if (overlap(outs[i], nb, queue, q_len * 4) || overlap(outs[i], nb, keep, q_len) ||
            overlap(outs[i], nb, offsets, (P + 1) * 8) || overlap(outs[i], nb, barrier, P) ||
            overlap(outs[i], nb, extra, extra_bytes))
            return true;
        for (int j = i + 1; j < 3; ++j)
            if (overlap(outs[i], nb, outs[j], nb)) return true;
    }
    return false;
}

Launch launch_of(ro_ctx *c)
{
    Launch L;
    L.stream = c->stream;
    L.num_cus = c->num_cus;
    L.ctl = c->ctl;
    L.desc = c->desc;
    L.desc_cap = c->desc_cap;
    L.tracer = c->tracer;
    return L;
}

template <typename T>
hipError_t dev_alloc(T **p, int64_t n)
{
    *p = nullptr;
    if (n <= 0) n = 1;
    return hipMalloc(reinterpret_cast<void **>(p), (size_t)n * sizeof(T));
}

int64_t tiles_for(int64_t n) { return (n + kTile - 1) / kTile + 1; }

// Make sure the look-back descriptors cover `tiles` tiles.
int ensure_desc(ro_ctx *c, int64_t tiles)
{
    if (tiles <= c->desc_cap) return RO_OK;
    if (hipStreamSynchronize(c->stream) != hipSuccess) return RO_EHIP;
    (void)hipFree(c->desc);
    c->desc = nullptr;
    c->desc_cap = 0;
    if (dev_alloc(&c->desc, tiles) != hipSuccess) return RO_EHIP;
    // zeroed on the context's stream: ordered before every later kernel on it
    if (launch_zero_u64(launch_of(c), c->desc, tiles) != hipSuccess) return RO_EHIP;
    c->desc_cap = tiles;
    return RO_OK;
}

int ensure_canon(ro_ctx *c, int64_t children)
{
    if (children <= c->canon_cap && c->canon) return RO_OK;
    if (hipStreamSynchronize(c->stream) != hipSuccess) return RO_EHIP;
    (void)hipFree(c->canon);
    (void)hipFree(c->sub_base);
    (void)hipFree(c->cmap);
    c->canon = nullptr;
    c->sub_base = nullptr;
    c->cmap = nullptr;
    c->canon_cap = 0;
    c->sub_cap = 0;
    c->cmap_cap = 0;
    const int64_t n = children > 0 ? children : 1;
    const int64_t subs = (n / kTile + 2) * (kTile / kSub);
    const int64_t maps = (n >> 3) + 4;          // coarse map: 8 bytes per 16 to 128 children
    if (dev_alloc(&c->canon, n) != hipSuccess || dev_alloc(&c->sub_base, subs) != hipSuccess ||
        dev_alloc(&c->cmap, maps) != hipSuccess ||
        launch_zero_u64(launch_of(c), reinterpret_cast<uint64_t *>(c->canon),
                        n * (int64_t)(sizeof(Canon) / sizeof(uint64_t))) != hipSuccess) {
        // leave no partial workspace behind: the next call starts from none
        (void)hipStreamSynchronize(c->stream);
        (void)hipFree(c->canon);
        (void)hipFree(c->sub_base);
        (void)hipFree(c->cmap);
        c->canon = nullptr;
        c->sub_base = nullptr;
        c->cmap = nullptr;
        return RO_EHIP;
    }
    c->canon_cap = n;
    c->sub_cap = subs;
    c->cmap_cap = maps;
    return ensure_desc(c, tiles_for(n));
}

int ensure_cnt(ro_ctx *c, int64_t parents)
{
    if (parents <= c->cnt_cap && c->cnt) return RO_OK;
    if (hipStreamSynchronize(c->stream) != hipSuccess) return RO_EHIP;
    (void)hipFree(c->cnt);
    (void)hipFree(c->gkey);
    c->cnt = nullptr;
    c->gkey = nullptr;
    c->cnt_cap = 0;
    const int64_t n = parents > 0 ? parents : 1;
    if (dev_alloc(&c->cnt, 3 * n) != hipSuccess || dev_alloc(&c->gkey, n) != hipSuccess ||
        launch_zero_u64(launch_of(c), c->gkey, n) != hipSuccess) {
        (void)hipStreamSynchronize(c->stream);
        (void)hipFree(c->cnt);
        (void)hipFree(c->gkey);
        c->cnt = nullptr;
        c->gkey = nullptr;
        return RO_EHIP;
    }
    c->cnt_cap = n;
    return RO_OK;
}

// Parent-bound reservation workspace for q queue entries and p parents (one
// allocation, 256-byte aligned arrays).
int ensure_pb(ro_ctx *c, int64_t q, int64_t p)
{
    if (q <= c->pb_cap && p <= c->pb_pcap && c->pb_block) return RO_OK;
    q = q > c->pb_cap ? q : c->pb_cap;
    p = p > c->pb_pcap ? p : c->pb_pcap;
    const int64_t qn = q > 0 ? q : 1, pn = p > 0 ? p : 1;
    const int64_t tiles = (qn + kPbTile * kPbSpan - 1) / (kPbTile * kPbSpan);   // histogram columns
    const size_t sizes[] = {
        (size_t)qn * 4, (size_t)qn * 4, (size_t)qn * 4, (size_t)qn * 8, (size_t)qn * 8,   // kc, k0, k1, v0, v1
        (size_t)qn * 4, (size_t)qn * 4,                                                    // fsize, bidx
        (size_t)pn * 4, (size_t)pn * 4,                                                    // pstart, pend
        (size_t)(kPbMaxBuckets * tiles) * 4, (size_t)(kPbMaxBuckets * tiles + 1) * 8,      // hist, hoff
        (size_t)2 * 8,                                                                     // m
    };
    constexpr int kArrays = (int)(sizeof(sizes) / sizeof(sizes[0]));
    size_t offs[kArrays], total = 0;
    for (int i = 0; i < kArrays; ++i) {
        offs[i] = total;
        total += (sizes[i] + 255) & ~(size_t)255;
    }
    if (hipStreamSynchronize(c->stream) != hipSuccess) return RO_EHIP;
    (void)hipFree(c->pb_block);
    c->pb_block = nullptr;
    c->pb_cap = c->pb_pcap = 0;
    char *b = nullptr;
    if (hipMalloc((void **)&b, total) != hipSuccess) return RO_EHIP;
    c->pb_block = b;
    c->pb.kc = (uint32_t *)(b + offs[0]);
    c->pb.k[0] = (uint32_t *)(b + offs[1]);
    c->pb.k[1] = (uint32_t *)(b + offs[2]);
    c->pb.v[0] = (uint64_t *)(b + offs[3]);
    c->pb.v[1] = (uint64_t *)(b + offs[4]);
    c->pb.fsize = (uint32_t *)(b + offs[5]);
    c->pb.bidx = (uint32_t *)(b + offs[6]);
    c->pb.pstart = (uint32_t *)(b + offs[7]);
    c->pb.pend = (uint32_t *)(b + offs[8]);
    c->pb.hist = (int32_t *)(b + offs[9]);
    c->pb.hoff = (int64_t *)(b + offs[10]);
    c->pb.m = (int64_t *)(b + offs[11]);
    c->pb_cap = q;
    c->pb_pcap = p;
    // descriptors: the compaction, the histogram scan and the two-chain group scan
    int64_t need = tiles_for(q);
    need = need > tiles_for(kPbMaxBuckets * tiles) ? need : tiles_for(kPbMaxBuckets * tiles);
    need = need > 2 * tiles_for(q) ? need : 2 * tiles_for(q);
    return ensure_desc(c, need);
}

int before_gather(ro_ctx *c)
{
    if (c->gathers + 1 > (int64_t)kMaxCanonEpoch) {
        if (launch_clear_tags(launch_of(c), c->canon, c->canon_cap) != hipSuccess) return RO_EHIP;
        // group-failure keys carry the same epoch
        if (c->gkey && launch_zero_u64(launch_of(c), c->gkey, c->cnt_cap) != hipSuccess) return RO_EHIP;
        c->gathers = 1;
    }
    c->gathers += 1;
    return RO_OK;
}

}  // namespace

extern "C" {

int ro_ctx_create(ro_ctx **out, void *hip_stream)
{
    if (out == nullptr) return RO_EINVAL;
    *out = nullptr;
    ro_ctx *c = (ro_ctx *)calloc(1, sizeof(ro_ctx));
    if (!c) return RO_EINVAL;
    c->tracer = new Tracer();
    c->stream = (hipStream_t)hip_stream;
    if (hipGetDevice(&c->device) != hipSuccess ||
        hipDeviceGetAttribute(&c->num_cus, hipDeviceAttributeMultiprocessorCount, c->device) != hipSuccess ||
        dev_alloc(&c->ctl, 1) != hipSuccess) {
        ro_ctx_destroy(c);
        return RO_EHIP;
    }
    if (c->num_cus <= 0) c->num_cus = 1;
    if (hipMemset(c->ctl, 0, sizeof(Ctl)) != hipSuccess ||
        launch_ctl_init(launch_of(c)) != hipSuccess || hipDeviceSynchronize() != hipSuccess ||
        ensure_desc(c, 64) != RO_OK) {
        ro_ctx_destroy(c);
        return RO_EHIP;
    }
    c->gathers = 1;           // the first gather runs at canonical epoch 1
    *out = c;
    return RO_OK;
}

int ro_ctx_set_stream(ro_ctx *c, void *hip_stream)
{
    if (!c) return RO_EINVAL;
    if (hipStreamSynchronize(c->stream) != hipSuccess) return RO_EHIP;
    c->stream = (hipStream_t)hip_stream;
    return RO_OK;
}

int ro_ctx_reserve(ro_ctx *c, int64_t max_children, int64_t max_parents, int64_t max_queue)
{
    if (!c || max_children < 0 || max_parents < 0 || max_queue < 0) return RO_EINVAL;
    int rc = ensure_canon(c, max_children);
    if (rc) return rc;
    rc = ensure_cnt(c, max_parents);
    if (rc) return rc;
    int64_t m = max_children > max_parents ? max_children : max_parents;
    m = m > max_queue ? m : max_queue;
    return ensure_desc(c, tiles_for(m));
}

int ro_ctx_status(ro_ctx *c)
{
    if (!c) return RO_EINVAL;
    if (hipStreamSynchronize(c->stream) != hipSuccess) return RO_EHIP;
    int32_t err = 0;
    if (hipMemcpy(&err, &c->ctl->err, sizeof(err), hipMemcpyDeviceToHost) != hipSuccess) return RO_EHIP;
    // cleared by a kernel on the context's stream, so that no later kernel of
    // the context can see the old error (a host-to-device copy may still be
    // in flight when it returns)
    if (err != 0 && launch_clear_err(launch_of(c)) != hipSuccess) return RO_EHIP;
    return err;
}

int ro_ctx_destroy(ro_ctx *c)
{
    if (!c) return RO_EINVAL;
    if (c->stream || c->ctl) (void)hipStreamSynchronize(c->stream);
    (void)hipFree(c->ctl);
    (void)hipFree(c->desc);
    (void)hipFree(c->canon);
    (void)hipFree(c->sub_base);
    (void)hipFree(c->cmap);
    (void)hipFree(c->cnt);
    (void)hipFree(c->gkey);
    (void)hipFree(c->pb_block);
    if (c->tracer) {
        for (hipEvent_t e : c->tracer->pool) (void)hipEventDestroy(e);
        delete c->tracer;
    }
    free(c);
    return RO_OK;
}

int ro_ctx_trace(ro_ctx *c, int enable)
{
    if (!c || !c->tracer) return RO_EINVAL;
    c->tracer->on = enable != 0;
    return RO_OK;
}

int ro_ctx_trace_read(ro_ctx *c, int64_t *launches, double *total_ms, int32_t n)
{
    if (!c || !c->tracer || n < 0 || (n > 0 && (!launches || !total_ms))) return RO_EINVAL;
    Tracer *t = c->tracer;
    if (hipStreamSynchronize(c->stream) != hipSuccess) return RO_EHIP;
    for (const Tracer::Rec &r : t->recs) {
        if (r.kind < 0 || r.kind >= n || !r.e0 || !r.e1) continue;
        float ms = 0.f;
        if (hipEventElapsedTime(&ms, r.e0, r.e1) != hipSuccess) continue;
        launches[r.kind] += 1;
        total_ms[r.kind] += (double)ms;
    }
    t->recs.clear();
    t->used = 0;
    return RO_OK;
}

int ro_expand(ro_ctx *c, const int32_t *counts, int64_t n_parents, int64_t *offsets,
              uint32_t *child_parent, uint32_t *child_ordinal, int64_t child_cap)
{
    if (!c || !offsets || n_parents < 0 || child_cap < 0 || (n_parents > 0 && !counts)) return RO_EINVAL;
    int rc = ensure_desc(c, tiles_for(n_parents));
    if (rc) return rc;
    return hip_fail(launch_expand(launch_of(c), counts, n_parents, offsets, child_parent, child_ordinal,
                                  child_cap));
}

int ro_batch(ro_ctx *c, const uint32_t *queue, const uint8_t *keep, int64_t q_len,
             const int64_t *offsets, int64_t n_parents, int32_t batch_size,
             uint32_t *out_child, uint32_t *out_parent, uint32_t *out_ordinal, int64_t out_cap,
             int64_t *n_out_dev, int64_t *n_batches_dev, const uint8_t *barrier)
{
    if (!c || !offsets || q_len < 0 || n_parents < 0 || batch_size <= 0 || out_cap < 0 ||
        (q_len > 0 && !queue))
        return RO_EINVAL;
    uint32_t *const outs[3] = {out_child, out_parent, out_ordinal};
    if (batch_outputs_alias(queue, keep, q_len, offsets, n_parents, barrier, outs, out_cap, nullptr, 0))
        return RO_EINVAL;
    int rc = ensure_desc(c, tiles_for(q_len));
    if (rc) return rc;
    return hip_fail(launch_batch(launch_of(c), queue, keep, q_len, offsets, n_parents, batch_size,
                                 out_child, out_parent, out_ordinal, out_cap, n_out_dev, n_batches_dev,
                                 c->cmap, c->cmap_cap, barrier));
}

int ro_batch_parent(ro_ctx *c, const uint32_t *queue, const uint8_t *keep, int64_t q_len,
                    const int64_t *offsets, int64_t n_parents, int32_t batch_size, uint32_t *out_child,
                    uint32_t *out_parent, uint32_t *out_ordinal, int64_t out_cap, int64_t *batch_off,
                    int64_t batch_cap, int64_t *n_out_dev, int64_t *n_batches_dev, const uint8_t *barrier)
{
    if (!c || !offsets || q_len < 0 || n_parents < 0 || batch_size <= 0 || out_cap < 0 || !batch_off ||
        batch_cap < 1 || (q_len > 0 && !queue))
        return RO_EINVAL;
    if (q_len >= ((int64_t)1 << 32) || n_parents >= ((int64_t)1 << 32)) return RO_EINVAL;
    uint32_t *const outs[3] = {out_child, out_parent, out_ordinal};
    if (batch_outputs_alias(queue, keep, q_len, offsets, n_parents, barrier, outs, out_cap, batch_off,
                            batch_cap * 8) ||
        overlap(batch_off, batch_cap * 8, queue, q_len * 4) || overlap(batch_off, batch_cap * 8, keep, q_len) ||
        overlap(batch_off, batch_cap * 8, offsets, (n_parents + 1) * 8) ||
        overlap(batch_off, batch_cap * 8, barrier, n_parents))
        return RO_EINVAL;
    int rc = ensure_pb(c, q_len, n_parents);
    if (rc) return rc;
    rc = ensure_desc(c, tiles_for(q_len));
    if (rc) return rc;
    return hip_fail(launch_batch_parent(launch_of(c), queue, keep, q_len, offsets, n_parents, batch_size,
                                        out_child, out_parent, out_ordinal, out_cap, batch_off, batch_cap,
                                        n_out_dev, n_batches_dev, c->cmap, c->cmap_cap, barrier, c->pb));
}

int ro_gather(ro_ctx *c, const ro_reports *r, const int64_t *offsets, int64_t n_parents,
              const ro_gather_out *o)
{
    if (!c || !r || !o || !offsets || n_parents < 0 || r->n < 0 || !o->out_off || o->out_cap < 0)
        return RO_EINVAL;
    if (r->n > 0 && (!r->parent || !r->ordinal || !r->state || !r->off)) return RO_EINVAL;
    if (o->out_data != nullptr && r->n > 0 && !r->data) return RO_EINVAL;
    if (o->barrier != nullptr && r->n >= ((int64_t)1 << 32)) return RO_EINVAL;   // report index is 32-bit
    // the canonical workspace must cover the expansion; its size is on the
    // device, so the report count is the host's best lower bound
    int rc = ensure_canon(c, c->canon_cap > r->n ? c->canon_cap : r->n);
    if (rc) return rc;
    rc = ensure_desc(c, tiles_for(c->canon_cap));
    if (rc) return rc;
    GatherArgs a;
    a.rp = r->parent;
    a.ro = r->ordinal;
    a.rs = r->state;
    a.roff = r->off;
    a.data = r->data;
    a.n = r->n;
    a.offsets = offsets;
    a.P = n_parents;
    a.out_off = o->out_off;
    a.out_data = o->out_data;
    a.out_cap = o->out_cap;
    a.ns = o->n_success;
    a.nf = o->n_failed;
    a.nk = o->n_skipped;
    a.complete = o->complete;
    a.pstate = o->parent_state;
    a.cdst = o->child_dst_off;
    a.barrier = o->barrier;
    a.n_rejected = o->n_rejected;
    if (a.barrier && (rc = ensure_cnt(c, n_parents))) return rc;
    if (!a.ns || !a.nf || !a.nk) {
        if ((rc = ensure_cnt(c, n_parents))) return rc;
        if (!a.ns) a.ns = c->cnt;
        if (!a.nf) a.nf = c->cnt + c->cnt_cap;
        if (!a.nk) a.nk = c->cnt + 2 * c->cnt_cap;
    }
    GatherWs w;
    w.canon = c->canon;
    w.canon_cap = c->canon_cap;
    w.sub_base = c->sub_base;
    w.sub_cap = c->sub_cap;
    w.gkey = c->gkey;
    if ((rc = before_gather(c))) return rc;
    return hip_fail(launch_gather(launch_of(c), a, w, (uint32_t)(c->gathers - 1)));
}

int ro_filter(ro_ctx *c, const uint8_t *x_state, const uint8_t *mask_state, const uint8_t *mask, int64_t n,
              uint8_t *out_state)
{
    if (!c || n < 0 || (n > 0 && (!x_state || !mask || !out_state))) return RO_EINVAL;
    if (n == 0) return RO_OK;
    return hip_fail(launch_filter(launch_of(c), x_state, mask_state, mask, n, out_state));
}

int ro_broadcast(ro_ctx *c, const uint32_t *const *maps, const int64_t *map_len, int32_t levels, int64_t n,
                 const uint8_t *x_state, int64_t n_ancestors, const uint8_t *like_state, uint32_t *out_ancestor,
                 uint8_t *out_state)
{
    if (!c || n < 0 || n_ancestors < 0 || levels < 1 || levels > kMaxBroadcastLevels) return RO_EINVAL;
    if (n > 0 && (!maps || !map_len || !x_state || !out_state)) return RO_EINVAL;
    for (int32_t l = 0; n > 0 && l < levels; ++l)
        if (!maps[l] || map_len[l] < 0) return RO_EINVAL;
    if (n == 0) return RO_OK;
    if (map_len[0] < n) return RO_EINVAL;
    return hip_fail(launch_broadcast(launch_of(c), maps, map_len, levels, n, x_state, n_ancestors, like_state,
                                     out_ancestor, out_state));
}

int ro_grains_create(ro_ctx *c, int64_t n_children, ro_grains **out)
{
    if (out) *out = nullptr;
    if (!c || !out || n_children < 0 || n_children >= ((int64_t)1 << 32)) return RO_EINVAL;
    const int64_t n = n_children > 0 ? n_children : 1;
    ro_grains *g = (ro_grains *)calloc(1, sizeof(ro_grains));
    if (!g) return RO_EINVAL;
    if (hipMalloc((void **)&g->g, (size_t)n * sizeof(Grain)) != hipSuccess) {
        free(g);
        return RO_EHIP;
    }
    g->ctx = c;
    g->n = n_children;
    g->epoch = 0;
    if (launch_grains_fill(launch_of(c), g->g, n) != hipSuccess) {
        (void)hipFree(g->g);
        free(g);
        return RO_EHIP;
    }
    *out = g;
    return RO_OK;
}

int ro_grains_reset(ro_ctx *c, ro_grains *g)
{
    if (!c || !g || g->ctx != c) return RO_EINVAL;
    g->epoch = 0;
    return hip_fail(launch_grains_fill(launch_of(c), g->g, g->n > 0 ? g->n : 1));
}

int ro_grains_destroy(ro_grains *g)
{
    if (!g) return RO_EINVAL;
    if (g->ctx) (void)hipStreamSynchronize(g->ctx->stream);
    (void)hipFree(g->g);
    if (g->tag) (void)hipFree(g->tag);
    free(g);
    return RO_OK;
}

int ro_grains_read(ro_ctx *c, ro_grains *g, uint32_t *phase, uint32_t *generation)
{
    if (!c || !g || g->ctx != c) return RO_EINVAL;
    if (g->n == 0 || (!phase && !generation)) return RO_OK;
    return hip_fail(launch_grains_read(launch_of(c), g->g, g->n, phase, generation));
}

int ro_grains_dispatch(ro_ctx *c, ro_grains *g, const uint32_t *child, int64_t n, uint32_t *out_generation)
{
    if (!c || !g || g->ctx != c || n < 0 || (n > 0 && !child)) return RO_EINVAL;
    if (n == 0) return RO_OK;
    return hip_fail(launch_grains_dispatch(launch_of(c), child, n, g->n, g->g, out_generation));
}

int ro_grains_retry(ro_ctx *c, ro_grains *g, const uint32_t *child, int64_t n)
{
    if (!c || !g || g->ctx != c || n < 0 || (n > 0 && !child)) return RO_EINVAL;
    if (n == 0) return RO_OK;
    return hip_fail(launch_grains_retry(launch_of(c), child, n, g->n, g->g));
}

int ro_grains_commit(ro_ctx *c, ro_grains *g, const ro_reports *r, const uint32_t *generation,
                     const int64_t *offsets, int64_t n_parents, uint8_t *state_out, int64_t *counts_dev)
{
    if (!c || !g || g->ctx != c || !r || !offsets || n_parents < 0 || r->n < 0) return RO_EINVAL;
    if (r->n >= ((int64_t)1 << 32)) return RO_EINVAL;                // report index is 32-bit
    if (r->n > 0 && (!r->parent || !r->ordinal || !r->state || !r->off || !generation || !state_out))
        return RO_EINVAL;
    const Launch L = launch_of(c);
    const int64_t need = r->n > 0 ? r->n : 1;
    if (need > g->tag_cap) {                  // grows with the largest call; starts untagged
        const int64_t cap = need > 2 * g->tag_cap ? need : 2 * g->tag_cap;
        uint32_t *t = nullptr;
        if (hipMalloc((void **)&t, (size_t)cap * sizeof(uint32_t)) != hipSuccess) return RO_EHIP;
        if (g->tag) {
            (void)hipStreamSynchronize(c->stream);
            (void)hipFree(g->tag);
        }
        g->tag = t;
        g->tag_cap = cap;
        if (launch_grains_zero_tags(L, g->tag, cap) != hipSuccess) return RO_EHIP;
    }
    if (g->epoch == 0xffffffffu) {            // keys and tags of every earlier call must read as old
        if (launch_grains_rekey(L, g->g, g->n > 0 ? g->n : 1) != hipSuccess) return RO_EHIP;
        if (launch_grains_zero_tags(L, g->tag, g->tag_cap) != hipSuccess) return RO_EHIP;
        g->epoch = 0;
    }
    g->epoch += 1;
    return hip_fail(launch_grains_commit(L, r->parent, r->ordinal, r->state, r->off, r->data, generation, r->n,
                                         offsets, n_parents, g->n, g->g, g->epoch, g->tag, state_out, counts_dev));
}

int ro_stream_create(ro_ctx *c, const int64_t *offsets, int64_t n_parents, int64_t n_children,
                     uint8_t *barrier, ro_stream **out)
{
    if (out) *out = nullptr;
    if (!c || !offsets || !out || n_parents < 0 || n_children < 0 || n_children >= ((int64_t)1 << 32))
        return RO_EINVAL;
    const int64_t P = n_parents, N = n_children;
    int rc = ensure_desc(c, stream_desc_tiles(P, N));
    if (rc) return rc;
    // one allocation, carved into 256-byte aligned arrays
    const size_t sizes[] = {
        (size_t)(N > 0 ? N : 1) * sizeof(Canon),            // canon
        (size_t)((N + 31) / 32 + 1) * sizeof(uint32_t),     // seen
        (size_t)stream_mid_size(N) * sizeof(int32_t),       // mid
        (size_t)stream_big_size(N) * sizeof(int32_t),       // big
        (size_t)(P + 1),                                    // emitted
        (size_t)(P + 1) * sizeof(int64_t),                  // ebase
        (size_t)(P + 2) * sizeof(int64_t),                  // evoff
        (size_t)(3 * (P + 1)) * sizeof(int32_t),            // ecnt
        (size_t)(N + 1) * sizeof(int64_t),                  // edst
        (size_t)(N + 1) * sizeof(uint64_t),                 // esrc
        (size_t)(P + 1) * sizeof(uint64_t),                 // gkey
        (size_t)(P + 1),                                    // ebar
        (size_t)(N > 0 ? N : 1) * sizeof(uint32_t),         // cpar
    };
    constexpr int kArrays = (int)(sizeof(sizes) / sizeof(sizes[0]));
    size_t offs[kArrays], total = 0;
    for (int i = 0; i < kArrays; ++i) {
        offs[i] = total;
        total += (sizes[i] + 255) & ~(size_t)255;
    }
    ro_stream *s = (ro_stream *)calloc(1, sizeof(ro_stream));
    if (!s) return RO_EINVAL;
    char *block = nullptr;
    if (hipStreamSynchronize(c->stream) != hipSuccess || hipMalloc((void **)&block, total) != hipSuccess) {
        free(s);
        return RO_EHIP;
    }
    if (launch_zero_u64(launch_of(c), reinterpret_cast<uint64_t *>(block), (int64_t)(total / 8)) != hipSuccess) {
        (void)hipFree(block);
        free(s);
        return RO_EHIP;
    }
    s->ctx = c;
    s->block = block;
    StreamState &st = s->st;
    st.offsets = offsets;
    st.P = P;
    st.N = N;
    st.canon = (Canon *)(block + offs[0]);
    st.seen = (uint32_t *)(block + offs[1]);
    st.mid = (int32_t *)(block + offs[2]);
    st.big = (int32_t *)(block + offs[3]);
    st.emitted = (uint8_t *)(block + offs[4]);
    st.ebase = (int64_t *)(block + offs[5]);
    st.evoff = (int64_t *)(block + offs[6]);
    st.ecnt = (int32_t *)(block + offs[7]);
    st.edst = (int64_t *)(block + offs[8]);
    st.esrc = (uint64_t *)(block + offs[9]);
    st.gkey = (uint64_t *)(block + offs[10]);
    st.ebar = (uint8_t *)(block + offs[11]);
    st.cpar = (uint32_t *)(block + offs[12]);
    st.barrier = barrier;
    st.run_epoch = 1;
    st.gf_epoch = 0;
    if (launch_stream_init(launch_of(c), st) != hipSuccess ||
        launch_expand_tags(launch_of(c), offsets, P, st.cpar, nullptr, N) != hipSuccess) {
        (void)hipStreamSynchronize(c->stream);     // a launch that did start still uses the block
        (void)hipFree(block);
        free(s);
        return RO_EHIP;
    }
    *out = s;
    return RO_OK;
}

int ro_stream_batch(ro_ctx *c, ro_stream *s, const uint32_t *queue, const uint8_t *keep, int64_t q_len,
                    int32_t batch_size, uint32_t *out_child, uint32_t *out_parent, uint32_t *out_ordinal,
                    int64_t out_cap, int64_t *n_out_dev, int64_t *n_batches_dev)
{
    if (!c || !s || s->ctx != c || q_len < 0 || batch_size <= 0 || out_cap < 0 || (q_len > 0 && !queue))
        return RO_EINVAL;
    const StreamState &st = s->st;
    uint32_t *const outs[3] = {out_child, out_parent, out_ordinal};
    if (batch_outputs_alias(queue, keep, q_len, st.offsets, st.P, st.barrier, outs, out_cap, nullptr, 0))
        return RO_EINVAL;
    int rc = ensure_desc(c, tiles_for(q_len));
    if (rc) return rc;
    return hip_fail(launch_batch(launch_of(c), queue, keep, q_len, st.offsets, st.P, batch_size, out_child,
                                 out_parent, out_ordinal, out_cap, n_out_dev, n_batches_dev, nullptr, 0, st.barrier,
                                 st.cpar, st.N));
}

int ro_stream_report(ro_ctx *c, ro_stream *s, const ro_reports *r, int64_t *n_rejected_dev)
{
    if (!c || !s || !r || s->ctx != c || r->n < 0) return RO_EINVAL;
    if (r->n > 0 && (!r->parent || !r->ordinal || !r->state || !r->off)) return RO_EINVAL;
    if (s->st.barrier != nullptr && r->n >= ((int64_t)1 << 32)) return RO_EINVAL;
    if (r->n == 0) return RO_OK;
    if (s->st.barrier != nullptr) {
        // a new epoch for this call's first group failures
        if (s->st.gf_epoch == 0xffffffffu) {
            if (launch_zero_u64(launch_of(c), s->st.gkey, s->st.P + 1) != hipSuccess) return RO_EHIP;
            s->st.gf_epoch = 0;
        }
        s->st.gf_epoch += 1;
    }
    return hip_fail(launch_stream_report(launch_of(c), s->st, r->parent, r->ordinal, r->state, r->off, r->data,
                                         r->n, n_rejected_dev));
}

int ro_stream_emit(ro_ctx *c, ro_stream *s, uint32_t *emit_parent, int64_t *emit_off,
                   uint8_t *emit_data, int64_t cap_parents, int64_t cap_bytes,
                   int32_t *n_success, int32_t *n_failed, int32_t *n_skipped,
                   uint8_t *parent_state, int64_t *n_emitted_dev, int64_t *n_bytes_dev)
{
    if (!c || !s || s->ctx != c || !emit_off || cap_parents < 0 || cap_bytes < 0) return RO_EINVAL;
    return hip_fail(launch_stream_emit(launch_of(c), s->st, emit_parent, emit_off, emit_data, cap_parents,
                                       cap_bytes, n_success, n_failed, n_skipped, parent_state, n_emitted_dev,
                                       n_bytes_dev));
}

int ro_stream_reset(ro_ctx *c, ro_stream *s)
{
    if (!c || !s || s->ctx != c) return RO_EINVAL;
    // a new slot epoch, so that the slots of the previous run read as unreported
    if (s->st.run_epoch + 1 > kMaxCanonEpoch) {
        if (launch_clear_tags(launch_of(c), s->st.canon, s->st.N) != hipSuccess) return RO_EHIP;
        s->st.run_epoch = 0;
    }
    s->st.run_epoch += 1;
    return hip_fail(launch_stream_reset(launch_of(c), s->st));
}

int ro_debug_epochs(ro_ctx *c, ro_stream *s, ro_grains *g, int64_t canon_left, int64_t run_left,
                    int64_t gf_left, int64_t fence_left)
{
    if (!c || (s && s->ctx != c) || (g && g->ctx != c)) return RO_EINVAL;
    if (canon_left >= 1 && canon_left < (int64_t)kMaxCanonEpoch) {
        // the next gather runs at epoch max - canon_left + 1
        const uint32_t e = (uint32_t)((int64_t)kMaxCanonEpoch - canon_left + 1);
        if (e > (uint32_t)c->gathers) c->gathers = e;
    }
    if (s) {
        if (run_left >= 1 && run_left < (int64_t)kMaxCanonEpoch &&
            (uint32_t)((int64_t)kMaxCanonEpoch - run_left) > s->st.run_epoch)
            s->st.run_epoch = (uint32_t)((int64_t)kMaxCanonEpoch - run_left);
        if (gf_left >= 1 && gf_left <= 0xffffffffll &&
            (uint32_t)(0xffffffffll - gf_left) > s->st.gf_epoch)
            s->st.gf_epoch = (uint32_t)(0xffffffffll - gf_left);
    }
    if (g && fence_left >= 1 && fence_left <= 0xffffffffll && (uint32_t)(0xffffffffll - fence_left) > g->epoch)
        g->epoch = (uint32_t)(0xffffffffll - fence_left);
    return RO_OK;
}

int ro_stream_destroy(ro_stream *s)
{
    if (!s) return RO_EINVAL;
    if (s->ctx) (void)hipStreamSynchronize(s->ctx->stream);
    (void)hipFree(s->block);
    free(s);
    return RO_OK;
}

}  // extern "C"
