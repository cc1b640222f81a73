/*
 * Test infrastructure: the library used from plain C, with no Python and no
 * torch.  Device memory and the stream come from the HIP runtime directly;
 * ro_expand, ro_batch and ro_gather run on seeded random cases and every
 * output is compared with the C oracle (linked from oracle/) bit for bit.
 * One more case plants a report with an out-of-range ordinal and checks that
 * ro_ctx_status returns RO_ERANGE, then that the context works again.  Then
 * parent-bound reservations, a stream fed in waves, filter and broadcast,
 * Grain phases with the generation fence, and the per-kernel trace, each
 * against the oracle.
 *
 * Exit status 0 and a last line "c abi ok" mean every case matched.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "ro.h"

int oracle_expand(const int32_t *, int64_t, int64_t *, uint32_t *, uint32_t *, int64_t);
int oracle_batch(const uint32_t *, const uint8_t *, int64_t, const int64_t *, int64_t, int32_t, uint32_t *,
                 uint32_t *, uint32_t *, int64_t, int64_t *, int64_t *, int64_t *, const uint8_t *);
int oracle_gather(const uint32_t *, const uint32_t *, const uint8_t *, const int64_t *, const uint8_t *, int64_t,
                  const int64_t *, int64_t, int64_t *, uint8_t *, int64_t, int32_t *, int32_t *, int32_t *,
                  uint8_t *, uint8_t *, int64_t *, uint8_t *, int64_t *);

typedef struct oracle_stream oracle_stream;
typedef struct oracle_grains oracle_grains;
int oracle_batch_parent(const uint32_t *, const uint8_t *, int64_t, const int64_t *, int64_t, int32_t, uint32_t *,
                        uint32_t *, uint32_t *, int64_t, int64_t *, int64_t *, int64_t *, const uint8_t *);
oracle_stream *oracle_stream_create(const int64_t *, int64_t);
void oracle_stream_destroy(oracle_stream *);
int oracle_stream_report(oracle_stream *, const uint32_t *, const uint32_t *, const uint8_t *, const int64_t *,
                         const uint8_t *, int64_t, int64_t *);
int oracle_stream_emit(oracle_stream *, uint32_t *, int64_t *, uint8_t *, int64_t, int64_t, int32_t *, int32_t *,
                       int32_t *, uint8_t *, int64_t *, int64_t *);
int oracle_filter(const uint8_t *, const uint8_t *, const uint8_t *, int64_t, uint8_t *);
int oracle_broadcast(const uint32_t *const *, int32_t, int64_t, const uint8_t *, int64_t, const uint8_t *,
                     uint32_t *, uint8_t *);
oracle_grains *oracle_grains_create(int64_t);
void oracle_grains_destroy(oracle_grains *);
const uint8_t *oracle_grains_phase(const oracle_grains *);
const uint32_t *oracle_grains_gen(const oracle_grains *);
int oracle_grains_dispatch(oracle_grains *, const uint32_t *, int64_t, uint32_t *);
int oracle_grains_retry(oracle_grains *, const uint32_t *, int64_t);
int oracle_grains_commit(oracle_grains *, const uint32_t *, const uint32_t *, const uint8_t *, const int64_t *,
                         const uint8_t *, const uint32_t *, int64_t, const int64_t *, int64_t, uint8_t *,
                         int64_t *);

#define HIP_OK(x) do { if ((x) != hipSuccess) { printf("HIP call failed at line %d\n", __LINE__); exit(2); } } while (0)
#define RO_OK_(x) do { int rc_ = (x); if (rc_ != RO_OK) { printf("ro call returned %d at line %d\n", rc_, __LINE__); exit(2); } } while (0)
#define EXPECT(c, what) do { if (!(c)) { printf("mismatch: %s (case %d)\n", what, case_id); exit(1); } } while (0)

static uint64_t rng = 0x243F6A8885A308D3ull;
static uint64_t rnd(void)                       /* xorshift64* */
{
    rng ^= rng >> 12;
    rng ^= rng << 25;
    rng ^= rng >> 27;
    return rng * 0x2545F4914F6CDD1Dull;
}
static int64_t below(int64_t n) { return n > 0 ? (int64_t)(rnd() % (uint64_t)n) : 0; }
static void *xmalloc(size_t n) { void *p = calloc(n ? n : 1, 1); if (!p) exit(3); return p; }
static void *dmalloc(size_t n) { void *p = NULL; HIP_OK(hipMalloc(&p, n ? n : 1)); return p; }
/* The context's stream does not synchronise with the null stream, so every
 * copy first waits for the work enqueued on it. */
static hipStream_t g_st;
static void up(void *d, const void *h, size_t n)
{
    HIP_OK(hipStreamSynchronize(g_st));
    if (n) HIP_OK(hipMemcpy(d, h, n, hipMemcpyHostToDevice));
}
static void down(void *h, const void *d, size_t n)
{
    HIP_OK(hipStreamSynchronize(g_st));
    if (n) HIP_OK(hipMemcpy(h, d, n, hipMemcpyDeviceToHost));
}
static void shuffle(uint32_t *a, int64_t n)
{
    for (int64_t i = n - 1; i > 0; --i) {
        const int64_t j = below(i + 1);
        const uint32_t t = a[i]; a[i] = a[j]; a[j] = t;
    }
}

static int case_id;

static void one_case(ro_ctx *ctx, hipStream_t st, int64_t P, int32_t B, int plant_error)
{
    /* ---- inputs ---- */
    int32_t *counts = xmalloc((size_t)P * 4);
    int64_t N = 0;
    for (int64_t p = 0; p < P; ++p) { counts[p] = (int32_t)below(7); N += counts[p]; }
    uint32_t *queue = xmalloc((size_t)N * 4);
    uint8_t *keep = xmalloc((size_t)N);
    for (int64_t i = 0; i < N; ++i) { queue[i] = (uint32_t)i; keep[i] = below(5) != 0; }
    shuffle(queue, N);

    /* ---- expand + batch on the device ---- */
    int32_t *d_counts = dmalloc((size_t)P * 4);
    int64_t *d_off = dmalloc((size_t)(P + 1) * 8);
    uint32_t *d_cp = dmalloc((size_t)N * 4), *d_co = dmalloc((size_t)N * 4);
    uint32_t *d_q = dmalloc((size_t)N * 4);
    uint8_t *d_keep = dmalloc((size_t)N);
    uint32_t *d_bc = dmalloc((size_t)N * 4), *d_bp = dmalloc((size_t)N * 4), *d_bo = dmalloc((size_t)N * 4);
    int64_t *d_sc = dmalloc(2 * 8);
    up(d_counts, counts, (size_t)P * 4);
    up(d_q, queue, (size_t)N * 4);
    up(d_keep, keep, (size_t)N);
    RO_OK_(ro_expand(ctx, d_counts, P, d_off, d_cp, d_co, N));
    RO_OK_(ro_batch(ctx, d_q, d_keep, N, d_off, P, B, d_bc, d_bp, d_bo, N, d_sc, d_sc + 1, NULL));
    RO_OK_(ro_ctx_status(ctx));

    /* ---- the same on the oracle ---- */
    int64_t *offs = xmalloc((size_t)(P + 1) * 8);
    uint32_t *cp = xmalloc((size_t)N * 4), *co = xmalloc((size_t)N * 4);
    uint32_t *bc = xmalloc((size_t)N * 4), *bp = xmalloc((size_t)N * 4), *bo = xmalloc((size_t)N * 4);
    int64_t M = 0, nb = 0;
    if (oracle_expand(counts, P, offs, cp, co, N) != 0) exit(4);
    if (oracle_batch(queue, keep, N, offs, P, B, bc, bp, bo, N, &M, &nb, NULL, NULL) != 0) exit(4);

    int64_t *g_offs = xmalloc((size_t)(P + 1) * 8), g_sc[2];
    uint32_t *g_cp = xmalloc((size_t)N * 4), *g_co = xmalloc((size_t)N * 4);
    uint32_t *g_bc = xmalloc((size_t)N * 4), *g_bp = xmalloc((size_t)N * 4), *g_bo = xmalloc((size_t)N * 4);
    down(g_offs, d_off, (size_t)(P + 1) * 8);
    down(g_cp, d_cp, (size_t)N * 4);
    down(g_co, d_co, (size_t)N * 4);
    down(g_sc, d_sc, 16);
    EXPECT(memcmp(g_offs, offs, (size_t)(P + 1) * 8) == 0, "expand offsets");
    EXPECT(memcmp(g_cp, cp, (size_t)N * 4) == 0 && memcmp(g_co, co, (size_t)N * 4) == 0, "lineage tags");
    EXPECT(g_sc[0] == M && g_sc[1] == nb, "batch counts");
    down(g_bc, d_bc, (size_t)M * 4);
    down(g_bp, d_bp, (size_t)M * 4);
    down(g_bo, d_bo, (size_t)M * 4);
    EXPECT(memcmp(g_bc, bc, (size_t)M * 4) == 0, "batch children");
    EXPECT(memcmp(g_bp, bp, (size_t)M * 4) == 0 && memcmp(g_bo, bo, (size_t)M * 4) == 0, "batch tags");

    /* ---- reports: every child once, in a random order, after a 3-byte lead ---- */
    uint32_t *order = xmalloc((size_t)N * 4);
    for (int64_t i = 0; i < N; ++i) order[i] = (uint32_t)i;
    shuffle(order, N);
    uint32_t *rp = xmalloc((size_t)N * 4), *ro_ = xmalloc((size_t)N * 4);
    uint8_t *rs = xmalloc((size_t)N);
    int64_t *roff = xmalloc((size_t)(N + 1) * 8);
    roff[0] = 3;
    static const uint8_t states[5] = {RO_SUCCESS, RO_SUCCESS, RO_SUCCESS, RO_FAILED, RO_SKIPPED};
    for (int64_t i = 0; i < N; ++i) {
        const uint32_t c = order[i];
        rp[i] = cp[c];
        ro_[i] = co[c];
        rs[i] = states[below(5)];
        roff[i + 1] = roff[i] + below(41);
    }
    if (plant_error && N > 0) ro_[N / 2] = (uint32_t)counts[rp[N / 2]];     /* one past the last ordinal */
    const int64_t bytes = roff[N];
    uint8_t *data = xmalloc((size_t)bytes + 16);
    for (int64_t i = 0; i < bytes + 16; ++i) data[i] = (uint8_t)rnd();

    uint32_t *d_rp = dmalloc((size_t)N * 4), *d_ro = dmalloc((size_t)N * 4);
    uint8_t *d_rs = dmalloc((size_t)N), *d_data = dmalloc((size_t)bytes + 16);
    int64_t *d_roff = dmalloc((size_t)(N + 1) * 8);
    up(d_rp, rp, (size_t)N * 4);
    up(d_ro, ro_, (size_t)N * 4);
    up(d_rs, rs, (size_t)N);
    up(d_roff, roff, (size_t)(N + 1) * 8);
    up(d_data, data, (size_t)bytes + 16);
    int64_t *d_oo = dmalloc((size_t)(P + 1) * 8);
    uint8_t *d_od = dmalloc((size_t)bytes + 16);
    int32_t *d_cnt = dmalloc((size_t)P * 12);
    uint8_t *d_comp = dmalloc((size_t)P), *d_pst = dmalloc((size_t)P);
    int64_t *d_cdst = dmalloc((size_t)(N + 1) * 8);

    ro_reports r = {d_rp, d_ro, d_rs, d_roff, d_data, N};
    ro_gather_out o;
    memset(&o, 0, sizeof o);
    o.out_off = d_oo;
    o.out_data = d_od;
    o.out_cap = bytes;
    o.n_success = d_cnt;
    o.n_failed = d_cnt + P;
    o.n_skipped = d_cnt + 2 * P;
    o.complete = d_comp;
    o.parent_state = d_pst;
    o.child_dst_off = d_cdst;
    RO_OK_(ro_gather(ctx, &r, d_off, P, &o));
    const int status = ro_ctx_status(ctx);
    if (plant_error && N > 0) {
        EXPECT(status == RO_ERANGE, "planted out-of-range ordinal is RO_ERANGE");
    } else {
        EXPECT(status == RO_OK, "gather status");
        int64_t *w_oo = xmalloc((size_t)(P + 1) * 8), *w_cdst = xmalloc((size_t)(N + 1) * 8);
        uint8_t *w_od = xmalloc((size_t)bytes + 1), *w_comp = xmalloc((size_t)P), *w_pst = xmalloc((size_t)P);
        int32_t *w_cnt = xmalloc((size_t)P * 12);
        if (oracle_gather(rp, ro_, rs, roff, data, N, offs, P, w_oo, w_od, bytes, w_cnt, w_cnt + P, w_cnt + 2 * P,
                          w_comp, w_pst, w_cdst, NULL, NULL) != 0)
            exit(4);
        int64_t *g_oo = xmalloc((size_t)(P + 1) * 8), *g_cdst = xmalloc((size_t)(N + 1) * 8);
        uint8_t *g_od = xmalloc((size_t)bytes + 1), *g_comp = xmalloc((size_t)P), *g_pst = xmalloc((size_t)P);
        int32_t *g_cnt = xmalloc((size_t)P * 12);
        down(g_oo, d_oo, (size_t)(P + 1) * 8);
        down(g_cdst, d_cdst, (size_t)(N + 1) * 8);
        down(g_comp, d_comp, (size_t)P);
        down(g_pst, d_pst, (size_t)P);
        down(g_cnt, d_cnt, (size_t)P * 12);
        const int64_t tot = w_oo[P];
        down(g_od, d_od, (size_t)tot);
        EXPECT(memcmp(g_oo, w_oo, (size_t)(P + 1) * 8) == 0, "slot offsets");
        EXPECT(memcmp(g_cdst, w_cdst, (size_t)(N + 1) * 8) == 0, "child positions");
        EXPECT(memcmp(g_cnt, w_cnt, (size_t)P * 12) == 0, "per-state counts");
        EXPECT(memcmp(g_comp, w_comp, (size_t)P) == 0 && memcmp(g_pst, w_pst, (size_t)P) == 0, "completion");
        EXPECT(memcmp(g_od, w_od, (size_t)tot) == 0, "slot bytes");
        free(w_oo); free(w_cdst); free(w_od); free(w_comp); free(w_pst); free(w_cnt);
        free(g_oo); free(g_cdst); free(g_od); free(g_comp); free(g_pst); free(g_cnt);
    }
    HIP_OK(hipStreamSynchronize(st));
    HIP_OK(hipFree(d_counts)); HIP_OK(hipFree(d_off)); HIP_OK(hipFree(d_cp)); HIP_OK(hipFree(d_co));
    HIP_OK(hipFree(d_q)); HIP_OK(hipFree(d_keep)); HIP_OK(hipFree(d_bc)); HIP_OK(hipFree(d_bp));
    HIP_OK(hipFree(d_bo)); HIP_OK(hipFree(d_sc)); HIP_OK(hipFree(d_rp)); HIP_OK(hipFree(d_ro));
    HIP_OK(hipFree(d_rs)); HIP_OK(hipFree(d_data)); HIP_OK(hipFree(d_roff)); HIP_OK(hipFree(d_oo));
    HIP_OK(hipFree(d_od)); HIP_OK(hipFree(d_cnt)); HIP_OK(hipFree(d_comp)); HIP_OK(hipFree(d_pst));
    HIP_OK(hipFree(d_cdst));
    free(counts); free(queue); free(keep); free(offs); free(cp); free(co); free(bc); free(bp); free(bo);
    free(g_offs); free(g_cp); free(g_co); free(g_bc); free(g_bp); free(g_bo); free(order); free(rp);
    free(ro_); free(rs); free(roff); free(data);
}

/* A random expansion: counts in [0, kmax), its offsets and lineage tags by
 * the oracle, and the same offsets on the device. */
typedef struct {
    int64_t P, N;
    int32_t *counts;
    int64_t *offs;
    uint32_t *cp, *co;
    int64_t *d_offs;
} expansion;

static expansion make_expansion(int64_t P, int kmax)
{
    expansion x;
    x.P = P;
    x.N = 0;
    x.counts = xmalloc((size_t)P * 4);
    for (int64_t p = 0; p < P; ++p) { x.counts[p] = (int32_t)below(kmax); x.N += x.counts[p]; }
    x.offs = xmalloc((size_t)(P + 1) * 8);
    x.cp = xmalloc((size_t)x.N * 4);
    x.co = xmalloc((size_t)x.N * 4);
    if (oracle_expand(x.counts, P, x.offs, x.cp, x.co, x.N) != 0) exit(4);
    x.d_offs = dmalloc((size_t)(P + 1) * 8);
    up(x.d_offs, x.offs, (size_t)(P + 1) * 8);
    return x;
}

static void free_expansion(expansion *x)
{
    HIP_OK(hipFree(x->d_offs));
    free(x->counts); free(x->offs); free(x->cp); free(x->co);
}

/* A gather whose output is its own report bytes: reports in canonical order,
 * failed and skipped ones without bytes, so every record already sits at its
 * output position; the result equals the oracle's and nothing moves.  Then
 * one failed report holding bytes shifts every later record: RO_EINVAL. */
static void case_in_place(ro_ctx *ctx, int64_t P)
{
    expansion x = make_expansion(P, 9);
    const int64_t N = x.N;
    uint8_t *rs = xmalloc((size_t)N);
    int64_t *roff = xmalloc((size_t)(N + 1) * 8);
    static const uint8_t states[5] = {RO_SUCCESS, RO_SUCCESS, RO_SUCCESS, RO_FAILED, RO_SKIPPED};
    int64_t bad = -1;
    for (int64_t c = 0; c < N; ++c) {
        rs[c] = states[below(5)];
        if (rs[c] == RO_FAILED && bad < 0 && c >= N / 3) bad = c;
    }
    uint32_t *d_rp = dmalloc((size_t)N * 4), *d_ro = dmalloc((size_t)N * 4);
    uint8_t *d_rs = dmalloc((size_t)N);
    int64_t *d_roff = dmalloc((size_t)(N + 1) * 8), *d_oo = dmalloc((size_t)(P + 1) * 8);
    int32_t *d_cnt = dmalloc((size_t)P * 12);
    uint8_t *d_comp = dmalloc((size_t)P), *d_pst = dmalloc((size_t)P);
    up(d_rp, x.cp, (size_t)N * 4);
    up(d_ro, x.co, (size_t)N * 4);
    up(d_rs, rs, (size_t)N);
    for (int moved = 0; moved < 2; ++moved) {
        roff[0] = 0;
        for (int64_t c = 0; c < N; ++c)
            roff[c + 1] = roff[c] + (rs[c] == RO_SUCCESS ? below(50) : (moved && c == bad ? 5 : 0));
        const int64_t bytes = roff[N];
        uint8_t *data = xmalloc((size_t)bytes + 16);
        for (int64_t i = 0; i < bytes + 16; ++i) data[i] = (uint8_t)rnd();
        uint8_t *d_data = dmalloc((size_t)bytes + 16);
        up(d_data, data, (size_t)bytes + 16);
        up(d_roff, roff, (size_t)(N + 1) * 8);
        ro_reports r = {d_rp, d_ro, d_rs, d_roff, d_data, N};
        ro_gather_out o;
        memset(&o, 0, sizeof o);
        o.out_off = d_oo;
        o.out_data = d_data;                 /* the report bytes themselves */
        o.out_cap = bytes + 16;
        o.n_success = d_cnt;
        o.n_failed = d_cnt + P;
        o.n_skipped = d_cnt + 2 * P;
        o.complete = d_comp;
        o.parent_state = d_pst;
        RO_OK_(ro_gather(ctx, &r, x.d_offs, P, &o));
        const int status = ro_ctx_status(ctx);
        if (moved) {
            EXPECT(bad < 0 || status == RO_EINVAL, "in-place gather with a record to move is RO_EINVAL");
        } else {
            EXPECT(status == RO_OK, "in-place gather status");
            int64_t *w_oo = xmalloc((size_t)(P + 1) * 8), *g_oo = xmalloc((size_t)(P + 1) * 8);
            uint8_t *w_od = xmalloc((size_t)bytes + 1), *g_od = xmalloc((size_t)bytes + 16);
            int32_t *w_cnt = xmalloc((size_t)P * 12), *g_cnt = xmalloc((size_t)P * 12);
            uint8_t *w_comp = xmalloc((size_t)P), *w_pst = xmalloc((size_t)P);
            uint8_t *g_comp = xmalloc((size_t)P), *g_pst = xmalloc((size_t)P);
            if (oracle_gather(x.cp, x.co, rs, roff, data, N, x.offs, P, w_oo, w_od, bytes, w_cnt, w_cnt + P,
                              w_cnt + 2 * P, w_comp, w_pst, NULL, NULL, NULL) != 0)
                exit(4);
            down(g_oo, d_oo, (size_t)(P + 1) * 8);
            down(g_od, d_data, (size_t)bytes + 16);
            down(g_cnt, d_cnt, (size_t)P * 12);
            down(g_comp, d_comp, (size_t)P);
            down(g_pst, d_pst, (size_t)P);
            EXPECT(memcmp(g_oo, w_oo, (size_t)(P + 1) * 8) == 0 && w_oo[P] == bytes, "in-place slot offsets");
            EXPECT(memcmp(g_cnt, w_cnt, (size_t)P * 12) == 0, "in-place counts");
            EXPECT(memcmp(g_comp, w_comp, (size_t)P) == 0 && memcmp(g_pst, w_pst, (size_t)P) == 0,
                   "in-place completion");
            EXPECT(memcmp(g_od, w_od, (size_t)bytes) == 0 && memcmp(g_od, data, (size_t)bytes + 16) == 0,
                   "in-place bytes: the oracle's slots, nothing moved");
            free(w_oo); free(g_oo); free(w_od); free(g_od); free(w_cnt); free(g_cnt);
            free(w_comp); free(w_pst); free(g_comp); free(g_pst);
        }
        HIP_OK(hipStreamSynchronize(g_st));
        HIP_OK(hipFree(d_data));
        free(data);
    }
    HIP_OK(hipFree(d_rp)); HIP_OK(hipFree(d_ro)); HIP_OK(hipFree(d_rs)); HIP_OK(hipFree(d_roff));
    HIP_OK(hipFree(d_oo)); HIP_OK(hipFree(d_cnt)); HIP_OK(hipFree(d_comp)); HIP_OK(hipFree(d_pst));
    free(rs); free(roff);
    free_expansion(&x);
}

/* Parent-bound reservations against the oracle. */
static void case_batch_parent(ro_ctx *ctx, int64_t P, int32_t B)
{
    expansion x = make_expansion(P, 9);
    const int64_t N = x.N;
    uint32_t *queue = xmalloc((size_t)N * 4);
    uint8_t *keep = xmalloc((size_t)N);
    for (int64_t i = 0; i < N; ++i) { queue[i] = (uint32_t)i; keep[i] = below(6) != 0; }
    shuffle(queue, N);
    uint32_t *w_c = xmalloc((size_t)N * 4), *w_p = xmalloc((size_t)N * 4), *w_o = xmalloc((size_t)N * 4);
    int64_t *w_sz = xmalloc((size_t)(N + 1) * 8), M = 0, nb = 0;
    if (oracle_batch_parent(queue, keep, N, x.offs, P, B, w_c, w_p, w_o, N, &M, &nb, w_sz, NULL) != 0) exit(4);

    uint32_t *d_q = dmalloc((size_t)N * 4), *d_c = dmalloc((size_t)N * 4), *d_p = dmalloc((size_t)N * 4);
    uint32_t *d_o = dmalloc((size_t)N * 4);
    uint8_t *d_k = dmalloc((size_t)N);
    int64_t *d_boff = dmalloc((size_t)(N + 2) * 8), *d_sc = dmalloc(16);
    up(d_q, queue, (size_t)N * 4);
    up(d_k, keep, (size_t)N);
    RO_OK_(ro_batch_parent(ctx, d_q, d_k, N, x.d_offs, P, B, d_c, d_p, d_o, N, d_boff, N + 2, d_sc, d_sc + 1, NULL));
    EXPECT(ro_ctx_status(ctx) == RO_OK, "parent-bound status");
    int64_t sc[2];
    down(sc, d_sc, 16);
    EXPECT(sc[0] == M && sc[1] == nb, "parent-bound counts");
    uint32_t *g = xmalloc((size_t)N * 4);
    down(g, d_c, (size_t)M * 4);
    EXPECT(memcmp(g, w_c, (size_t)M * 4) == 0, "parent-bound children");
    down(g, d_p, (size_t)M * 4);
    EXPECT(memcmp(g, w_p, (size_t)M * 4) == 0, "parent-bound parents");
    down(g, d_o, (size_t)M * 4);
    EXPECT(memcmp(g, w_o, (size_t)M * 4) == 0, "parent-bound ordinals");
    int64_t *boff = xmalloc((size_t)(nb + 1) * 8);
    down(boff, d_boff, (size_t)(nb + 1) * 8);
    int64_t at = 0;
    for (int64_t j = 0; j < nb; ++j) {
        EXPECT(boff[j] == at, "batch offsets");
        at += w_sz[j];
    }
    EXPECT(boff[nb] == M, "last batch offset");
    HIP_OK(hipStreamSynchronize(g_st));
    HIP_OK(hipFree(d_q)); HIP_OK(hipFree(d_c)); HIP_OK(hipFree(d_p)); HIP_OK(hipFree(d_o));
    HIP_OK(hipFree(d_k)); HIP_OK(hipFree(d_boff)); HIP_OK(hipFree(d_sc));
    free(queue); free(keep); free(w_c); free(w_p); free(w_o); free(w_sz); free(g); free(boff);
    free_expansion(&x);
}

/* A stream fed in `waves` waves, every emission against the oracle's. */
static void case_stream(ro_ctx *ctx, int64_t P, int waves)
{
    expansion x = make_expansion(P, 6);
    const int64_t N = x.N;
    uint32_t *order = xmalloc((size_t)N * 4);
    for (int64_t i = 0; i < N; ++i) order[i] = (uint32_t)i;
    shuffle(order, N);
    uint32_t *rp = xmalloc((size_t)N * 4), *ro_ = xmalloc((size_t)N * 4);
    uint8_t *rs = xmalloc((size_t)N);
    int64_t *roff = xmalloc((size_t)(N + 1) * 8);
    roff[0] = 5;
    for (int64_t i = 0; i < N; ++i) {
        rp[i] = x.cp[order[i]];
        ro_[i] = x.co[order[i]];
        rs[i] = (uint8_t)(below(8) == 0 ? RO_FAILED : (below(8) == 0 ? RO_SKIPPED : RO_SUCCESS));
        roff[i + 1] = roff[i] + below(50);
    }
    const int64_t bytes = roff[N];
    uint8_t *arena = xmalloc((size_t)bytes + 16);
    for (int64_t i = 0; i < bytes + 16; ++i) arena[i] = (uint8_t)rnd();
    uint32_t *d_rp = dmalloc((size_t)N * 4), *d_ro = dmalloc((size_t)N * 4);
    uint8_t *d_rs = dmalloc((size_t)N), *d_arena = dmalloc((size_t)bytes + 16);
    int64_t *d_roff = dmalloc((size_t)(N + 1) * 8);
    up(d_rp, rp, (size_t)N * 4);
    up(d_ro, ro_, (size_t)N * 4);
    up(d_rs, rs, (size_t)N);
    up(d_roff, roff, (size_t)(N + 1) * 8);
    up(d_arena, arena, (size_t)bytes + 16);

    ro_stream *s = NULL;
    RO_OK_(ro_stream_create(ctx, x.d_offs, P, N, NULL, &s));
    oracle_stream *os = oracle_stream_create(x.offs, P);
    if (!os) exit(4);
    uint32_t *d_ep = dmalloc((size_t)P * 4), *w_ep = xmalloc((size_t)P * 4), *g_ep = xmalloc((size_t)P * 4);
    int64_t *d_eo = dmalloc((size_t)(P + 1) * 8), *w_eo = xmalloc((size_t)(P + 1) * 8);
    int64_t *g_eo = xmalloc((size_t)(P + 1) * 8), *d_sc = dmalloc(16);
    uint8_t *d_ed = dmalloc((size_t)bytes + 1), *w_ed = xmalloc((size_t)bytes + 1), *g_ed = xmalloc((size_t)bytes + 1);
    int32_t *d_cnt = dmalloc((size_t)P * 12), *w_cnt = xmalloc((size_t)P * 12), *g_cnt = xmalloc((size_t)P * 12);
    uint8_t *d_pst = dmalloc((size_t)P), *w_pst = xmalloc((size_t)P), *g_pst = xmalloc((size_t)P);
    int64_t lo = 0, total_emitted = 0;
    for (int w = 0; w < waves; ++w) {
        const int64_t hi = N * (w + 1) / waves;
        ro_reports r = {d_rp + lo, d_ro + lo, d_rs + lo, d_roff + lo, d_arena, hi - lo};
        RO_OK_(ro_stream_report(ctx, s, &r, NULL));
        RO_OK_(ro_stream_emit(ctx, s, d_ep, d_eo, d_ed, P, bytes, d_cnt, d_cnt + P, d_cnt + 2 * P, d_pst, d_sc,
                              d_sc + 1));
        EXPECT(ro_ctx_status(ctx) == RO_OK, "stream status");
        int64_t rej = 0, ne = 0, nb = 0;
        if (oracle_stream_report(os, rp + lo, ro_ + lo, rs + lo, roff + lo, arena, hi - lo, &rej) != 0) exit(4);
        if (oracle_stream_emit(os, w_ep, w_eo, w_ed, P, bytes, w_cnt, w_cnt + P, w_cnt + 2 * P, w_pst, &ne, &nb) != 0)
            exit(4);
        int64_t sc[2];
        down(sc, d_sc, 16);
        EXPECT(sc[0] == ne && sc[1] == nb, "emitted parents and bytes");
        down(g_ep, d_ep, (size_t)ne * 4);
        down(g_eo, d_eo, (size_t)(ne + 1) * 8);
        down(g_ed, d_ed, (size_t)nb);
        down(g_cnt, d_cnt, (size_t)P * 12);
        down(g_pst, d_pst, (size_t)ne);
        EXPECT(memcmp(g_ep, w_ep, (size_t)ne * 4) == 0, "emitted parents");
        EXPECT(memcmp(g_eo, w_eo, (size_t)(ne + 1) * 8) == 0, "emitted slot offsets");
        EXPECT(memcmp(g_ed, w_ed, (size_t)nb) == 0, "emitted bytes");
        for (int k = 0; k < 3; ++k)
            EXPECT(memcmp(g_cnt + k * P, w_cnt + k * P, (size_t)ne * 4) == 0, "emitted counts");
        EXPECT(memcmp(g_pst, w_pst, (size_t)ne) == 0, "emitted states");
        total_emitted += ne;
        lo = hi;
    }
    EXPECT(total_emitted == P, "every parent emitted once");
    RO_OK_(ro_stream_destroy(s));
    oracle_stream_destroy(os);
    HIP_OK(hipFree(d_rp)); HIP_OK(hipFree(d_ro)); HIP_OK(hipFree(d_rs)); HIP_OK(hipFree(d_arena));
    HIP_OK(hipFree(d_roff)); HIP_OK(hipFree(d_ep)); HIP_OK(hipFree(d_eo)); HIP_OK(hipFree(d_sc));
    HIP_OK(hipFree(d_ed)); HIP_OK(hipFree(d_cnt)); HIP_OK(hipFree(d_pst));
    free(order); free(rp); free(ro_); free(rs); free(roff); free(arena); free(w_ep); free(g_ep); free(w_eo);
    free(g_eo); free(w_ed); free(g_ed); free(w_cnt); free(g_cnt); free(w_pst); free(g_pst);
    free_expansion(&x);
}

/* F.filter over n items and a two-level F.broadcast, against the oracle. */
static void case_filter_broadcast(ro_ctx *ctx, int64_t P)
{
    expansion up1 = make_expansion(P, 5);             /* top -> mid */
    expansion up2 = make_expansion(up1.N, 5);         /* mid -> leaf */
    const int64_t n = up2.N;
    uint8_t *xs = xmalloc((size_t)n), *ms = xmalloc((size_t)n), *mk = xmalloc((size_t)n);
    uint8_t *top = xmalloc((size_t)P), *w = xmalloc((size_t)n), *g = xmalloc((size_t)n);
    for (int64_t i = 0; i < n; ++i) { xs[i] = (uint8_t)below(4); ms[i] = (uint8_t)below(4); mk[i] = (uint8_t)below(2); }
    for (int64_t p = 0; p < P; ++p) top[p] = (uint8_t)below(4);
    uint8_t *d_xs = dmalloc((size_t)n), *d_ms = dmalloc((size_t)n), *d_mk = dmalloc((size_t)n), *d_out = dmalloc((size_t)n);
    uint8_t *d_top = dmalloc((size_t)P);
    up(d_xs, xs, (size_t)n);
    up(d_ms, ms, (size_t)n);
    up(d_mk, mk, (size_t)n);
    up(d_top, top, (size_t)P);
    RO_OK_(ro_filter(ctx, d_xs, d_ms, d_mk, n, d_out));
    EXPECT(ro_ctx_status(ctx) == RO_OK, "filter status");
    if (oracle_filter(xs, ms, mk, n, w) != 0) exit(4);
    down(g, d_out, (size_t)n);
    EXPECT(memcmp(g, w, (size_t)n) == 0, "filter states");

    uint32_t *d_m0 = dmalloc((size_t)n * 4), *d_m1 = dmalloc((size_t)up1.N * 4), *d_anc = dmalloc((size_t)n * 4);
    up(d_m0, up2.cp, (size_t)n * 4);
    up(d_m1, up1.cp, (size_t)up1.N * 4);
    const uint32_t *dmaps[2] = {d_m0, d_m1};
    const uint32_t *hmaps[2] = {up2.cp, up1.cp};
    const int64_t lens[2] = {n, up1.N};
    RO_OK_(ro_broadcast(ctx, dmaps, lens, 2, n, d_top, P, d_xs, d_anc, d_out));
    EXPECT(ro_ctx_status(ctx) == RO_OK, "broadcast status");
    uint32_t *w_anc = xmalloc((size_t)n * 4), *g_anc = xmalloc((size_t)n * 4);
    if (oracle_broadcast(hmaps, 2, n, top, P, xs, w_anc, w) != 0) exit(4);
    down(g, d_out, (size_t)n);
    down(g_anc, d_anc, (size_t)n * 4);
    EXPECT(memcmp(g, w, (size_t)n) == 0 && memcmp(g_anc, w_anc, (size_t)n * 4) == 0, "broadcast");
    HIP_OK(hipStreamSynchronize(g_st));
    HIP_OK(hipFree(d_xs)); HIP_OK(hipFree(d_ms)); HIP_OK(hipFree(d_mk)); HIP_OK(hipFree(d_out));
    HIP_OK(hipFree(d_top)); HIP_OK(hipFree(d_m0)); HIP_OK(hipFree(d_m1)); HIP_OK(hipFree(d_anc));
    free(xs); free(ms); free(mk); free(top); free(w); free(g); free(w_anc); free(g_anc);
    free_expansion(&up1);
    free_expansion(&up2);
}

/* Grain phases and the fence: dispatch every child, commit 90% of them (with
 * identical repeats), retry the rest, dispatch them again and commit them
 * together with stale reports of the first attempt. */
static void case_grains(ro_ctx *ctx, int64_t P)
{
    expansion x = make_expansion(P, 6);
    const int64_t N = x.N;
    ro_grains *g = NULL;
    RO_OK_(ro_grains_create(ctx, N, &g));
    oracle_grains *og = oracle_grains_create(N);
    if (!og) exit(4);
    uint32_t *child = xmalloc((size_t)N * 4);
    for (int64_t i = 0; i < N; ++i) child[i] = (uint32_t)i;
    shuffle(child, N);
    uint32_t *d_child = dmalloc((size_t)N * 4), *d_gen = dmalloc((size_t)N * 4);
    uint32_t *w_gen = xmalloc((size_t)N * 4), *g_gen = xmalloc((size_t)N * 4);
    up(d_child, child, (size_t)N * 4);
    RO_OK_(ro_grains_dispatch(ctx, g, d_child, N, d_gen));
    if (oracle_grains_dispatch(og, child, N, w_gen) != 0) exit(4);
    down(g_gen, d_gen, (size_t)N * 4);
    EXPECT(memcmp(g_gen, w_gen, (size_t)N * 4) == 0, "dispatch generations");

    /* call 1: the first 90% in dispatch order, each possibly followed later by a repeat */
    const int64_t n1 = N * 9 / 10;
    const int64_t cap = 2 * N + 1;
    uint32_t *rp = xmalloc((size_t)cap * 4), *ro_ = xmalloc((size_t)cap * 4), *rg = xmalloc((size_t)cap * 4);
    uint8_t *rs = xmalloc((size_t)cap);
    int64_t *roff = xmalloc((size_t)(cap + 1) * 8);
    int64_t n = 0;
    roff[0] = 0;
    for (int64_t i = 0; i < n1; ++i) {
        const uint32_t c = child[i];
        rp[n] = x.cp[c]; ro_[n] = x.co[c]; rg[n] = 0; rs[n] = (uint8_t)(below(6) == 0 ? RO_FAILED : RO_SUCCESS);
        roff[n + 1] = roff[n] + (rs[n] == RO_SUCCESS ? 8 : 0);
        ++n;
    }
    const int64_t firsts = n;
    for (int64_t i = 0; i < firsts; ++i) {
        if (below(10) != 0) continue;
        rp[n] = rp[i]; ro_[n] = ro_[i]; rg[n] = 0; rs[n] = rs[i];
        roff[n + 1] = roff[n] + (roff[i + 1] - roff[i]);
        ++n;
    }
    int64_t bytes = roff[n];
    const size_t data_cap = (size_t)(8 * cap) + 16;          /* both calls' bytes fit */
    uint8_t *data = xmalloc(data_cap);
    for (int64_t i = 0; i < firsts; ++i)
        for (int64_t b = roff[i]; b < roff[i + 1]; ++b) data[b] = (uint8_t)(rp[i] * 31u + ro_[i] * 7u + (uint32_t)b);
    for (int64_t i = firsts, j = 0; i < n; ++i) {
        while (!(rp[j] == rp[i] && ro_[j] == ro_[i])) ++j;     /* the repeat copies its original's bytes */
        memcpy(data + roff[i], data + roff[j], (size_t)(roff[i + 1] - roff[i]));
    }
    uint32_t *d_rp = dmalloc((size_t)cap * 4), *d_ro = dmalloc((size_t)cap * 4), *d_rg = dmalloc((size_t)cap * 4);
    uint8_t *d_rs = dmalloc((size_t)cap), *d_so = dmalloc((size_t)cap), *d_data = dmalloc(data_cap);
    int64_t *d_roff = dmalloc((size_t)(cap + 1) * 8), *d_cnt = dmalloc(32);
    uint8_t *w_so = xmalloc((size_t)cap), *g_so = xmalloc((size_t)cap);
    int64_t w_cnt[4], g_cnt[4];
    for (int call = 0; call < 2; ++call) {
        up(d_rp, rp, (size_t)n * 4);
        up(d_ro, ro_, (size_t)n * 4);
        up(d_rg, rg, (size_t)n * 4);
        up(d_rs, rs, (size_t)n);
        up(d_roff, roff, (size_t)(n + 1) * 8);
        up(d_data, data, (size_t)bytes);
        ro_reports r = {d_rp, d_ro, d_rs, d_roff, d_data, n};
        RO_OK_(ro_grains_commit(ctx, g, &r, d_rg, x.d_offs, P, d_so, d_cnt));
        EXPECT(ro_ctx_status(ctx) == RO_OK, "commit status");
        if (oracle_grains_commit(og, rp, ro_, rs, roff, data, rg, n, x.offs, P, w_so, w_cnt) != 0) exit(4);
        down(g_so, d_so, (size_t)n);
        down(g_cnt, d_cnt, 32);
        EXPECT(memcmp(g_so, w_so, (size_t)n) == 0, "commit outcomes");
        EXPECT(memcmp(g_cnt, w_cnt, 32) == 0, "commit counts");
        if (call == 1) break;
        /* retry the lost 10% and dispatch them again at generation 1 */
        const int64_t nl = N - n1;
        RO_OK_(ro_grains_retry(ctx, g, d_child + n1, nl));
        RO_OK_(ro_grains_dispatch(ctx, g, d_child + n1, nl, d_gen));
        if (oracle_grains_retry(og, child + n1, nl) != 0 || oracle_grains_dispatch(og, child + n1, nl, w_gen) != 0)
            exit(4);
        EXPECT(ro_ctx_status(ctx) == RO_OK, "retry status");
        down(g_gen, d_gen, (size_t)nl * 4);
        EXPECT(memcmp(g_gen, w_gen, (size_t)nl * 4) == 0, "retry generations");
        /* call 2: the retried children at generation 1, and stale generation-0 reports of some */
        n = 0;
        for (int64_t i = n1; i < N; ++i) {
            const uint32_t c = child[i];
            rp[n] = x.cp[c]; ro_[n] = x.co[c]; rg[n] = 1; rs[n] = RO_SUCCESS;
            roff[n + 1] = roff[n] + 4;
            ++n;
            if (below(2) == 0) {
                rp[n] = x.cp[c]; ro_[n] = x.co[c]; rg[n] = 0; rs[n] = RO_FAILED;
                roff[n + 1] = roff[n];
                ++n;
            }
        }
        bytes = roff[n];
        for (int64_t b = 0; b < bytes; ++b) data[b] = (uint8_t)rnd();
    }
    uint32_t *g_ph = xmalloc((size_t)N * 4);
    uint32_t *d_ph = dmalloc((size_t)N * 4);
    RO_OK_(ro_grains_read(ctx, g, d_ph, d_gen));
    down(g_ph, d_ph, (size_t)N * 4);
    down(g_gen, d_gen, (size_t)N * 4);
    const uint8_t *w_ph = oracle_grains_phase(og);
    const uint32_t *w_g = oracle_grains_gen(og);
    for (int64_t c = 0; c < N; ++c)
        EXPECT(g_ph[c] == w_ph[c] && g_gen[c] == w_g[c], "final phases and generations");
    HIP_OK(hipStreamSynchronize(g_st));
    RO_OK_(ro_grains_destroy(g));
    oracle_grains_destroy(og);
    HIP_OK(hipFree(d_child)); HIP_OK(hipFree(d_gen)); HIP_OK(hipFree(d_rp)); HIP_OK(hipFree(d_ro));
    HIP_OK(hipFree(d_rg)); HIP_OK(hipFree(d_rs)); HIP_OK(hipFree(d_so)); HIP_OK(hipFree(d_data));
    HIP_OK(hipFree(d_roff)); HIP_OK(hipFree(d_cnt)); HIP_OK(hipFree(d_ph));
    free(child); free(w_gen); free(g_gen); free(rp); free(ro_); free(rg); free(rs); free(roff); free(data);
    free(w_so); free(g_so); free(g_ph);
    free_expansion(&x);
}

int main(void)
{
    hipStream_t st;
    HIP_OK(hipSetDevice(0));
    HIP_OK(hipStreamCreateWithFlags(&st, hipStreamNonBlocking));
    g_st = st;
    ro_ctx *ctx = NULL;
    RO_OK_(ro_ctx_create(&ctx, (void *)st));
    static const int64_t sizes[] = {1, 7, 300, 1500, 5000, 20000};
    static const int32_t bs[] = {1, 3, 64, 7, 256, 1000};
    for (case_id = 0; case_id < 6; ++case_id) {
        printf("case %d: %ld parents, B = %d\n", case_id, (long)sizes[case_id], bs[case_id]);
        fflush(stdout);
        one_case(ctx, st, sizes[case_id], bs[case_id], 0);
    }
    printf("case %d: planted error\n", case_id);
    fflush(stdout);
    one_case(ctx, st, 500, 16, 1);
    ++case_id;
    printf("case %d: after the error\n", case_id);
    fflush(stdout);
    one_case(ctx, st, 800, 5, 0);
    ++case_id;
    printf("case %d: gather in place\n", case_id);
    fflush(stdout);
    case_in_place(ctx, 4000);
    ++case_id;
    printf("case %d: parent-bound reservation\n", case_id);
    fflush(stdout);
    case_batch_parent(ctx, 3000, 5);
    ++case_id;
    printf("case %d: stream, 4 waves\n", case_id);
    fflush(stdout);
    case_stream(ctx, 2000, 4);
    ++case_id;
    printf("case %d: filter and broadcast\n", case_id);
    fflush(stdout);
    case_filter_broadcast(ctx, 700);
    ++case_id;
    printf("case %d: grains and the fence\n", case_id);
    fflush(stdout);
    case_grains(ctx, 2500);
    ++case_id;
    printf("case %d: per-kernel trace\n", case_id);
    fflush(stdout);
    {
        int64_t launches[RO_K_COUNT];
        double ms[RO_K_COUNT];
        memset(launches, 0, sizeof launches);
        memset(ms, 0, sizeof ms);
        RO_OK_(ro_ctx_trace(ctx, 1));
        one_case(ctx, st, 100, 4, 0);
        RO_OK_(ro_ctx_trace(ctx, 0));
        RO_OK_(ro_ctx_trace_read(ctx, launches, ms, RO_K_COUNT));
        EXPECT(launches[RO_K_EXPAND_SCAN] >= 1 && launches[RO_K_GATHER_COPY] >= 1 && ms[RO_K_GATHER_COPY] >= 0.0,
               "trace records the launches");
    }
    RO_OK_(ro_ctx_destroy(ctx));
    HIP_OK(hipStreamDestroy(st));
    printf("c abi ok\n");
    return 0;
}
