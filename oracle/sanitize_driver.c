/*
 * Test infrastructure: drives every oracle entry point on seeded random
 * inputs (and on the error paths) so that a build with AddressSanitizer and
 * UndefinedBehaviorSanitizer can check the oracle's own memory and integer
 * behaviour.  It checks no result values: the pins do that.  Exit status 0
 * means every call returned and no sanitizer fired.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

typedef struct oracle_stream oracle_stream;
typedef struct oracle_grains oracle_grains;
int oracle_expand(const int32_t *, int64_t, int64_t *, uint32_t *, uint32_t *, int64_t);
int oracle_batch(const uint32_t *, const uint8_t *, int64_t, const int64_t *, int64_t, int32_t, uint32_t *,
                 uint32_t *, uint32_t *, int64_t, int64_t *, int64_t *, int64_t *, const uint8_t *);
int oracle_batch_parent(const uint32_t *, const uint8_t *, int64_t, const int64_t *, int64_t, int32_t, uint32_t *,
                        uint32_t *, uint32_t *, int64_t, int64_t *, int64_t *, int64_t *, const uint8_t *);
int oracle_gather(const uint32_t *, const uint32_t *, const uint8_t *, const int64_t *, const uint8_t *, int64_t,
                  const int64_t *, int64_t, int64_t *, uint8_t *, int64_t, int32_t *, int32_t *, int32_t *,
                  uint8_t *, uint8_t *, int64_t *, uint8_t *, int64_t *);
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
int oracle_grains_dispatch(oracle_grains *, const uint32_t *, int64_t, uint32_t *);
int oracle_grains_retry(oracle_grains *, const uint32_t *, int64_t);
int oracle_grains_commit(oracle_grains *, const uint32_t *, const uint32_t *, const uint8_t *, const int64_t *,
                         const uint8_t *, const uint32_t *, int64_t, const int64_t *, int64_t, uint8_t *,
                         int64_t *);

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static uint64_t rnd(void)          /* xorshift64* */
{
    rng_state ^= rng_state >> 12;
    rng_state ^= rng_state << 25;
    rng_state ^= rng_state >> 27;
    return rng_state * 0x2545F4914F6CDD1Dull;
}
static int64_t rint_(int64_t n) { return n > 0 ? (int64_t)(rnd() % (uint64_t)n) : 0; }

static void *xmalloc(size_t n) { void *p = malloc(n ? n : 1); if (!p) exit(3); return p; }

static void shuffle(uint32_t *a, int64_t n)
{
    for (int64_t i = n - 1; i > 0; --i) {
        int64_t j = rint_(i + 1);
        uint32_t t = a[i]; a[i] = a[j]; a[j] = t;
    }
}

static void one_case(int64_t P, int32_t B)
{
    int32_t *counts = xmalloc(sizeof(int32_t) * (size_t)P);
    for (int64_t p = 0; p < P; ++p) counts[p] = (int32_t)rint_(7);
    int64_t *offs = xmalloc(sizeof(int64_t) * (size_t)(P + 1));
    if (oracle_expand(counts, P, offs, NULL, NULL, 0)) exit(4);
    int64_t N = offs[P];
    uint32_t *cp = xmalloc(4 * (size_t)N), *co = xmalloc(4 * (size_t)N);
    if (oracle_expand(counts, P, offs, cp, co, N)) exit(4);
    (void)oracle_expand(counts, P, offs, cp, co, N - 1 < 0 ? 0 : N - 1);     /* capacity error path */

    uint32_t *queue = xmalloc(4 * (size_t)N);
    uint8_t *keep = xmalloc((size_t)N), *bar = xmalloc((size_t)P);
    for (int64_t i = 0; i < N; ++i) { queue[i] = (uint32_t)i; keep[i] = rint_(10) != 0; }
    shuffle(queue, N);
    for (int64_t p = 0; p < P; ++p) bar[p] = rint_(5) == 0;
    uint32_t *oc = xmalloc(4 * (size_t)N), *op = xmalloc(4 * (size_t)N), *oo = xmalloc(4 * (size_t)N);
    int64_t *sizes = xmalloc(8 * (size_t)(N + 1));
    int64_t m = 0, nb = 0;
    for (int pol = 0; pol < 2; ++pol) {
        int (*fn)(const uint32_t *, const uint8_t *, int64_t, const int64_t *, int64_t, int32_t, uint32_t *,
                  uint32_t *, uint32_t *, int64_t, int64_t *, int64_t *, int64_t *, const uint8_t *) =
            pol ? oracle_batch_parent : oracle_batch;
        if (fn(queue, keep, N, offs, P, B, oc, op, oo, N, &m, &nb, sizes, NULL)) exit(5);
        if (fn(queue, NULL, N, offs, P, B, oc, op, oo, N, &m, &nb, sizes, bar)) exit(5);
        (void)fn(queue, NULL, N, offs, P, B, oc, op, oo, N / 2, &m, &nb, sizes, NULL);   /* ECAP */
    }

    /* reports in batch order, some PENDING, random lengths */
    if (oracle_batch(queue, NULL, N, offs, P, B, oc, op, oo, N, &m, &nb, sizes, NULL)) exit(6);
    uint8_t *st = xmalloc((size_t)N);
    int64_t *roff = xmalloc(8 * (size_t)(N + 1));
    roff[0] = 0;
    for (int64_t i = 0; i < N; ++i) {
        st[i] = (uint8_t)rint_(4);
        roff[i + 1] = roff[i] + (st[i] == 0 ? rint_(40) : 0);
    }
    uint8_t *data = xmalloc((size_t)roff[N]);
    for (int64_t b = 0; b < roff[N]; ++b) data[b] = (uint8_t)rnd();
    int64_t *out_off = xmalloc(8 * (size_t)(P + 1)), *cdst = xmalloc(8 * (size_t)(N + 1));
    uint8_t *out = xmalloc((size_t)roff[N]);
    int32_t *ns = xmalloc(4 * (size_t)P), *nf = xmalloc(4 * (size_t)P), *nk = xmalloc(4 * (size_t)P);
    uint8_t *cpl = xmalloc((size_t)P), *pst = xmalloc((size_t)P), *gbar = xmalloc((size_t)P);
    memset(gbar, 0, (size_t)P);
    int64_t nrej = 0;
    if (oracle_gather(op, oo, st, roff, data, N, offs, P, out_off, out, roff[N], ns, nf, nk, cpl, pst, cdst, NULL,
                      NULL)) exit(7);
    uint8_t *st4 = xmalloc((size_t)N);
    for (int64_t i = 0; i < N; ++i) st4[i] = rint_(50) == 0 ? 4 : st[i];       /* some group failures */
    if (oracle_gather(op, oo, st4, roff, data, N, offs, P, out_off, out, roff[N], ns, nf, nk, cpl, pst, cdst, gbar,
                      &nrej)) exit(7);
    (void)oracle_gather(op, oo, st, roff, data, N, offs, P, out_off, out, roff[N] / 2, ns, nf, nk, cpl, pst, NULL,
                        NULL, NULL);                                            /* ECAP */
    if (N > 1) {                                                               /* duplicate */
        uint32_t sp = op[1], so = oo[1];
        op[1] = op[0]; oo[1] = oo[0];
        (void)oracle_gather(op, oo, st, roff, data, N, offs, P, out_off, out, roff[N], ns, nf, nk, cpl, pst, NULL,
                            NULL, NULL);
        op[1] = sp; oo[1] = so;
    }

    /* streaming: the same reports in three waves */
    oracle_stream *s = oracle_stream_create(offs, P);
    if (!s) exit(8);
    uint32_t *ep = xmalloc(4 * (size_t)(P + 1));
    int64_t *eoff = xmalloc(8 * (size_t)(P + 1));
    uint8_t *edata = xmalloc((size_t)roff[N] + 1);
    int64_t ne = 0, nbytes = 0;
    for (int w = 0; w < 3; ++w) {
        int64_t a = N * w / 3, b = N * (w + 1) / 3;
        int64_t *woff = xmalloc(8 * (size_t)(b - a + 1));
        for (int64_t i = a; i <= b; ++i) woff[i - a] = roff[i];
        if (oracle_stream_report(s, op + a, oo + a, st + a, woff, data, b - a, &nrej)) exit(9);
        if (oracle_stream_emit(s, ep, eoff, edata, P, roff[N], ns, nf, nk, pst, &ne, &nbytes)) exit(9);
        free(woff);
    }
    oracle_stream_destroy(s);

    /* filter and broadcast */
    uint8_t *xs = xmalloc((size_t)N), *ms = xmalloc((size_t)N), *mv = xmalloc((size_t)N), *fo = xmalloc((size_t)N);
    for (int64_t i = 0; i < N; ++i) { xs[i] = (uint8_t)rint_(4); ms[i] = (uint8_t)rint_(4); mv[i] = rnd() & 1; }
    if (oracle_filter(xs, ms, mv, N, fo)) exit(10);
    uint8_t *px = xmalloc((size_t)P);
    for (int64_t p = 0; p < P; ++p) px[p] = (uint8_t)rint_(4);
    const uint32_t *maps[1] = {cp};
    uint32_t *anc = xmalloc(4 * (size_t)N);
    if (oracle_broadcast(maps, 1, N, px, P, xs, anc, fo)) exit(11);
    (void)oracle_broadcast(maps, 1, N, px, P / 2, xs, anc, fo);                /* ERANGE */

    /* grains: dispatch all, commit with repeats and stale reports, retry the rest */
    oracle_grains *g = oracle_grains_create(N);
    if (!g) exit(12);
    uint32_t *gen = xmalloc(4 * (size_t)N), *rg = xmalloc(4 * (size_t)N);
    if (oracle_grains_dispatch(g, queue, N, gen)) exit(12);
    for (int64_t i = 0; i < N; ++i) rg[i] = rint_(6) == 0 ? 7u : 0u;
    uint8_t *so = xmalloc((size_t)N);
    int64_t gc[4];
    if (oracle_grains_commit(g, op, oo, st, roff, data, rg, N, offs, P, so, gc)) exit(13);
    if (oracle_grains_commit(g, op, oo, st, roff, data, rg, N, offs, P, so, gc)) exit(13);
    (void)oracle_grains_retry(g, queue, N);                                    /* sealed ones: ESTATE */
    oracle_grains_destroy(g);

    free(counts); free(offs); free(cp); free(co); free(queue); free(keep); free(bar); free(oc); free(op); free(oo);
    free(sizes); free(st); free(roff); free(data); free(out_off); free(cdst); free(out); free(ns); free(nf);
    free(nk); free(cpl); free(pst); free(gbar); free(st4); free(ep); free(eoff); free(edata); free(xs); free(ms);
    free(mv); free(fo); free(px); free(anc); free(gen); free(rg); free(so);
}

int main(void)
{
    const int64_t Ps[] = {0, 1, 2, 7, 50, 400};
    const int32_t Bs[] = {1, 3, 64};
    for (int rep = 0; rep < 4; ++rep)
        for (size_t i = 0; i < sizeof(Ps) / sizeof(Ps[0]); ++i)
            for (size_t j = 0; j < sizeof(Bs) / sizeof(Bs[0]); ++j)
                one_case(Ps[i], Bs[j]);
    printf("sanitize driver: ok\n");
    return 0;
}
