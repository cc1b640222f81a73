/*
 * Test infrastructure: the library used from plain C, with no Python and no
 * torch.  Device memory and the stream come from the HIP runtime directly;
 * ro_expand, ro_batch and ro_gather run on seeded random cases and every
 * output is compared with the C oracle (linked from oracle/) bit for bit.
 * One more case plants a report with an out-of-range ordinal and checks that
 * ro_ctx_status returns RO_ERANGE, then that the context works again.
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
static void up(void *d, const void *h, size_t n) { if (n) HIP_OK(hipMemcpy(d, h, n, hipMemcpyHostToDevice)); }
static void down(void *h, const void *d, size_t n) { if (n) HIP_OK(hipMemcpy(h, d, n, hipMemcpyDeviceToHost)); }
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

int main(void)
{
    hipStream_t st;
    HIP_OK(hipSetDevice(0));
    HIP_OK(hipStreamCreateWithFlags(&st, hipStreamNonBlocking));
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
    RO_OK_(ro_ctx_destroy(ctx));
    HIP_OK(hipStreamDestroy(st));
    printf("c abi ok\n");
    return 0;
}
