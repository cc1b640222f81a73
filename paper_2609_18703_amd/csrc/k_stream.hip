// Streaming completion on gfx950: reports arrive wave by wave; after each
// wave, every parent whose children are now all terminal is emitted once, in
// ascending parent order, with its ordered bytes, counts and state.
//
// RayOrch (arXiv 2609.18703): a parent can finalise and proceed as soon as all
// of its required child results are terminal (Sec. 1; Sec. 4 Reduce rule);
// facts are published once and conflicting repeats are rejected (Sec. 4,
// publication rules).
//
// Per wave:   report  -> canonical slots + seen bits + one count per report.
// Per emit:   select  -> ascending list of newly complete parents and the
//                        exclusive scan of their child counts (two look-back
//                        chains in one pass over all parents): a "virtual"
//                        expansion whose children are the emitted parents'
//                        children, in order;
//             vmap    -> canonical slot of every virtual child;
//             then the gather's canonical scan (slot offsets and per-state
//             counts of the emitted parents) and copy kernels run over the
//             virtual expansion, and finish closes the call.
#include "ro_device.h"

namespace ro {

constexpr uint32_t kStreamEpoch = 1;      // slot tag epoch of an accepted stream report

// Reports of a parent with many children would all add to one counter, and
// atomics on one address serialise.  A parent with at least kBig children
// counts into kSpread counters on separate lines instead, indexed by its
// first child >> kBigShift (two such parents never share that index, since
// each spans kBig children or more).
constexpr int kBigShift = 10;
constexpr int64_t kBig = (int64_t)1 << kBigShift;
constexpr int kSpread = 16;

int64_t stream_big_slots(int64_t N) { return (N >> kBigShift) + 1; }
int64_t stream_big_size(int64_t N) { return (int64_t)kSpread * stream_big_slots(N); }

__device__ __forceinline__ int64_t reported(const int32_t *__restrict__ cnt, const int32_t *__restrict__ big,
                                            int64_t nslots, int64_t p, int64_t st, int64_t k)
{
    if (k < kBig) return cnt[p];
    const int64_t j = st >> kBigShift;
    int64_t s = 0;
#pragma unroll
    for (int l = 0; l < kSpread; ++l) s += big[(int64_t)l * nslots + j];
    return s;
}

// Validates the expansion once: offsets[0] = 0, nondecreasing, offsets[P] = N.
__global__ void k_stream_check(const int64_t *__restrict__ offsets, int64_t P, int64_t N, Ctl *ctl)
{
    const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    bool bad = (g == 0) && (offsets[0] != 0 || offsets[P] != N);
    for (int64_t p = g; p < P; p += (int64_t)gridDim.x * blockDim.x)
        if (offsets[p + 1] < offsets[p]) bad = true;
    if (bad) raise_err(ctl, RO_EINVAL);
}

__global__ __launch_bounds__(kBlock) void k_stream_report(
    const uint32_t *__restrict__ rp, const uint32_t *__restrict__ ro_, const uint8_t *__restrict__ rs,
    const int64_t *__restrict__ roff, const uint8_t *data, int64_t n, const int64_t *__restrict__ offsets,
    int64_t P, int64_t N, Canon *__restrict__ canon, uint32_t *__restrict__ seen, int32_t *__restrict__ cnt,
    int32_t *__restrict__ big, int64_t nslots, Ctl *ctl)
{
    const int64_t gtid = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    const int64_t gstride = (int64_t)gridDim.x * kBlock;
    const int64_t spread = (int64_t)(((blockIdx.x << 2) + (threadIdx.x >> 6)) & (kSpread - 1)) * nslots;
    int err = 0;
    if (gtid == 0 && n > 0 && roff[0] < 0) err = RO_EINVAL;
    for (int64_t i = gtid; i < n; i += gstride) {
        const uint32_t s = rs[i];
        const int64_t o0 = roff[i], o1 = roff[i + 1];
        if (o1 < o0) { err = RO_EINVAL; continue; }
        if (s > RO_PENDING) { err = RO_ESTATE; continue; }
        if (s == RO_PENDING) continue;
        const uint32_t p = rp[i];
        if ((int64_t)p >= P) { err = RO_ERANGE; continue; }
        const int64_t st = offsets[p];
        const int64_t k = offsets[p + 1] - st;
        const uint32_t o = ro_[i];
        if ((int64_t)o >= k) { err = RO_ERANGE; continue; }
        const int64_t c = st + (int64_t)o;
        if (st < 0 || c >= N) { err = RO_EINVAL; continue; }
        const int64_t len = s == RO_SUCCESS ? o1 - o0 : 0;
        if (len >= ((int64_t)1 << 32)) { err = RO_EOVERFLOW; continue; }
        // first report of this child, in this wave or any earlier one
        const uint32_t bit = 1u << (c & 31);
        const uint32_t old = atomicOr(&seen[c >> 5], bit);
        if (old & bit) { err = RO_EDUP; continue; }
        Canon e;
        e.src = reinterpret_cast<uint64_t>(data) + (uint64_t)o0;
        e.len = (uint32_t)len;
        e.tag = (kStreamEpoch << 2) | s;
        canon[c] = e;
        if (k < kBig) atomicAdd(&cnt[p], 1);
        else atomicAdd(&big[spread + (st >> kBigShift)], 1);
    }
    if (err) raise_err(ctl, err);
}

// Newly complete parents, compacted in ascending order (one tile = 4096
// parents), and the exclusive scan of their child counts: two look-back
// chains, one over emitted parents and one over their children.
__global__ __launch_bounds__(kBlock) void k_stream_select(
    const int64_t *__restrict__ offsets, int64_t P, const int32_t *__restrict__ cnt,
    const int32_t *__restrict__ big, int64_t nslots, uint8_t *__restrict__ emitted,
    uint32_t *__restrict__ elist, int64_t *__restrict__ evoff, uint32_t *__restrict__ emit_parent,
    int32_t *__restrict__ ecnt, int64_t ecnt_stride, int64_t cap_parents, int64_t *n_emitted, Ctl *ctl,
    uint64_t *desc, uint64_t *desc_kids, int64_t desc_cap, int64_t ntiles)
{
    const uint32_t epoch = scan_epoch(ctl);
    __shared__ int64_t s_wave[kBlock / 64];
    __shared__ uint64_t s_b;
    __shared__ int64_t s_t;
    __shared__ int32_t s_last;
    for (;;) {
        const int64_t t = next_ticket(ctl, &s_t);
        if (t >= ntiles) break;
        const int64_t p0 = t * kTile + (int64_t)threadIdx.x * kItems;
        uint32_t fmask = 0;
        uint32_t kk[kItems];
        int64_t kids = 0;
#pragma unroll
        for (int k = 0; k < kItems; ++k) {
            const int64_t p = p0 + k;
            kk[k] = 0;
            if (p < P && !emitted[p]) {
                const int64_t st = offsets[p];
                const int64_t kp = offsets[p + 1] - st;
                if (reported(cnt, big, nslots, p, st, kp) == kp) {
                    fmask |= 1u << k;
                    kk[k] = (uint32_t)kp;
                    kids += kp;
                }
            }
        }
        int64_t tot, totk;
        const int64_t ex = block_excl_scan(__popc(fmask), s_wave, tot);
        const int64_t exk = block_excl_scan(kids, s_wave, totk);
        const uint64_t pre = tile_prefix(desc, t, epoch, (uint64_t)tot, &s_b, ctl);
        const uint64_t prek = tile_prefix(desc_kids, t, epoch, (uint64_t)totk, &s_b, ctl);
        int64_t e = (int64_t)pre + ex;
        int64_t run = (int64_t)prek + exk;
        bool over = false;
#pragma unroll
        for (int k = 0; k < kItems; ++k) {
            if (!(fmask & (1u << k))) continue;
            const int64_t p = p0 + k;
            if (e < cap_parents) {
                elist[e] = (uint32_t)p;
                evoff[e] = run;
                if (emit_parent) emit_parent[e] = (uint32_t)p;
                ecnt[e] = 0;
                ecnt[ecnt_stride + e] = 0;
                ecnt[2 * ecnt_stride + e] = 0;
                emitted[p] = 1;
            } else {
                if (e == cap_parents) {
                    // the emission stops here: its virtual children end at run
                    evoff[e] = run;
                    ctl->n_virtual = run;
                }
                over = true;
            }
            ++e;
            run += kk[k];
        }
        if (over) raise_err(ctl, RO_ECAP);
        if (t == ntiles - 1 && threadIdx.x == 0) {
            const int64_t E = (int64_t)pre + tot;
            if (n_emitted) *n_emitted = E;
            ctl->n_items = E < cap_parents ? E : cap_parents;
            if (E <= cap_parents) {
                evoff[E] = (int64_t)prek + totk;
                ctl->n_virtual = (int64_t)prek + totk;
            }
        }
    }
    ticket_done(ctl, epoch, desc, desc_cap, &s_last);
}

// vmap[v] = canonical slot of virtual child v: the (v - evoff[e])-th child of
// emitted parent elist[e].  16 consecutive virtual children per thread.
__global__ __launch_bounds__(kBlock) void k_stream_vmap(const int64_t *__restrict__ evoff,
                                                        const uint32_t *__restrict__ elist,
                                                        const int64_t *__restrict__ offsets,
                                                        uint32_t *__restrict__ vmap, Ctl *ctl)
{
    const int64_t E = ctl->n_items;
    const int64_t V = ctl->n_virtual;
    const int64_t nthreads = (V + kItems - 1) / kItems;
    for (int64_t g = (int64_t)blockIdx.x * kBlock + threadIdx.x; g < nthreads;
         g += (int64_t)gridDim.x * kBlock) {
        const int64_t v0 = g * kItems;
        int64_t e = upper_bound_g(evoff, 0, E + 1, v0) - 1;
        int64_t start = evoff[e];
        int64_t base = offsets[elist[e]];
        for (int k = 0; k < kItems; ++k) {
            const int64_t v = v0 + k;
            if (v >= V) break;
            if (v >= evoff[e + 1]) {
                e = advance_parent(evoff, E, e, v);
                start = evoff[e];
                base = offsets[elist[e]];
            }
            vmap[v] = (uint32_t)(base + (v - start));
        }
    }
}

// After the scan: counts and state of every emitted parent, trailing slot
// offsets, capacity check (before the copy).
__global__ void k_stream_emit_check(int64_t *__restrict__ emit_off, const int64_t *__restrict__ evoff,
                                    const int32_t *__restrict__ ecnt, int64_t ecnt_stride,
                                    int32_t *__restrict__ ns, int32_t *__restrict__ nf, int32_t *__restrict__ nk,
                                    uint8_t *__restrict__ pstate, int64_t cap_bytes, int has_data,
                                    int64_t *n_bytes, Ctl *ctl)
{
    const int64_t E = ctl->n_items;
    const int64_t V = ctl->n_virtual;
    const int64_t total = V > 0 ? ctl->total : 0;
    const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (g == 0) {
        emit_off[E] = total;
        if (n_bytes) *n_bytes = total;
        if (has_data && total > cap_bytes) raise_err(ctl, RO_ECAP);
    }
    for (int64_t e = g; e < E; e += (int64_t)gridDim.x * blockDim.x) {
        // emitted parents without children at the very end get the total
        if (evoff[e] >= V) emit_off[e] = total;
        const int32_t a = ecnt[e], f = ecnt[ecnt_stride + e], s = ecnt[2 * ecnt_stride + e];
        if (ns) ns[e] = a;
        if (nf) nf[e] = f;
        if (nk) nk[e] = s;
        if (pstate) pstate[e] = f > 0 ? RO_FAILED : RO_SUCCESS;
    }
}

__global__ void k_stream_finish(Ctl *ctl)
{
    if (threadIdx.x == 0) {
        ctl->n_items = 0;
        ctl->n_virtual = 0;
        ctl->total = 0;
        ctl->n_filled = 0;    // counted by the canonical scan, unused here
    }
}

// Forgets every report and emission: seen bits, counters and emitted flags
// back to zero.  Canonical slots need no clearing, since a slot is read only
// for children of emitted parents, and those were all reported.
__global__ void k_stream_clear(uint32_t *__restrict__ seen, int64_t n_seen, int32_t *__restrict__ cnt,
                               int64_t n_cnt, int32_t *__restrict__ big, int64_t n_big,
                               uint8_t *__restrict__ emitted, int64_t n_emitted)
{
    const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = g; i < n_seen; i += stride) seen[i] = 0;
    for (int64_t i = g; i < n_cnt; i += stride) cnt[i] = 0;
    for (int64_t i = g; i < n_big; i += stride) big[i] = 0;
    for (int64_t i = g; i < n_emitted; i += stride) emitted[i] = 0;
}

hipError_t launch_stream_reset(const Launch &L, StreamState &s)
{
    RO_LAUNCH(L, RO_K_MISC, k_stream_clear, dim3((unsigned)L.num_cus * 4), dim3(256), 0, L.stream, s.seen,
              (s.N + 31) / 32 + 1, s.cnt, s.P + 1, s.big, stream_big_size(s.N), s.emitted, s.P + 1);
    return launch_stream_init(L, s);
}

hipError_t launch_stream_init(const Launch &L, StreamState &s)
{
    RO_LAUNCH(L, RO_K_MISC, k_stream_check, dim3((unsigned)L.num_cus), dim3(256), 0, L.stream, s.offsets, s.P,
              s.N, L.ctl);
    return hipGetLastError();
}

hipError_t launch_stream_report(const Launch &L, StreamState &s, const uint32_t *rp, const uint32_t *ro,
                                const uint8_t *rs, const int64_t *roff, const uint8_t *data, int64_t n)
{
    int64_t grid = (n + kBlock - 1) / kBlock;
    grid = grid < 1 ? 1 : (grid > (int64_t)L.num_cus * 8 ? (int64_t)L.num_cus * 8 : grid);
    RO_LAUNCH(L, RO_K_STREAM_REPORT, k_stream_report, dim3((unsigned)grid), dim3(kBlock), 0, L.stream, rp, ro,
              rs, roff, data, n, s.offsets, s.P, s.N, s.canon, s.seen, s.cnt, s.big, stream_big_slots(s.N),
              L.ctl);
    return hipGetLastError();
}

hipError_t launch_virtual_scan(const Launch &L, const int64_t *voff, const int64_t *E_dev, const uint32_t *vmap,
                               const Canon *canon, int64_t canon_cap, int64_t *emit_off, int32_t *ns,
                               int32_t *nf, int32_t *nk, int64_t *sub_base);
hipError_t launch_virtual_copy(const Launch &L, const int64_t *voff, const int64_t *E_dev, const uint32_t *vmap,
                               const Canon *canon, int64_t canon_cap, const int64_t *sub_base, uint8_t *out);

int64_t stream_desc_tiles(int64_t P, int64_t N)
{
    const int64_t tp = (P + kTile - 1) / kTile + 1, tn = (N + kTile - 1) / kTile + 1;
    return 2 * tp > tn ? 2 * tp : tn;
}

hipError_t launch_stream_emit(const Launch &L, StreamState &s, uint32_t *emit_parent, int64_t *emit_off,
                              uint8_t *emit_data, int64_t cap_parents, int64_t cap_bytes, int32_t *ns,
                              int32_t *nf, int32_t *nk, uint8_t *pstate, int64_t *n_emitted,
                              int64_t *n_bytes)
{
    const int64_t ntiles = s.P > 0 ? (s.P + kTile - 1) / kTile : 1;
    if (2 * ntiles > L.desc_cap) return hipErrorInvalidValue;
    const int64_t grid = ntiles < (int64_t)L.num_cus * 4 ? ntiles : (int64_t)L.num_cus * 4;
    const int64_t es = s.P + 1;
    RO_LAUNCH(L, RO_K_STREAM_SELECT, k_stream_select, dim3((unsigned)grid), dim3(kBlock), 0, L.stream,
              s.offsets, s.P, s.cnt, s.big, stream_big_slots(s.N), s.emitted, s.elist, s.evoff, emit_parent,
              s.ecnt, es, cap_parents, n_emitted, L.ctl, L.desc, L.desc + ntiles, L.desc_cap, ntiles);
    RO_LAUNCH(L, RO_K_STREAM_SELECT, k_stream_vmap, dim3((unsigned)L.num_cus * 8), dim3(kBlock), 0, L.stream,
              s.evoff, s.elist, s.offsets, s.vmap, L.ctl);
    hipError_t e = launch_virtual_scan(L, s.evoff, &L.ctl->n_items, s.vmap, s.canon, s.N, emit_off, s.ecnt,
                                       s.ecnt + es, s.ecnt + 2 * es, s.sub_base);
    if (e != hipSuccess) return e;
    RO_LAUNCH(L, RO_K_STREAM_FINISH, k_stream_emit_check, dim3((unsigned)L.num_cus), dim3(256), 0, L.stream,
              emit_off, s.evoff, s.ecnt, es, ns, nf, nk, pstate, cap_bytes, emit_data != nullptr ? 1 : 0, n_bytes,
              L.ctl);
    if (emit_data != nullptr) {
        e = launch_virtual_copy(L, s.evoff, &L.ctl->n_items, s.vmap, s.canon, s.N, s.sub_base, emit_data);
        if (e != hipSuccess) return e;
    }
    RO_LAUNCH(L, RO_K_STREAM_FINISH, k_stream_finish, dim3(1), dim3(64), 0, L.stream, L.ctl);
    return hipGetLastError();
}

}  // namespace ro
