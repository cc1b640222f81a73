// Streaming completion on gfx950: reports arrive wave by wave; after each
// wave, every parent whose children are now all terminal is emitted once, in
// ascending parent order, with its ordered bytes, counts and state.
//
// RayOrch (arXiv 2609.18703): a parent can finalise and proceed as soon as all
// of its required child results are terminal (Sec. 1; Sec. 4 Reduce rule);
// facts are published once and conflicting repeats are rejected (Sec. 4,
// publication rules).
//
// Per wave:   report  -> canonical slots + seen bits (+ a count for parents
//                        with many children).
// Per emit:   select  -> ascending list of newly complete parents and the
//                        exclusive scan of their child counts (two look-back
//                        chains in one pass over all parents): a "virtual"
//                        expansion whose children are the emitted parents'
//                        children, in order;
//             scan    -> over the virtual children: each one's canonical slot,
//                        output position and source, the emitted slot
//                        offsets and per-state counts;
//             out     -> counts, states, trailing offsets, capacity, and the
//                        emitted bytes from the per-child positions.
#include "ro_copy.h"

namespace ro {

// How many children of a parent have reported, by its size k:
//   k < kMid   the seen bits of its children (at most three words), no counter;
//   k < kBig   one counter, indexed by its first child >> kMidShift;
//   k >= kBig  kSpread counters on separate lines, indexed by its first
//              child >> kBigShift: the reports of a parent with many children
//              would otherwise all add to one address, and atomics on one
//              address serialise.
// A parent of at least 2^s children is the only one whose first child falls
// in its 2^s-child block, so these indices never collide.
constexpr int kMidShift = 6, kBigShift = 10;
constexpr int64_t kMid = (int64_t)1 << kMidShift, kBig = (int64_t)1 << kBigShift;
constexpr int kSpread = 16;

int64_t stream_mid_size(int64_t N) { return (N >> kMidShift) + 1; }
int64_t stream_big_slots(int64_t N) { return (N >> kBigShift) + 1; }
int64_t stream_big_size(int64_t N) { return (int64_t)kSpread * stream_big_slots(N); }

__device__ __forceinline__ int64_t reported(const uint32_t *__restrict__ seen, const int32_t *__restrict__ mid,
                                            const int32_t *__restrict__ big, int64_t nslots, int64_t st,
                                            int64_t k)
{
    if (k <= 0) return 0;
    if (k < kMid) {
        const int64_t c1 = st + k;                  // children [st, c1)
        int64_t n = 0;
        for (int64_t w = st >> 5; w <= (c1 - 1) >> 5; ++w) {
            uint32_t m = seen[w];
            const int64_t b0 = w << 5;
            if (st > b0) m &= 0xffffffffu << (st - b0);
            if (c1 < b0 + 32) m &= 0xffffffffu >> (b0 + 32 - c1);
            n += __popc(m);
        }
        return n;
    }
    if (k < kBig) return mid[st >> kMidShift];
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

// One wave of reports.  Accepted slots are tagged with the run's epoch.
// With a group-failure barrier, reports commit in order after every earlier
// wave: one of a barred parent, or one after its parent's first group
// failure in this wave, is rejected (counted into *n_rejected).
__global__ __launch_bounds__(kBlock) void k_stream_report(
    const uint32_t *__restrict__ rp, const uint32_t *__restrict__ ro_, const uint8_t *__restrict__ rs,
    const int64_t *__restrict__ roff, const uint8_t *data, int64_t n, const int64_t *__restrict__ offsets,
    int64_t P, int64_t N, Canon *__restrict__ canon, uint32_t *__restrict__ seen, int32_t *__restrict__ mid,
    int32_t *__restrict__ big, int64_t nslots, uint32_t run_epoch, const uint8_t *__restrict__ barrier,
    const uint64_t *__restrict__ gkey, uint32_t gf_epoch, int64_t *n_rejected, Ctl *ctl)
{
    __shared__ int64_t s_wave[kBlock / 64];
    const int64_t gtid = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    const int64_t gstride = (int64_t)gridDim.x * kBlock;
    const int64_t spread = (int64_t)(((blockIdx.x << 2) + (threadIdx.x >> 6)) & (kSpread - 1)) * nslots;
    int err = 0;
    int64_t rej = 0;
    if (gtid == 0 && n > 0 && roff[0] < 0) err = RO_EINVAL;
    for (int64_t i = gtid; i < n; i += gstride) {
        uint32_t s = rs[i];
        const int64_t o0 = roff[i], o1 = roff[i + 1];
        if (o1 < o0) { err = RO_EINVAL; continue; }
        if (s > RO_PENDING && !(s == RO_GROUP_FAILED && barrier)) { err = RO_ESTATE; continue; }
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
        if (gf_rejected(barrier, gkey, gf_epoch, p, i)) { ++rej; continue; }
        if (s == RO_GROUP_FAILED) s = RO_FAILED;
        // first report of this child, in this wave or any earlier one
        const uint32_t bit = 1u << (c & 31);
        const uint32_t old = atomicOr(&seen[c >> 5], bit);
        if (old & bit) { err = RO_EDUP; continue; }
        Canon e;
        e.src = reinterpret_cast<uint64_t>(data) + (uint64_t)o0;
        e.len = (uint32_t)len;
        e.tag = (run_epoch << 2) | s;
        canon[c] = e;
        if (k >= kBig) atomicAdd(&big[spread + (st >> kBigShift)], 1);
        else if (k >= kMid) atomicAdd(&mid[st >> kMidShift], 1);
    }
    if (err) raise_err(ctl, err);
    if (barrier) {
        const int64_t r = block_sum(rej, s_wave);
        if (threadIdx.x == 0 && r && n_rejected)
            __hip_atomic_fetch_add(n_rejected, r, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// Newly complete parents, compacted in ascending order (one tile = 2048
// parents, eight per thread), and the exclusive scan of their child counts:
// two look-back chains, one over emitted parents and one over their children.
constexpr int kSTile = 2048;
constexpr int kSItems = kSTile / kBlock;

__global__ __launch_bounds__(kBlock) void k_stream_select(
    const int64_t *__restrict__ offsets, int64_t P, const uint32_t *__restrict__ seen,
    const int32_t *__restrict__ mid, const int32_t *__restrict__ big, int64_t nslots,
    const uint8_t *__restrict__ barrier, uint8_t *__restrict__ ebar, uint8_t *__restrict__ emitted,
    int64_t *__restrict__ ebase, int64_t *__restrict__ evoff, uint32_t *__restrict__ emit_parent,
    int32_t *__restrict__ ecnt, int64_t ecnt_stride, int64_t cap_parents, int64_t *n_emitted, Ctl *ctl,
    uint64_t *desc, uint64_t *desc_kids, int64_t desc_cap, int64_t ntiles)
{
    const uint32_t epoch = scan_epoch(ctl);
    __shared__ int64_t s_wave[kBlock / 64];
    __shared__ uint64_t s_b2[2];
    __shared__ int64_t s_t;
    __shared__ int32_t s_last;
    for (;;) {
        const int64_t t = next_ticket(ctl, &s_t);
        if (t >= ntiles) break;
        const int64_t p0 = t * kSTile + (int64_t)threadIdx.x * kSItems;
        uint32_t fmask = 0;
        uint32_t kk[kSItems];
        int64_t kids = 0;
#pragma unroll
        for (int k = 0; k < kSItems; ++k) {
            const int64_t p = p0 + k;
            kk[k] = 0;
            if (p < P && !emitted[p]) {
                const int64_t st = offsets[p];
                const int64_t kp = offsets[p + 1] - st;
                // a barred parent is complete: its uncommitted children are suppressed
                if ((barrier && barrier[p]) || reported(seen, mid, big, nslots, st, kp) == kp) {
                    fmask |= 1u << k;
                    kk[k] = (uint32_t)kp;
                    kids += kp;
                }
            }
        }
        int64_t tot, totk;
        const int64_t ex = block_excl_scan(__popc(fmask), s_wave, tot);
        const int64_t exk = block_excl_scan(kids, s_wave, totk);
        uint64_t pre, prek;
        tile_prefix2(desc, (uint64_t)tot, desc_kids, (uint64_t)totk, t, epoch, s_b2, pre, prek, ctl);
        int64_t e = (int64_t)pre + ex;
        int64_t run = (int64_t)prek + exk;
        bool over = false;
#pragma unroll
        for (int k = 0; k < kSItems; ++k) {
            if (!(fmask & (1u << k))) continue;
            const int64_t p = p0 + k;
            if (e < cap_parents) {
                ebase[e] = offsets[p] - run;      // canonical slot of virtual child v: ebase[e] + v
                evoff[e] = run;
                ebar[e] = (barrier && barrier[p]) ? 1 : 0;
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

// Byte scan over the virtual children of this emission, 1024 per tile (four
// consecutive per thread; small tiles spread the random slot reads over many
// compute units).  Virtual child v of emitted parent e lives in canonical
// slot ebase[e] + v.  Writes each child's output position edst[v] and source
// address esrc[v] for the copy, the emitted slot offsets, and per-state
// counts (run lengths, aggregated in LDS).  Only the first min(grid, tiles)
// workgroups take part.
constexpr int kETile = 1024;
constexpr int kEItems = kETile / kBlock;
constexpr int kECntLds = 256;

__global__ __launch_bounds__(kBlock) void k_emit_scan(
    const int64_t *__restrict__ evoff, const int64_t *__restrict__ ebase, const Canon *__restrict__ canon,
    int64_t *__restrict__ edst, uint64_t *__restrict__ esrc, int64_t *__restrict__ emit_off,
    int32_t *__restrict__ ecnt, int64_t ecnt_stride, uint32_t run_epoch, Ctl *ctl, uint64_t *desc,
    int64_t desc_cap)
{
    const int64_t E = ctl->n_items;
    const int64_t V = ctl->n_virtual;
    const int64_t ntiles = (V + kETile - 1) / kETile;
    if ((int64_t)blockIdx.x >= ntiles) return;
    const uint32_t parts = (uint32_t)min64((int64_t)gridDim.x, ntiles);
    const uint32_t sepoch = scan_epoch(ctl);
    __shared__ int64_t s_wave[kBlock / 64];
    __shared__ uint64_t s_b;
    __shared__ int64_t s_t;
    __shared__ int32_t s_last;
    __shared__ int64_t s_p[3];
    __shared__ int16_t s_off[kETile + 2];         // evoff[pf..pl+1] - vt0, clamped to [-1, kETile + 1]
    __shared__ int64_t s_base[kETile + 1];        // ebase[pf..pl]
    __shared__ int32_t s_cnt[3][kECntLds];
    for (;;) {
        const int64_t t = next_ticket(ctl, &s_t);
        if (t >= ntiles) break;
        const int64_t vt0 = t * kETile;
        const int64_t vt1 = min64(vt0 + kETile, V);
        // emitted parents of the tile: pf holds child vt0, pl holds vt1 - 1,
        // q0 is the first one starting at or after vt0
        if (threadIdx.x < 3 * 64) {
            const int w = (int)(threadIdx.x >> 6);
            int64_t r;
            if (w == 0) r = wave_last_le(evoff, 0, E + 1, vt0);
            else if (w == 1) r = wave_last_le(evoff, 0, E + 1, vt1 - 1);
            else r = vt0 == 0 ? 0 : wave_last_le(evoff, 0, E + 1, vt0 - 1) + 1;
            if (lane_id() == 0) s_p[w] = r;
        }
        __syncthreads();
        const int64_t pf = s_p[0], pl = s_p[1], q0t = s_p[2];
        const int64_t Rp = pl - pf + 1;
        const int64_t R = min64(Rp, kECntLds);
        const bool lds_ok = Rp <= kETile;
        if (lds_ok) {
            for (int64_t j = threadIdx.x; j <= Rp; j += kBlock) {
                const int64_t x = evoff[pf + j] - vt0;
                s_off[j] = (int16_t)(x < -1 ? -1 : (x > kETile + 1 ? kETile + 1 : x));
                if (j < Rp) s_base[j] = ebase[pf + j];
            }
        }
        for (int j = threadIdx.x; j < 3 * kECntLds; j += kBlock) (&s_cnt[0][0])[j] = 0;
        __syncthreads();
        // this thread's four virtual children: slot, length, state, source
        const int64_t v0 = vt0 + (int64_t)threadIdx.x * kEItems;
        int64_t e0 = 0;
        uint32_t len[kEItems], stv[kEItems];
        uint64_t src[kEItems];
        int64_t sum = 0;
#pragma unroll
        for (int k = 0; k < kEItems; ++k) {
            len[k] = 0;
            stv[k] = 4;
            src[k] = 0;
        }
        if (v0 < vt1) {
            int64_t e = lds_ok ? pf + lds_last_le(s_off, 0, (int)Rp, (int)(v0 - vt0))
                               : upper_bound_g(evoff, pf, pl + 1, v0) - 1;
            e0 = e;
#pragma unroll
            for (int k = 0; k < kEItems; ++k) {
                const int64_t v = v0 + k;
                if (v >= vt1) break;
                if (lds_ok) {
                    const int rv = (int)(v - vt0);
                    if (rv >= s_off[e - pf + 1]) e = pf + lds_last_le(s_off, (int)(e - pf) + 1, (int)Rp, rv);
                } else if (v >= evoff[e + 1]) {
                    e = advance_parent(evoff, E, e, v);
                }
                const int64_t c = (lds_ok ? s_base[e - pf] : ebase[e]) + v;
                const Canon x = canon[c];
                if ((x.tag >> 2) == run_epoch) {
                    stv[k] = x.tag & 3u;
                    len[k] = stv[k] == RO_SUCCESS ? x.len : 0;
                    src[k] = x.src;
                }
                sum += len[k];
            }
        }
        int64_t tot;
        const int64_t ex = block_excl_scan(sum, s_wave, tot);
        const uint64_t pre = tile_prefix(desc, t, sepoch, (uint64_t)tot, &s_b, ctl);
        if (v0 < vt1) {
            int64_t pos = (int64_t)pre + ex;
            int64_t e = e0;
            int32_t run[3] = {0, 0, 0};
            auto flush = [&](int64_t q) {
#pragma unroll
                for (int s = 0; s < 3; ++s) {
                    if (run[s]) {
                        if (q - pf < R) atomicAdd(&s_cnt[s][q - pf], run[s]);
                        else atomicAdd(&ecnt[s * ecnt_stride + q], run[s]);
                        run[s] = 0;
                    }
                }
            };
            // emitted parents whose first child is v0 (empty ones included)
            if (evoff[e] == v0) {
                const int64_t qa = v0 == vt0 ? q0t : lower_bound_g(evoff, pf, e + 1, v0);
                for (int64_t q = qa; q <= e; ++q) emit_off[q] = pos;
            }
#pragma unroll
            for (int k = 0; k < kEItems; ++k) {
                const int64_t v = v0 + k;
                if (v >= vt1) break;
                if (v >= evoff[e + 1]) {
                    flush(e);
                    const int64_t en = advance_parent(evoff, E, e, v);
                    for (int64_t q = e + 1; q <= en; ++q) emit_off[q] = pos;
                    e = en;
                }
                if (stv[k] < 3) run[stv[k]] += 1;
                edst[v] = pos;
                esrc[v] = src[k];
                pos += len[k];
            }
            flush(e);
        }
        __syncthreads();
        for (int64_t j = threadIdx.x; j < R; j += kBlock) {
#pragma unroll
            for (int s = 0; s < 3; ++s) {
                const int32_t x = s_cnt[s][j];
                if (x) atomicAdd(&ecnt[s * ecnt_stride + pf + j], x);
            }
        }
        if (t == ntiles - 1 && threadIdx.x == 0) {
            const int64_t total = (int64_t)pre + tot;
            ctl->total = total;
            edst[V] = total;
            if (pre >= kSat) raise_err(ctl, RO_EOVERFLOW);
        }
        __syncthreads();
    }
    ticket_done_n(ctl, sepoch, desc, desc_cap, &s_last, parts);
}

// Outputs of the emission once its scan is done: per emitted parent its
// counts, state and (for parents without children at the very end) slot
// offset; then the bytes.  The output is cut into byte units as in the
// gather's copy, kEmitMinUnit bytes or more (a unit costs a search over the
// positions, not a re-read of slot records, so small units pay here); a unit
// finds its first child by a wave search over the output positions and takes
// the children it covers 256 at a time, each clipped to the unit.
#ifndef RO_EMIT_MIN_UNIT
#define RO_EMIT_MIN_UNIT 1024
#endif
constexpr int64_t kEmitMinUnit = RO_EMIT_MIN_UNIT;
#ifndef RO_EMIT_GRID
#define RO_EMIT_GRID 4                      // emission copy workgroups per CU
#endif
#ifndef RO_EMIT_UNITS
#define RO_EMIT_UNITS 1                     // byte units per wave of the grid
#endif
constexpr int64_t kEmitUnits = RO_EMIT_UNITS;
#ifndef RO_EMIT_STEPS
#define RO_EMIT_STEPS 4
#endif

__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(4))) void k_emit_out(
    int64_t *__restrict__ emit_off, const int64_t *__restrict__ evoff, const int32_t *__restrict__ ecnt,
    int64_t ecnt_stride, const uint8_t *__restrict__ ebar, int32_t *__restrict__ ns, int32_t *__restrict__ nf,
    int32_t *__restrict__ nk, uint8_t *__restrict__ pstate, int64_t *n_bytes, const int64_t *__restrict__ edst,
    const uint64_t *__restrict__ esrc, uint8_t *__restrict__ out, int64_t cap_bytes, Ctl *ctl)
{
    constexpr int kWaves = kBlock / 64;
    __shared__ int32_t s_dst_all[kWaves][kSub + 1];
    __shared__ uint64_t s_src_all[kWaves][kSub];
    __shared__ int32_t s_edge_all[kWaves][kEdgeCap];
    __shared__ int16_t s_edger_all[kWaves][kEdgeCap];
    const int64_t E = ctl->n_items;
    const int64_t V = ctl->n_virtual;
    const int64_t T = V > 0 ? ctl->total : 0;
    const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (g == 0) {
        emit_off[E] = T;
        if (n_bytes) *n_bytes = T;
        if (out && T > cap_bytes) raise_err(ctl, RO_ECAP);
    }
    for (int64_t e = g; e < E; e += (int64_t)gridDim.x * blockDim.x) {
        if (evoff[e] >= V) emit_off[e] = T;
        const int32_t a = ecnt[e], f = ecnt[ecnt_stride + e], k = ecnt[2 * ecnt_stride + e];
        if (ns) ns[e] = a;
        if (nf) nf[e] = f;
        if (nk) nk[e] = k;
        if (pstate) pstate[e] = (f > 0 || ebar[e]) ? RO_FAILED : RO_SUCCESS;
    }
    if (out == nullptr || T <= 0 || T > cap_bytes || read_err(ctl) != 0) return;
    const uint64_t outa = reinterpret_cast<uint64_t>(out);
    const int64_t mis = (int64_t)(outa & 15);
    const int64_t nwaves = (int64_t)gridDim.x * kWaves;
    int64_t G = (T + nwaves * kEmitUnits - 1) / (nwaves * kEmitUnits);
    G = (G + 15) & ~(int64_t)15;
    G = G < kEmitMinUnit ? kEmitMinUnit : (G > ((int64_t)1 << 30) ? ((int64_t)1 << 30) : G);
    const int64_t nunits = (T + mis + G - 1) / G;
    const int wave = uni32((int)(threadIdx.x >> 6)), lane = lane_id();
    int32_t *s_dst = s_dst_all[wave];
    uint64_t *s_src = s_src_all[wave];
    int32_t *s_edge = s_edge_all[wave];
    int16_t *s_edger = s_edger_all[wave];
    for (int64_t u = (int64_t)blockIdx.x * kWaves + wave; u < nunits; u += nwaves) {
        const int64_t lo = max64(u * G - mis, 0);
        const int64_t hi = min64((u + 1) * G - mis, T);
        for (int64_t r0 = uni64(wave_last_le(edst, 0, V, lo)); r0 < V; r0 += kSub) {
            // children r0 .. r0 + kSub - 1, their starts clipped to [ws, we)
            const int64_t dend = edst[min64(r0 + kSub, V)];
            const int64_t ws = max64(lo, edst[r0]);
            const int64_t we = min64(hi, dend);
            if (we <= ws) {
                if (dend >= hi) break;
                continue;                          // only empty children here
            }
            // positions 64 at a time, stopping after the group that reaches
            // the window's end: a small unit covers a few children, and the
            // rest of the 256 are set empty without being read
            bool past = false;
#pragma unroll
            for (int k = 0; k < kSub / 64; ++k) {
                const int i = k * 64 + lane;
                const int64_t v = r0 + i;
                if (past) {
                    s_dst[i] = (int32_t)(we - ws);
                    s_src[i] = 0;
                    continue;
                }
                const int64_t d = v < V ? edst[v] : T;
                const int64_t cs = min64(max64(d, ws), we);
                s_dst[i] = (int32_t)(cs - ws);
                s_src[i] = (v < V ? esrc[v] : 0) + (uint64_t)(cs - d);
                past = __shfl(d, 63, 64) >= we;
            }
            if (lane == 0) s_dst[kSub] = (int32_t)(we - ws);
            __builtin_amdgcn_wave_barrier();
            copy_window_nb<RO_EMIT_STEPS>(s_dst, s_src, s_edge, s_edger, (int)(we - ws), outa, ws, lane);
            __builtin_amdgcn_wave_barrier();
            if (dend >= hi) break;
        }
    }
}

// Forgets every report and emission: seen bits, counters and emitted flags
// back to zero.  Canonical slots need no clearing, since a slot is read only
// for children of emitted parents, and those were all reported.
__global__ void k_stream_clear(uint32_t *__restrict__ seen, int64_t n_seen, int32_t *__restrict__ mid,
                               int64_t n_mid, int32_t *__restrict__ big, int64_t n_big,
                               uint8_t *__restrict__ emitted, uint8_t *__restrict__ barrier, int64_t n_emitted)
{
    const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = g; i < n_seen; i += stride) seen[i] = 0;
    for (int64_t i = g; i < n_mid; i += stride) mid[i] = 0;
    for (int64_t i = g; i < n_big; i += stride) big[i] = 0;
    for (int64_t i = g; i < n_emitted; i += stride) {
        emitted[i] = 0;
        if (barrier) barrier[i] = 0;
    }
}

hipError_t launch_stream_reset(const Launch &L, StreamState &s)
{
    RO_LAUNCH(L, RO_K_MISC, k_stream_clear, dim3((unsigned)L.num_cus * 4), dim3(256), 0, L.stream, s.seen,
              (s.N + 31) / 32 + 1, s.mid, stream_mid_size(s.N), s.big, stream_big_size(s.N), s.emitted,
              s.barrier, s.P);
    return launch_stream_init(L, s);
}

hipError_t launch_stream_init(const Launch &L, StreamState &s)
{
    RO_LAUNCH(L, RO_K_MISC, k_stream_check, dim3((unsigned)L.num_cus), dim3(256), 0, L.stream, s.offsets, s.P,
              s.N, L.ctl);
    return hipGetLastError();
}

hipError_t launch_stream_report(const Launch &L, StreamState &s, const uint32_t *rp, const uint32_t *ro,
                                const uint8_t *rs, const int64_t *roff, const uint8_t *data, int64_t n,
                                int64_t *n_rejected)
{
    if (s.barrier) {
        const hipError_t e = launch_first_gf(L, rs, rp, n, s.P, s.barrier, s.gkey, s.gf_epoch);
        if (e != hipSuccess) return e;
    }
    int64_t grid = (n + kBlock - 1) / kBlock;
    grid = grid < 1 ? 1 : (grid > (int64_t)L.num_cus * 8 ? (int64_t)L.num_cus * 8 : grid);
    RO_LAUNCH(L, RO_K_STREAM_REPORT, k_stream_report, dim3((unsigned)grid), dim3(kBlock), 0, L.stream, rp, ro,
              rs, roff, data, n, s.offsets, s.P, s.N, s.canon, s.seen, s.mid, s.big, stream_big_slots(s.N),
              s.run_epoch, s.barrier, s.gkey, s.gf_epoch, n_rejected, L.ctl);
    if (s.barrier) return launch_gf_fold(L, rs, rp, n, s.P, s.barrier, s.gkey, s.gf_epoch);
    return hipGetLastError();
}

int64_t stream_desc_tiles(int64_t P, int64_t N)
{
    const int64_t tp = (P + kSTile - 1) / kSTile + 1, tn = (N + kETile - 1) / kETile + 1;
    return 2 * tp > tn ? 2 * tp : tn;
}

hipError_t launch_stream_emit(const Launch &L, StreamState &s, uint32_t *emit_parent, int64_t *emit_off,
                              uint8_t *emit_data, int64_t cap_parents, int64_t cap_bytes, int32_t *ns,
                              int32_t *nf, int32_t *nk, uint8_t *pstate, int64_t *n_emitted,
                              int64_t *n_bytes)
{
    const int64_t ntiles = s.P > 0 ? (s.P + kSTile - 1) / kSTile : 1;
    if (2 * ntiles > L.desc_cap || (s.N + kETile - 1) / kETile > L.desc_cap) return hipErrorInvalidValue;
    const int64_t grid = ntiles < (int64_t)L.num_cus * 4 ? ntiles : (int64_t)L.num_cus * 4;
    const int64_t es = s.P + 1;
    RO_LAUNCH(L, RO_K_STREAM_SELECT, k_stream_select, dim3((unsigned)grid), dim3(kBlock), 0, L.stream,
              s.offsets, s.P, s.seen, s.mid, s.big, stream_big_slots(s.N), s.barrier, s.ebar, s.emitted, s.ebase,
              s.evoff, emit_parent,
              s.ecnt, es, cap_parents, n_emitted, L.ctl, L.desc, L.desc + ntiles, L.desc_cap, ntiles);
    const int64_t grid_s = (int64_t)L.num_cus * 2;
    RO_LAUNCH(L, RO_K_STREAM_SCAN, k_emit_scan, dim3((unsigned)grid_s), dim3(kBlock), 0, L.stream, s.evoff,
              s.ebase, s.canon, s.edst, s.esrc, emit_off, s.ecnt, es, s.run_epoch, L.ctl, L.desc, L.desc_cap);
    const int64_t grid_c = (int64_t)L.num_cus * RO_EMIT_GRID;
    RO_LAUNCH(L, RO_K_STREAM_COPY, k_emit_out, dim3((unsigned)grid_c), dim3(kBlock), 0, L.stream, emit_off,
              s.evoff, s.ecnt, es, s.ebar, ns, nf, nk, pstate, n_bytes, s.edst, s.esrc, emit_data, cap_bytes, L.ctl);
    return hipGetLastError();
}

}  // namespace ro
