// Per-Call FIFO Ready Queue with elastic reservation on gfx950.
//
// RayOrch (arXiv 2609.18703), Sec. 4 "Scheduling Ready Grains": ready Grains
// sit in one FIFO queue in enqueue order; each elastic reservation removes at
// most B entries from the head and may mix parents.  Taking the reservations
// one after another until the queue is empty is a stable compaction of the
// ready entries cut into consecutive chunks of B, which is what this kernel
// computes in one pass: a workgroup scan of the ready flags and a decoupled
// look-back across tiles give every ready entry its FIFO slot.  A barred
// parent's entries (Sec. 4 "Commit, Failure, and Recovery": queued siblings
// of a group failure are suppressed before dispatch) are simply not ready.
#include "ro_device.h"

namespace ro {

// Coarse child -> parent map, one 8-byte entry per block of 2^s children:
// for block j, x = the parent p0 of child j 2^s, with bit 31 set when the
// whole block lies in p0, and y = the ordinal of child j 2^s in p0.  A child
// of a one-parent block has its tags from its entry alone; any other child's
// parent lies between p0 and the next entry's parent, and the search for it
// starts from offsets[p0] = j 2^s - y without reading it.  Built for fewer
// than 2^31 parents (the flag bit); otherwise the offsets are searched whole.
// The block size follows the mean fan-out N / P (map_shift): blocks of 16
// children for small parents keep the searches short, blocks of 128 for
// large ones keep the map small enough to stay in cache (workload 2, mean
// 411: 128; the documents' levels, means 9 and 15: 16).
constexpr uint32_t kMapOne = 0x80000000u;

// Tag outputs of a queue too long for the caches are written with
// non-temporal stores: they are read once, by a later call, and kept out of
// L2 they leave the coarse map and offsets there for this kernel's lookups
// (workload 2's 41M-entry ready-queue batch 0.46 -> 0.42 ms, and the gather's
// report scatter that reads them 1.55 -> 1.53 ms).  A shorter queue's tags
// are stored normally: they then still sit in cache when the gather reads
// them (the documents' 2.7M-entry batch).
constexpr int64_t kTagNtEntries = (int64_t)8 << 20;   // 32 MB per tag array, the size of all L2s
__device__ __forceinline__ void st_tag_nt(uint32_t *p, uint32_t v) { __builtin_nontemporal_store(v, p); }

// The tile's staged outputs s_out[0, lim) to dst[base, base + lim): two
// loops, since one store with a chosen hint is folded into a plain store.
__device__ __forceinline__ void write_tags(uint32_t *__restrict__ dst, int64_t base, const uint32_t *s_out,
                                           int64_t lim, bool nt)
{
    if (nt) {
        for (int64_t j = threadIdx.x; j < lim; j += kBlock) st_tag_nt(dst + base + j, s_out[j]);
    } else {
        for (int64_t j = threadIdx.x; j < lim; j += kBlock) dst[base + j] = s_out[j];
    }
}

// log2 of the children per map block: the smallest power of two from 16 to
// 128 that is at least the mean number of children per parent.
__device__ __forceinline__ int map_shift(int64_t N, int64_t P)
{
    int s = 4;
    while (s < 7 && ((int64_t)1 << s) * P < N) ++s;
    return s;
}

// entries of a thread whose lookups are in flight together
#ifndef RO_BATCH_LOOKUPS
#define RO_BATCH_LOOKUPS 4
#endif

__global__ void k_batch_cmap(const int64_t *__restrict__ offsets, int64_t P, uint2 *__restrict__ map,
                             int64_t map_cap)
{
    const int64_t N = offsets[P];
    const int sh = map_shift(N, P);
    int64_t nmap = (N + (1 << sh) - 1) >> sh;
    nmap = nmap < map_cap ? nmap : map_cap;
    for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < nmap;
         j += (int64_t)gridDim.x * blockDim.x) {
        const int64_t c0 = j << sh;
        const int64_t p0 = upper_bound_g(offsets, 0, P + 1, c0) - 1;
        const int64_t last = c0 + (1 << sh) - 1 < N ? c0 + (1 << sh) - 1 : N - 1;
        const bool one = offsets[p0 + 1] > last;
        map[j] = make_uint2((uint32_t)p0 | (one ? kMapOne : 0u), (uint32_t)(c0 - offsets[p0]));
    }
}

// Parent and ordinal of K children at once (bit k of `live`: entry k is a
// child id below N; the others are left alone).  Every step's loads are in
// flight together: the map entries of all K, then the rounds of a lockstep
// binary search for the children of blocks that hold several parents (or
// that lie past the map).  Needs P < 2^31 when nmap > 0.
template <int K>
__device__ __forceinline__ void tags_of(const uint2 *__restrict__ map, int64_t nmap, int sh,
                                        const int64_t *__restrict__ offsets, int64_t P, const uint32_t (&c)[K],
                                        uint32_t live, uint32_t (&par)[K], uint32_t (&ord)[K])
{
    if (nmap == 0) {
#pragma unroll
        for (int k = 0; k < K; ++k) {
            if (!((live >> k) & 1u)) continue;
            const int64_t p = upper_bound_g(offsets, 0, P + 1, (int64_t)c[k]) - 1;
            par[k] = (uint32_t)p;
            ord[k] = (uint32_t)((int64_t)c[k] - offsets[p]);
        }
        return;
    }
    uint32_t l[K], h[K];
    int64_t vl[K];
    {
        // a child past the map (the map is sized by the workspace, the
        // expansion may be larger) searches all parents, from offsets[0]
        const int64_t off0 = offsets[0];
        uint2 e[K];
        uint32_t hx[K];
#pragma unroll
        for (int k = 0; k < K; ++k) {
            const int64_t j = (int64_t)(c[k] >> sh);
            const int64_t jj = (((live >> k) & 1u) && j < nmap) ? j : 0;
            e[k] = map[jj];
            hx[k] = map[jj + 1 < nmap ? jj + 1 : jj].x;
        }
#pragma unroll
        for (int k = 0; k < K; ++k) {
            const int64_t j = (int64_t)(c[k] >> sh);
            const uint32_t p0 = e[k].x & ~kMapOne;
            const uint32_t hi = j + 1 < nmap ? (hx[k] & ~kMapOne) : (uint32_t)(P - 1);
            if (((live >> k) & 1u) == 0) {
                l[k] = 0;
                h[k] = 1;
                vl[k] = 0;
            } else if (j >= nmap) {
                l[k] = 0;
                h[k] = (uint32_t)P;
                vl[k] = off0;
            } else {
                l[k] = p0;
                vl[k] = (j << sh) - (int64_t)e[k].y;
                h[k] = (e[k].x & kMapOne) ? p0 + 1 : hi + 1;
            }
        }
    }
    // the parent is the largest p in [l, h) with offsets[p] <= c
    for (;;) {
        bool any = false;
#pragma unroll
        for (int k = 0; k < K; ++k) any |= h[k] - l[k] > 1;
        if (!any) break;
        uint32_t mid[K];
        int64_t v[K];
#pragma unroll
        for (int k = 0; k < K; ++k) {
            mid[k] = h[k] - l[k] > 1 ? (l[k] + h[k]) >> 1 : l[k];
            v[k] = offsets[mid[k]];
        }
#pragma unroll
        for (int k = 0; k < K; ++k) {
            if (h[k] - l[k] > 1) {
                if (v[k] <= (int64_t)c[k]) {
                    l[k] = mid[k];
                    vl[k] = v[k];
                } else {
                    h[k] = mid[k];
                }
            }
        }
    }
#pragma unroll
    for (int k = 0; k < K; ++k) {
        if (!((live >> k) & 1u)) continue;
        par[k] = l[k];
        ord[k] = (uint32_t)((int64_t)c[k] - vl[k]);
    }
}

template <bool kByMap>
__global__ __launch_bounds__(kBlock) void k_batch(
    const uint32_t *__restrict__ queue, const uint8_t *__restrict__ keep, int64_t Q,
    const int64_t *__restrict__ offsets, int64_t P, const uint2 *__restrict__ cmap, int64_t cmap_cap,
    int32_t B, uint32_t *__restrict__ out_child, uint32_t *__restrict__ out_parent,
    uint32_t *__restrict__ out_ordinal, int64_t out_cap, int64_t *n_out, int64_t *n_batches,
    const uint8_t *__restrict__ barrier, const uint32_t *__restrict__ cpar, int64_t cpar_n, Ctl *ctl,
    uint64_t *desc, int64_t desc_cap, int64_t ntiles, int vec_ok)
{
    const uint32_t epoch = scan_epoch(ctl);
    __shared__ uint32_t s_out[kTile];          // one output array of a tile, in slot order
    __shared__ int64_t s_wave[kBlock / 64];
    __shared__ uint64_t s_b;
    __shared__ int64_t s_t;
    __shared__ int32_t s_last;
    const int64_t N = cpar ? min64(offsets[P], cpar_n) : offsets[P];   // ids past the map are out of range
    const int sh = map_shift(offsets[P], P);     // the map's block size, as k_batch_cmap built it
    int64_t nmap = (N + (1 << sh) - 1) >> sh;
    nmap = nmap < cmap_cap ? nmap : cmap_cap;
    const bool want_tags = out_parent != nullptr || out_ordinal != nullptr;
    const bool nt = Q > kTagNtEntries;
    for (;;) {
        const int64_t t = next_ticket(ctl, &s_t);
        if (t >= ntiles) break;
        const int64_t i0 = t * kTile + (int64_t)threadIdx.x * kItems;
        uint32_t q[kItems];
        uint32_t kmask = 0;
        if (vec_ok && i0 + kItems <= Q) {
            const uint4 *qp = reinterpret_cast<const uint4 *>(queue + i0);
#pragma unroll
            for (int k = 0; k < kItems / 4; ++k) {
                const uint4 x = qp[k];
                q[4 * k] = x.x; q[4 * k + 1] = x.y; q[4 * k + 2] = x.z; q[4 * k + 3] = x.w;
            }
            if (keep) {
                const uint4 kv = *reinterpret_cast<const uint4 *>(keep + i0);
                const uint32_t w[4] = {kv.x, kv.y, kv.z, kv.w};
#pragma unroll
                for (int k = 0; k < kItems; ++k)
                    kmask |= (((w[k >> 2] >> (8 * (k & 3))) & 0xffu) != 0 ? 1u : 0u) << k;
            } else {
                kmask = 0xffffu;
            }
        } else {
#pragma unroll
            for (int k = 0; k < kItems; ++k) {
                const int64_t i = i0 + k;
                q[k] = 0;
                if (i < Q) {
                    q[k] = queue[i];
                    if (keep == nullptr || keep[i] != 0) kmask |= 1u << k;
                }
            }
        }
        // lineage tags of the ready entries, RO_BATCH_LOOKUPS of a thread's
        // entries at a time with all their lookups in flight; an entry of a
        // barred parent is not ready
        uint32_t par[kItems], ord[kItems];
        bool bad_range = false;
        uint32_t live = 0;
#pragma unroll
        for (int k = 0; k < kItems; ++k) {
            par[k] = 0xffffffffu;
            ord[k] = 0xffffffffu;
            if (kmask & (1u << k)) {
                if ((int64_t)q[k] >= N) bad_range = true;
                else live |= 1u << k;
            }
        }
        if (want_tags || barrier) {
            if constexpr (kByMap) {
#pragma unroll
                for (int k = 0; k < kItems; ++k) {
                    if (!((live >> k) & 1u)) continue;
                    const int64_t p = (int64_t)cpar[q[k]];
                    par[k] = (uint32_t)p;
                    ord[k] = (uint32_t)((int64_t)q[k] - offsets[p]);
                }
            } else {
                constexpr int H = RO_BATCH_LOOKUPS;
#pragma unroll
                for (int hf = 0; hf < kItems / H; ++hf) {
                    uint32_t cc[H], pp[H], oo[H];
#pragma unroll
                    for (int k = 0; k < H; ++k) cc[k] = q[hf * H + k];
                    tags_of<H>(cmap, nmap, sh, offsets, P, cc, (live >> (hf * H)) & ((1u << H) - 1u), pp, oo);
#pragma unroll
                    for (int k = 0; k < H; ++k) {
                        if ((live >> (hf * H + k)) & 1u) {
                            par[hf * H + k] = pp[k];
                            ord[hf * H + k] = oo[k];
                        }
                    }
                }
            }
            if (barrier) {
#pragma unroll
                for (int k = 0; k < kItems; ++k) {
                    if (((live >> k) & 1u) && barrier[par[k]]) {
                        kmask &= ~(1u << k);                             // suppressed: takes no slot
                        par[k] = 0xffffffffu;
                        ord[k] = 0xffffffffu;
                    }
                }
            }
        }
        if (bad_range) raise_err(ctl, RO_ERANGE);
        const int cnt = __popc(kmask);
        int64_t tot;
        const int64_t ex = block_excl_scan(cnt, s_wave, tot);
        const uint64_t pre = tile_prefix(desc, t, epoch, (uint64_t)tot, &s_b, ctl);
        const int64_t base = (int64_t)pre;
        if (base + tot > out_cap && threadIdx.x == 0) raise_err(ctl, RO_ECAP);
        const int64_t lim = out_cap - base < tot ? (out_cap - base > 0 ? out_cap - base : 0) : tot;
        // stage each requested output array in LDS in slot order, then write
        // the tile's contiguous slot range with coalesced stores
#pragma unroll 1
        for (int which = 0; which < 3; ++which) {
            uint32_t *dst = which == 0 ? out_child : (which == 1 ? out_parent : out_ordinal);
            if (dst == nullptr) continue;
            int slot = (int)ex;
#pragma unroll
            for (int k = 0; k < kItems; ++k) {
                if (kmask & (1u << k)) {
                    s_out[slot] = which == 0 ? q[k] : (which == 1 ? par[k] : ord[k]);
                    ++slot;
                }
            }
            __syncthreads();
            write_tags(dst, base, s_out, lim, nt);
            __syncthreads();
        }
        if (t == ntiles - 1 && threadIdx.x == 0) {
            const int64_t m = (int64_t)pre + tot;
            if (n_out) *n_out = m;
            if (n_batches) *n_batches = (m + B - 1) / B;
        }
    }
    ticket_done(ctl, epoch, desc, desc_cap, &s_last);
}

// The ready queue with a dispatch mask and no barrier: an entry is ready iff
// its mask byte is set, so a tile's count of ready entries is known from the
// mask alone, before any lineage lookup.  A workgroup takes kBatchSuper
// consecutive tiles per ticket (four times fewer tickets and look-back
// steps), counts them, publishes their aggregate and finishes the look-back
// first; only then does it look up the tags of each tile's ready entries and
// write them, staged in LDS, to the tile's contiguous slot range.
constexpr int kBatchSuper = 4;

__global__ __launch_bounds__(kBlock) void k_batch_keep(
    const uint32_t *__restrict__ queue, const uint8_t *__restrict__ keep, int64_t Q,
    const int64_t *__restrict__ offsets, int64_t P, const uint2 *__restrict__ cmap, int64_t cmap_cap, int32_t B,
    uint32_t *__restrict__ out_child, uint32_t *__restrict__ out_parent, uint32_t *__restrict__ out_ordinal,
    int64_t out_cap, int64_t *n_out, int64_t *n_batches, Ctl *ctl, uint64_t *desc, int64_t desc_cap,
    int64_t nsuper, int vec_ok)
{
    const uint32_t epoch = scan_epoch(ctl);
    __shared__ uint32_t s_out[kTile];
    __shared__ int64_t s_wave[kBlock / 64];
    __shared__ int64_t s_sub[kBatchSuper];
    __shared__ uint64_t s_b;
    __shared__ int64_t s_t;
    __shared__ int32_t s_last;
    const int64_t N = offsets[P];
    const int sh = map_shift(offsets[P], P);     // the map's block size, as k_batch_cmap built it
    int64_t nmap = (N + (1 << sh) - 1) >> sh;
    nmap = nmap < cmap_cap ? nmap : cmap_cap;
    const bool want_tags = out_parent != nullptr || out_ordinal != nullptr;
    const bool nt = Q > kTagNtEntries;
    for (;;) {
        const int64_t t = next_ticket(ctl, &s_t);
        if (t >= nsuper) break;
        // ready flags of the super-tile's entries: bit k of km[s] is entry
        // (tile s, this thread, item k)
        uint32_t km[kBatchSuper];
#pragma unroll
        for (int s = 0; s < kBatchSuper; ++s) {
            const int64_t i0 = (t * kBatchSuper + s) * kTile + (int64_t)threadIdx.x * kItems;
            km[s] = 0;
            if (vec_ok && i0 + kItems <= Q) {
                const uint4 kv = *reinterpret_cast<const uint4 *>(keep + i0);
                const uint32_t w[4] = {kv.x, kv.y, kv.z, kv.w};
#pragma unroll
                for (int k = 0; k < kItems; ++k)
                    km[s] |= (((w[k >> 2] >> (8 * (k & 3))) & 0xffu) != 0 ? 1u : 0u) << k;
            } else {
                for (int k = 0; k < kItems; ++k)
                    if (i0 + k < Q && keep[i0 + k] != 0) km[s] |= 1u << k;
            }
        }
        int64_t ex[kBatchSuper];
        int64_t agg = 0;
#pragma unroll
        for (int s = 0; s < kBatchSuper; ++s) {
            int64_t tot;
            ex[s] = block_excl_scan(__popc(km[s]), s_wave, tot);
            if (threadIdx.x == 0) s_sub[s] = agg;
            agg += tot;
        }
        const int64_t pre = (int64_t)tile_prefix(desc, t, epoch, (uint64_t)agg, &s_b, ctl);
        if (pre + agg > out_cap && threadIdx.x == 0) raise_err(ctl, RO_ECAP);
        bool bad_range = false;
#pragma unroll 1
        for (int s = 0; s < kBatchSuper; ++s) {
            const int64_t i0 = (t * kBatchSuper + s) * kTile + (int64_t)threadIdx.x * kItems;
            uint32_t q[kItems];
            if (vec_ok && i0 + kItems <= Q) {
                const uint4 *qp = reinterpret_cast<const uint4 *>(queue + i0);
#pragma unroll
                for (int k = 0; k < kItems / 4; ++k) {
                    const uint4 x = qp[k];
                    q[4 * k] = x.x; q[4 * k + 1] = x.y; q[4 * k + 2] = x.z; q[4 * k + 3] = x.w;
                }
            } else {
#pragma unroll
                for (int k = 0; k < kItems; ++k) q[k] = i0 + k < Q ? queue[i0 + k] : 0u;
            }
            uint32_t live = 0;
#pragma unroll
            for (int k = 0; k < kItems; ++k) {
                if (km[s] & (1u << k)) {
                    if ((int64_t)q[k] >= N) bad_range = true;
                    else live |= 1u << k;
                }
            }
            uint32_t par[kItems], ord[kItems];
#pragma unroll
            for (int k = 0; k < kItems; ++k) {
                par[k] = 0xffffffffu;
                ord[k] = 0xffffffffu;
            }
            if (want_tags) {
                constexpr int H = RO_BATCH_LOOKUPS;
#pragma unroll
                for (int hf = 0; hf < kItems / H; ++hf) {
                    uint32_t cc[H], pp[H], oo[H];
#pragma unroll
                    for (int k = 0; k < H; ++k) cc[k] = q[hf * H + k];
                    tags_of<H>(cmap, nmap, sh, offsets, P, cc, (live >> (hf * H)) & ((1u << H) - 1u), pp, oo);
#pragma unroll
                    for (int k = 0; k < H; ++k) {
                        if ((live >> (hf * H + k)) & 1u) {
                            par[hf * H + k] = pp[k];
                            ord[hf * H + k] = oo[k];
                        }
                    }
                }
            }
            const int64_t base = pre + s_sub[s];
            const int64_t cnt_s = (s + 1 < kBatchSuper ? s_sub[s + 1] : agg) - s_sub[s];
            const int64_t lim = out_cap - base < cnt_s ? (out_cap - base > 0 ? out_cap - base : 0) : cnt_s;
#pragma unroll 1
            for (int which = 0; which < 3; ++which) {
                uint32_t *dst = which == 0 ? out_child : (which == 1 ? out_parent : out_ordinal);
                if (dst == nullptr) continue;
                int slot = (int)ex[s];
#pragma unroll
                for (int k = 0; k < kItems; ++k) {
                    if (km[s] & (1u << k)) {
                        s_out[slot] = which == 0 ? q[k] : (which == 1 ? par[k] : ord[k]);
                        ++slot;
                    }
                }
                __syncthreads();
                write_tags(dst, base, s_out, lim, nt);
                __syncthreads();
            }
        }
        if (bad_range) raise_err(ctl, RO_ERANGE);
        if (t == nsuper - 1 && threadIdx.x == 0) {
            const int64_t m = pre + agg;
            if (n_out) *n_out = m;
            if (n_batches) *n_batches = (m + B - 1) / B;
        }
    }
    ticket_done(ctl, epoch, desc, desc_cap, &s_last);
}

// First index i in [0, n) with a[i] > x (n if none), for K keys at once
// (n >= 1, a nondecreasing).  The halving is branch-free and its trip count
// depends on n only, so the K searches step together and each step's K loads
// are in flight at the same time.
template <int K>
__device__ __forceinline__ void upper_bound_k(const int64_t *a, int64_t n, const int64_t (&x)[K], int64_t (&r)[K])
{
    int64_t base[K];
#pragma unroll
    for (int k = 0; k < K; ++k) base[k] = 0;
    int64_t len = n;
    while (len > 1) {
        const int64_t half = len >> 1;
        int64_t v[K];
#pragma unroll
        for (int k = 0; k < K; ++k) v[k] = a[base[k] + half];
#pragma unroll
        for (int k = 0; k < K; ++k) base[k] = v[k] <= x[k] ? base[k] + half : base[k];
        len -= half;
    }
#pragma unroll
    for (int k = 0; k < K; ++k) r[k] = base[k] + (a[base[k]] <= x[k] ? 1 : 0);
}

// Every queue entry is ready (no mask): the FIFO compaction is the identity,
// slot i holds queue[i], so no scan is needed and each entry is independent.
// A block takes 1024 consecutive entries, lane-contiguous, so every load and
// store instruction of a wave covers 256 contiguous bytes.
constexpr int kAllPer = 4;

template <bool kByMap>
__global__ __launch_bounds__(kBlock) void k_batch_all(
    const uint32_t *__restrict__ queue, int64_t Q, const int64_t *__restrict__ offsets, int64_t P,
    const uint2 *__restrict__ cmap, int64_t cmap_cap, int32_t B, uint32_t *__restrict__ out_child,
    uint32_t *__restrict__ out_parent, uint32_t *__restrict__ out_ordinal, int64_t out_cap, int64_t *n_out,
    int64_t *n_batches, const uint32_t *__restrict__ cpar, int64_t cpar_n, Ctl *ctl)
{
    const int64_t N = cpar ? min64(offsets[P], cpar_n) : offsets[P];   // ids past the map are out of range
    const int sh = map_shift(offsets[P], P);     // the map's block size, as k_batch_cmap built it
    int64_t nmap = (N + (1 << sh) - 1) >> sh;
    nmap = nmap < cmap_cap ? nmap : cmap_cap;
    const bool want_tags = out_parent != nullptr || out_ordinal != nullptr;
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        if (Q > out_cap) raise_err(ctl, RO_ECAP);
        if (n_out) *n_out = Q;
        if (n_batches) *n_batches = (Q + B - 1) / B;
    }
    const int64_t lim = Q < out_cap ? Q : out_cap;
    bool bad_range = false;
    for (int64_t i0 = (int64_t)blockIdx.x * (kBlock * kAllPer); i0 < Q;
         i0 += (int64_t)gridDim.x * (kBlock * kAllPer)) {
        uint32_t q[kAllPer];
#pragma unroll
        for (int k = 0; k < kAllPer; ++k) {
            const int64_t i = i0 + k * kBlock + threadIdx.x;
            q[k] = i < Q ? queue[i] : 0u;
        }
        // the entries' parents: from the stream's own map, from the coarse
        // map (all lookups in flight together), or without it from one
        // lockstep search of the offsets (ids out of range search for N - 1
        // and are reported below)
        uint32_t par[kAllPer], ord[kAllPer];
        if (want_tags && !kByMap) {
            if (nmap == 0) {
                int64_t key[kAllPer], pp[kAllPer];
#pragma unroll
                for (int k = 0; k < kAllPer; ++k) key[k] = (int64_t)q[k] < N ? (int64_t)q[k] : N - 1;
                if (N > 0) {
                    upper_bound_k<kAllPer>(offsets, P + 1, key, pp);
#pragma unroll
                    for (int k = 0; k < kAllPer; ++k) {
                        par[k] = (uint32_t)(pp[k] - 1);
                        ord[k] = (uint32_t)(key[k] - offsets[pp[k] - 1]);
                    }
                }
            } else {
                uint32_t live = 0;
#pragma unroll
                for (int k = 0; k < kAllPer; ++k)
                    if (i0 + k * kBlock + threadIdx.x < Q && (int64_t)q[k] < N) live |= 1u << k;
                tags_of<kAllPer>(cmap, nmap, sh, offsets, P, q, live, par, ord);
            }
        }
#pragma unroll
        for (int k = 0; k < kAllPer; ++k) {
            const int64_t i = i0 + k * kBlock + threadIdx.x;
            if (i >= Q) continue;
            const int64_t c = q[k];
            if (c >= N) {
                bad_range = true;
                continue;
            }
            if (i >= lim) continue;
            if (out_child) out_child[i] = q[k];
            if (want_tags) {
                if constexpr (kByMap) {
                    const int64_t p = (int64_t)cpar[c];
                    par[k] = (uint32_t)p;
                    ord[k] = (uint32_t)(c - offsets[p]);
                }
                if (out_parent) out_parent[i] = par[k];
                if (out_ordinal) out_ordinal[i] = ord[k];
            }
        }
    }
    if (bad_range) raise_err(ctl, RO_ERANGE);
}

hipError_t launch_batch(const Launch &L, const uint32_t *queue, const uint8_t *keep,
                        int64_t Q, const int64_t *offsets, int64_t P, int32_t B,
                        uint32_t *out_child, uint32_t *out_parent, uint32_t *out_ordinal,
                        int64_t out_cap, int64_t *n_out, int64_t *n_batches, uint32_t *cmap_words,
                        int64_t cmap_words_cap, const uint8_t *barrier, const uint32_t *cpar, int64_t cpar_n)
{
    // the coarse map takes two words a block; its parent field keeps a flag bit
    uint2 *cmap = reinterpret_cast<uint2 *>(cmap_words);
    int64_t cmap_cap = P < ((int64_t)1 << 31) ? cmap_words_cap / 2 : 0;
    // The coarse map costs a search per 128 children; a short unmasked queue
    // (fewer entries than parents, such as one wave of a stream) searches
    // the offsets directly instead and skips the extra launch.
    const bool tags = out_parent != nullptr || out_ordinal != nullptr;
    const bool use_map = cpar == nullptr && (tags || barrier != nullptr) && cmap_cap > 0 &&
                         !(keep == nullptr && barrier == nullptr && Q < P);
    if (use_map) {
        const int64_t grid_m = (int64_t)L.num_cus * 4;
        RO_LAUNCH(L, RO_K_BATCH_SAMPLES, k_batch_cmap, dim3((unsigned)grid_m), dim3(256), 0, L.stream,
                  offsets, P, cmap, cmap_cap);
    } else {
        cmap_cap = 0;
    }
    if (keep == nullptr && barrier == nullptr) {
        int64_t grid_a = (Q + kBlock * kAllPer - 1) / (kBlock * kAllPer);
        grid_a = grid_a < 1 ? 1 : (grid_a > (int64_t)L.num_cus * 8 ? (int64_t)L.num_cus * 8 : grid_a);
        if (cpar)
            RO_LAUNCH(L, RO_K_BATCH, k_batch_all<true>, dim3((unsigned)grid_a), dim3(kBlock), 0, L.stream, queue,
                      Q, offsets, P, cmap, cmap_cap, B, out_child, out_parent, out_ordinal, out_cap, n_out,
                      n_batches, cpar, cpar_n, L.ctl);
        else
            RO_LAUNCH(L, RO_K_BATCH, k_batch_all<false>, dim3((unsigned)grid_a), dim3(kBlock), 0, L.stream, queue,
                      Q, offsets, P, cmap, cmap_cap, B, out_child, out_parent, out_ordinal, out_cap, n_out,
                      n_batches, cpar, cpar_n, L.ctl);
        return hipGetLastError();
    }
    const int64_t ntiles = Q > 0 ? (Q + kTile - 1) / kTile : 1;
    const int64_t cap_grid = (int64_t)L.num_cus * 4;
    const int64_t grid = ntiles < cap_grid ? ntiles : cap_grid;
    const bool aligned = ((reinterpret_cast<uintptr_t>(queue) | reinterpret_cast<uintptr_t>(keep)) & 15u) == 0;
    if (barrier == nullptr && cpar == nullptr) {
        const int64_t nsuper = (ntiles + kBatchSuper - 1) / kBatchSuper;
        const int64_t grid_k = nsuper < cap_grid ? nsuper : cap_grid;
        RO_LAUNCH(L, RO_K_BATCH, k_batch_keep, dim3((unsigned)grid_k), dim3(kBlock), 0, L.stream, queue, keep, Q,
                  offsets, P, cmap, cmap_cap, B, out_child, out_parent, out_ordinal, out_cap, n_out, n_batches,
                  L.ctl, L.desc, L.desc_cap, nsuper, aligned ? 1 : 0);
        return hipGetLastError();
    }
    if (cpar)
        RO_LAUNCH(L, RO_K_BATCH, k_batch<true>, dim3((unsigned)grid), dim3(kBlock), 0, L.stream, queue, keep, Q,
                  offsets, P, cmap, cmap_cap, B, out_child, out_parent, out_ordinal, out_cap, n_out, n_batches,
                  barrier, cpar, cpar_n, L.ctl, L.desc, L.desc_cap, ntiles, aligned ? 1 : 0);
    else
        RO_LAUNCH(L, RO_K_BATCH, k_batch<false>, dim3((unsigned)grid), dim3(kBlock), 0, L.stream, queue, keep, Q,
                  offsets, P, cmap, cmap_cap, B, out_child, out_parent, out_ordinal, out_cap, n_out, n_batches,
                  barrier, cpar, cpar_n, L.ctl, L.desc, L.desc_cap, ntiles, aligned ? 1 : 0);
    return hipGetLastError();
}

}  // namespace ro
