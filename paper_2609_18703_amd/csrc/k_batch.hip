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

// Coarse child -> parent map: cmap[j] = parent of child j << kCmapShift.  A
// child's parent then lies between cmap[j] and cmap[j+1], a handful of
// offsets that sit in L2.
constexpr int kCmapShift = 6;

__global__ void k_batch_cmap(const int64_t *__restrict__ offsets, int64_t P, uint32_t *__restrict__ cmap,
                             int64_t cmap_cap)
{
    const int64_t N = offsets[P];
    int64_t nmap = (N + (1 << kCmapShift) - 1) >> kCmapShift;
    nmap = nmap < cmap_cap ? nmap : cmap_cap;
    for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < nmap;
         j += (int64_t)gridDim.x * blockDim.x)
        cmap[j] = (uint32_t)(upper_bound_g(offsets, 0, P + 1, j << kCmapShift) - 1);
}

// Parent of child c < N.
__device__ __forceinline__ int64_t parent_of(const uint32_t *__restrict__ cmap, int64_t nmap,
                                             const int64_t *__restrict__ offsets, int64_t P, int64_t c)
{
    const int64_t j = c >> kCmapShift;
    if (j >= nmap) return upper_bound_g(offsets, 0, P + 1, c) - 1;
    const int64_t lo = cmap[j];
    const int64_t hi = j + 1 < nmap ? (int64_t)cmap[j + 1] : P - 1;
    return upper_bound_g(offsets, lo, hi + 1, c) - 1;
}

template <bool kByMap>
__global__ __launch_bounds__(kBlock) void k_batch(
    const uint32_t *__restrict__ queue, const uint8_t *__restrict__ keep, int64_t Q,
    const int64_t *__restrict__ offsets, int64_t P, const uint32_t *__restrict__ cmap, int64_t cmap_cap,
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
    int64_t nmap = (N + (1 << kCmapShift) - 1) >> kCmapShift;
    nmap = nmap < cmap_cap ? nmap : cmap_cap;
    const bool want_tags = out_parent != nullptr || out_ordinal != nullptr;
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
        // lineage tags of the ready entries (independent lookups, all in
        // flight); an entry of a barred parent is not ready
        uint32_t par[kItems], ord[kItems];
        bool bad_range = false;
#pragma unroll
        for (int k = 0; k < kItems; ++k) {
            par[k] = 0xffffffffu;
            ord[k] = 0xffffffffu;
            if (kmask & (1u << k)) {
                const int64_t c = q[k];
                if (c >= N) {
                    bad_range = true;
                } else if (want_tags || barrier) {
                    int64_t p;
                    if constexpr (kByMap) p = (int64_t)cpar[c];
                    else p = parent_of(cmap, nmap, offsets, P, c);
                    if (barrier && barrier[p]) {
                        kmask &= ~(1u << k);                             // suppressed: takes no slot
                    } else {
                        par[k] = (uint32_t)p;
                        ord[k] = (uint32_t)(c - offsets[p]);
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
            for (int64_t j = threadIdx.x; j < lim; j += kBlock) dst[base + j] = s_out[j];
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
    const uint32_t *__restrict__ cmap, int64_t cmap_cap, int32_t B, uint32_t *__restrict__ out_child,
    uint32_t *__restrict__ out_parent, uint32_t *__restrict__ out_ordinal, int64_t out_cap, int64_t *n_out,
    int64_t *n_batches, const uint32_t *__restrict__ cpar, int64_t cpar_n, Ctl *ctl)
{
    const int64_t N = cpar ? min64(offsets[P], cpar_n) : offsets[P];   // ids past the map are out of range
    int64_t nmap = (N + (1 << kCmapShift) - 1) >> kCmapShift;
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
        // without the coarse map, the entries' parents come from one
        // lockstep search of the offsets (ids out of range search for N - 1
        // and are reported below)
        int64_t par[kAllPer];
        if (!kByMap && want_tags && nmap == 0) {
            int64_t key[kAllPer];
#pragma unroll
            for (int k = 0; k < kAllPer; ++k) key[k] = (int64_t)q[k] < N ? (int64_t)q[k] : N - 1;
            if (N > 0) {
                upper_bound_k<kAllPer>(offsets, P + 1, key, par);
#pragma unroll
                for (int k = 0; k < kAllPer; ++k) par[k] -= 1;
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
                int64_t p;
                if constexpr (kByMap) p = (int64_t)cpar[c];
                else p = nmap == 0 ? par[k] : parent_of(cmap, nmap, offsets, P, c);
                if (out_parent) out_parent[i] = (uint32_t)p;
                if (out_ordinal) out_ordinal[i] = (uint32_t)(c - offsets[p]);
            }
        }
    }
    if (bad_range) raise_err(ctl, RO_ERANGE);
}

hipError_t launch_batch(const Launch &L, const uint32_t *queue, const uint8_t *keep,
                        int64_t Q, const int64_t *offsets, int64_t P, int32_t B,
                        uint32_t *out_child, uint32_t *out_parent, uint32_t *out_ordinal,
                        int64_t out_cap, int64_t *n_out, int64_t *n_batches, uint32_t *cmap,
                        int64_t cmap_cap, const uint8_t *barrier, const uint32_t *cpar, int64_t cpar_n)
{
    // The coarse map costs a search per 64 children; a short unmasked queue
    // (fewer entries than parents, such as one wave of a stream) searches
    // the offsets directly instead and skips the extra launch.
    const bool tags = out_parent != nullptr || out_ordinal != nullptr;
    const bool use_map = cpar == nullptr && (tags || barrier != nullptr) &&
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
