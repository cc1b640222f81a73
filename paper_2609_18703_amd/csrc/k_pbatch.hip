// Parent-bound reservation on gfx950.
//
// RayOrch (arXiv 2609.18703), Sec. 4 "Scheduling Ready Grains": a
// parent-bound reservation takes up to B siblings of the first ready parent,
// and the entries it leaves keep their order.  Run to the end of the queue,
// the reservations have a closed form that needs no sequential loop: rank
// every ready entry within its parent in queue order; the entries of ranks
// jB .. jB + B - 1 of one parent leave together (the head is always the
// earliest entry left, and it always opens such a group, since the group
// before it in its parent left whole), and the groups leave in the queue
// order of their first entries.
//
// On the GPU: the ready entries are compacted in queue order (the FIFO
// batch's compaction), sorted by parent with a stable LSD radix sort that
// carries each entry's child and queue position (so each parent's entries
// stay in queue order and an entry's rank is its distance from its parent's
// first sorted entry), every group's first entry marks its queue position
// with the group size, one scan over queue positions numbers the groups and
// gives their slot offsets, and every entry is written to its group's slot
// range.
#include "ro_device.h"

namespace ro {

constexpr int kRTile = (int)kPbTile;         // sort tile: 8 entries per thread
constexpr int kRMaxBits = 9;                 // digit width; at most 512 buckets
constexpr int kRMaxBuckets = 1 << kRMaxBits;
constexpr int kRSpan = (int)kPbSpan;          // tiles per histogram column
constexpr int64_t kRSpanLen = (int64_t)kRTile * kRSpan;
static_assert(kRMaxBuckets == kPbMaxBuckets, "histogram layout");

__device__ __forceinline__ int64_t tiles_of(int64_t m) { return (m + kRTile - 1) / kRTile; }

// Digit histograms per span of kRSpan tiles, digit-major:
// hist[d * spans_cap + st].  Spans past the ready count write zeros, so the
// scan over all spans_cap columns is the scan over the real ones.
__global__ __launch_bounds__(kBlock) void k_rs_hist(const uint32_t *__restrict__ keys, const int64_t *m_dev,
                                                   int shift, int width, int32_t *__restrict__ hist,
                                                   int64_t spans_cap)
{
    __shared__ int32_t s_h[kRMaxBuckets];
    const int64_t M = *m_dev;
    const int nb = 1 << width;
    const uint32_t mask = (uint32_t)nb - 1;
    for (int64_t st = blockIdx.x; st < spans_cap; st += gridDim.x) {
        for (int d = threadIdx.x; d < nb; d += kBlock) s_h[d] = 0;
        __syncthreads();
        const int64_t i0 = st * kRSpanLen;
        const int64_t i1 = min64(i0 + kRSpanLen, M);
        // four keys a thread at a time (a span starts 16-byte aligned)
        for (int64_t i = i0 + 4 * (int64_t)threadIdx.x; i < i1; i += 4 * kBlock) {
            if (i + 4 <= i1) {
                const uint4 k4 = *reinterpret_cast<const uint4 *>(keys + i);
                atomicAdd(&s_h[(k4.x >> shift) & mask], 1);
                atomicAdd(&s_h[(k4.y >> shift) & mask], 1);
                atomicAdd(&s_h[(k4.z >> shift) & mask], 1);
                atomicAdd(&s_h[(k4.w >> shift) & mask], 1);
            } else {
                for (int64_t j = i; j < i1; ++j) atomicAdd(&s_h[(keys[j] >> shift) & mask], 1);
            }
        }
        __syncthreads();
        for (int d = threadIdx.x; d < nb; d += kBlock) hist[(int64_t)d * spans_cap + st] = s_h[d];
        __syncthreads();
    }
}

// Stable scatter of one digit pass.  A workgroup takes a span of kRSpan
// tiles in order, starting each digit at the span's offset from the
// histogram scan.  Per tile: the tile's digit counts (LDS atomics) give where
// each digit's run starts in the tile; each wave ranks its own quarter of
// the tile (eight rounds of 64 entries, in order) among the quarter's entries
// of the same digit, with a wave-private running count per digit plus the
// lanes below with the same digit (one ballot per digit bit); the waves'
// counts become per-digit bases, the tile is sorted by digit in LDS and
// written out so that consecutive lanes store consecutive places of a
// digit's run; the span's digit offsets then move past the tile.  Values are
// (child << 32 | queue position); vin == nullptr: built from the compacted
// children and the positions.
__global__ __launch_bounds__(kBlock) void k_rs_scatter(const uint32_t *__restrict__ kin,
                                                      const uint64_t *__restrict__ vin,
                                                      const uint32_t *__restrict__ kc, uint32_t *__restrict__ kout,
                                                      uint64_t *__restrict__ vout, const int64_t *m_dev, int shift,
                                                      int width, const int64_t *__restrict__ hoff, int64_t spans_cap)
{
    constexpr int kWaves = kBlock / 64;
    constexpr int kQuarter = kRTile / kWaves;          // entries per wave
    constexpr int kWRounds = kQuarter / 64;
    static_assert(kRMaxBuckets == 2 * kBlock, "two digits per thread");
    __shared__ int64_t s_base[kRMaxBuckets];
    __shared__ int32_t s_tex[kRMaxBuckets];
    __shared__ int32_t s_cnt[kWaves][kRMaxBuckets];
    __shared__ uint32_t s_k[kRTile];
    __shared__ uint64_t s_v[kRTile];
    __shared__ int64_t s_wave[kWaves];
    const int64_t M = *m_dev;
    const int64_t nspans = (M + kRSpanLen - 1) / kRSpanLen;
    const int nb = 1 << width;
    const uint32_t mask = (uint32_t)nb - 1;
    const int wave = (int)(threadIdx.x >> 6), lane = lane_id();
    const uint64_t lt = (1ull << lane) - 1;
    int32_t *cnt = s_cnt[wave];
    const int d0 = 2 * (int)threadIdx.x, d1 = d0 + 1;
    for (int64_t sp = blockIdx.x; sp < nspans; sp += gridDim.x) {
        if (d0 < nb) s_base[d0] = hoff[(int64_t)d0 * spans_cap + sp];
        if (d1 < nb) s_base[d1] = hoff[(int64_t)d1 * spans_cap + sp];
        for (int64_t t0 = sp * kRSpanLen; t0 < min64((sp + 1) * kRSpanLen, M); t0 += kRTile) {
            // load the tile; count its digits
            for (int d = threadIdx.x; d < nb; d += kBlock) s_tex[d] = 0;
            __syncthreads();
            const int64_t i0 = t0 + (int64_t)wave * kQuarter;
            uint32_t key[kWRounds];
            uint64_t val[kWRounds];
            int32_t rank[kWRounds];
#pragma unroll
            for (int r = 0; r < kWRounds; ++r) {
                const int64_t i = i0 + r * 64 + lane;
                const bool valid = i < M;
                key[r] = valid ? kin[i] : 0;
                val[r] = !valid ? 0 : (vin ? vin[i] : ((uint64_t)kc[i] << 32 | (uint64_t)i));
                if (valid) atomicAdd(&s_tex[(key[r] >> shift) & mask], 1);
            }
            for (int d = lane; d < nb; d += 64) cnt[d] = 0;
            __syncthreads();
            // the tile's digit counts -> where each digit's run starts in the tile
            const int32_t c0 = d0 < nb ? s_tex[d0] : 0;
            const int32_t c1 = d1 < nb ? s_tex[d1] : 0;
            int64_t tot;
            const int32_t ex = (int32_t)block_excl_scan((int64_t)c0 + c1, s_wave, tot);
            if (d0 < nb) s_tex[d0] = ex;
            if (d1 < nb) s_tex[d1] = ex + c0;
            // this wave's quarter: ranks among its entries of the same digit
#pragma unroll
            for (int r = 0; r < kWRounds; ++r) {
                const bool valid = i0 + r * 64 + lane < M;
                const uint32_t d = (key[r] >> shift) & mask;
                uint64_t peers = __ballot(valid);
                for (int b = 0; b < width; ++b) {
                    const bool bit = (d >> b) & 1u;
                    const uint64_t m = __ballot(valid && bit);
                    peers &= bit ? m : ~m;
                }
                const int below = (int)__popcll(peers & lt);
                rank[r] = valid ? cnt[d] + below : 0;
                __builtin_amdgcn_wave_barrier();
                if (valid && below == 0) cnt[d] += (int32_t)__popcll(peers);
                __builtin_amdgcn_wave_barrier();
            }
            __syncthreads();
            // wave counts -> wave bases inside the tile
            for (int d = threadIdx.x; d < nb; d += kBlock) {
                int32_t run = s_tex[d];
#pragma unroll
                for (int w = 0; w < kWaves; ++w) {
                    const int32_t x = s_cnt[w][d];
                    s_cnt[w][d] = run;
                    run += x;
                }
            }
            __syncthreads();
#pragma unroll
            for (int r = 0; r < kWRounds; ++r) {
                if (i0 + r * 64 + lane >= M) continue;
                const int32_t lp = cnt[(key[r] >> shift) & mask] + rank[r];
                s_k[lp] = key[r];
                s_v[lp] = val[r];
            }
            __syncthreads();
            const int n_t = (int)min64(kRTile, M - t0);
            for (int j = threadIdx.x; j < n_t; j += kBlock) {
                const uint32_t k = s_k[j];
                const uint32_t d = (k >> shift) & mask;
                const int64_t g = s_base[d] + (j - s_tex[d]);
                kout[g] = k;
                vout[g] = s_v[j];
            }
            __syncthreads();
            // the span's digit offsets move past this tile
            if (d0 < nb) s_base[d0] += c0;
            if (d1 < nb) s_base[d1] += c1;
        }
        __syncthreads();
    }
}

// First and end sorted index of every parent that has ready entries.  After
// an error (an id out of range leaves its entry's parent unset) the parents
// are not trusted: every kernel from here on returns at once.
__global__ void k_pb_bounds(const uint32_t *__restrict__ key, const int64_t *m_dev, int64_t P,
                            uint32_t *__restrict__ pstart, uint32_t *__restrict__ pend, uint32_t *__restrict__ fsize,
                            Ctl *ctl)
{
    if (read_err(ctl) != 0) return;
    const int64_t M = *m_dev;
    for (int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; s < M; s += (int64_t)gridDim.x * blockDim.x) {
        fsize[s] = 0;                            // group sizes are set next, at group firsts only
        const uint32_t p = key[s];
        if ((int64_t)p >= P) continue;
        if (s == 0 || key[s - 1] != p) pstart[p] = (uint32_t)s;
        if (s == M - 1 || key[s + 1] != p) pend[p] = (uint32_t)(s + 1);
    }
}

// The queue position of every group's first entry (rank a multiple of B)
// gets the group's size; the other positions stay zero.
__global__ void k_pb_firsts(const uint32_t *__restrict__ key, const uint64_t *__restrict__ val, const int64_t *m_dev,
                            int64_t P, const uint32_t *__restrict__ pstart, const uint32_t *__restrict__ pend,
                            int32_t B, uint32_t *__restrict__ fsize, Ctl *ctl)
{
    if (read_err(ctl) != 0) return;
    const int64_t M = *m_dev;
    for (int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; s < M; s += (int64_t)gridDim.x * blockDim.x) {
        const uint32_t p = key[s];
        if ((int64_t)p >= P) continue;
        const int64_t r = s - (int64_t)pstart[p];
        if (r % B != 0) continue;
        const int64_t left = (int64_t)pend[p] - s;
        fsize[(uint32_t)val[s]] = (uint32_t)(left < B ? left : B);
    }
}

// Groups in queue order of their first entries: one pass over the queue
// positions with two look-back chains (groups so far, entries so far).  A
// group's first position gets its batch number; batch_off[b] is batch b's
// first slot; the last tile writes batch_off[n_batches] and the totals.
__global__ __launch_bounds__(kBlock) void k_pb_scan(const uint32_t *__restrict__ fsize, const int64_t *m_dev,
                                                   int64_t out_cap, uint32_t *__restrict__ bidx,
                                                   int64_t *__restrict__ batch_off, int64_t batch_cap, int64_t *n_out,
                                                   int64_t *n_batches, Ctl *ctl, uint64_t *desc, uint64_t *desc_b,
                                                   int64_t desc_cap)
{
    const uint32_t epoch = scan_epoch(ctl);
    __shared__ int64_t s_wave[kBlock / 64];
    __shared__ uint64_t s_b2[2];
    __shared__ int64_t s_t;
    __shared__ int32_t s_last;
    const int64_t M = *m_dev;
    const int64_t ntiles = (M + kTile - 1) / kTile;
    if (M > out_cap && blockIdx.x == 0 && threadIdx.x == 0) raise_err(ctl, RO_ECAP);
    if (M == 0 && blockIdx.x == 0 && threadIdx.x == 0) {
        if (batch_cap < 1) raise_err(ctl, RO_ECAP);
        else batch_off[0] = 0;
        if (n_out) *n_out = 0;
        if (n_batches) *n_batches = 0;
    }
    for (;;) {
        const int64_t t = next_ticket(ctl, &s_t);
        if (t >= ntiles) break;
        const int64_t i0 = t * kTile + (int64_t)threadIdx.x * kItems;
        uint32_t f[kItems];
        int64_t cnt = 0, sum = 0;
#pragma unroll
        for (int k = 0; k < kItems; ++k) {
            const int64_t i = i0 + k;
            f[k] = i < M ? fsize[i] : 0u;
            cnt += f[k] != 0;
            sum += f[k];
        }
        int64_t tc, ts;
        const int64_t ec = block_excl_scan(cnt, s_wave, tc);
        const int64_t es = block_excl_scan(sum, s_wave, ts);
        uint64_t pc, ps;
        tile_prefix2(desc, (uint64_t)tc, desc_b, (uint64_t)ts, t, epoch, s_b2, pc, ps, ctl);
        int64_t b = (int64_t)pc + ec, o = (int64_t)ps + es;
        bool over = false;
#pragma unroll
        for (int k = 0; k < kItems; ++k) {
            if (f[k] == 0) continue;
            bidx[i0 + k] = (uint32_t)b;
            if (b < batch_cap) batch_off[b] = o;
            else over = true;
            ++b;
            o += f[k];
        }
        if (over) raise_err(ctl, RO_ECAP);
        if (t == ntiles - 1 && threadIdx.x == 0) {
            const int64_t nbat = (int64_t)pc + tc;
            if (nbat < batch_cap) batch_off[nbat] = (int64_t)ps + ts;
            else raise_err(ctl, RO_ECAP);
            if (n_out) *n_out = (int64_t)ps + ts;
            if (n_batches) *n_batches = nbat;
        }
    }
    ticket_done(ctl, epoch, desc, desc_cap, &s_last);
}

// Every entry to its group's slots: slot = batch_off[batch of the group's
// first entry] + rank mod B.
__global__ void k_pb_place(const uint32_t *__restrict__ key, const uint64_t *__restrict__ val, const int64_t *m_dev,
                           int64_t P, const uint32_t *__restrict__ pstart, int32_t B, const uint32_t *__restrict__ bidx,
                           const int64_t *__restrict__ batch_off, const int64_t *__restrict__ offsets, uint32_t *__restrict__ out_child,
                           uint32_t *__restrict__ out_parent, uint32_t *__restrict__ out_ordinal, int64_t out_cap,
                           Ctl *ctl)
{
    if (read_err(ctl) != 0) return;          // a capacity error leaves the outputs unwritten
    const int64_t M = *m_dev;
    if (M > out_cap) return;
    for (int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; s < M; s += (int64_t)gridDim.x * blockDim.x) {
        const uint32_t p = key[s];
        if ((int64_t)p >= P) continue;
        const int64_t st = (int64_t)pstart[p];
        const int64_t r = s - st;
        const uint32_t qf = (uint32_t)val[st + (r / B) * B];
        const int64_t b = (int64_t)bidx[qf];
        const int64_t slot = batch_off[b] + r % B;
        const uint32_t c = (uint32_t)(val[s] >> 32);
        if (out_child) out_child[slot] = c;
        if (out_parent) out_parent[slot] = p;
        if (out_ordinal) out_ordinal[slot] = (uint32_t)((int64_t)c - offsets[p]);
    }
}

static int64_t grid_for(const Launch &L, int64_t n, int64_t per_block)
{
    int64_t grid = (n + per_block - 1) / per_block;
    return grid < 1 ? 1 : (grid > (int64_t)L.num_cus * 8 ? (int64_t)L.num_cus * 8 : grid);
}

hipError_t launch_batch_parent(const Launch &L, const uint32_t *queue, const uint8_t *keep, int64_t Q,
                               const int64_t *offsets, int64_t P, int32_t B, uint32_t *out_child,
                               uint32_t *out_parent, uint32_t *out_ordinal, int64_t out_cap, int64_t *batch_off,
                               int64_t batch_cap, int64_t *n_out, int64_t *n_batches, uint32_t *cmap,
                               int64_t cmap_cap, const uint8_t *barrier, const PbWs &w)
{
    // ready entries in queue order: children and parents, count in w.m
    hipError_t e = launch_batch(L, queue, keep, Q, offsets, P, B, w.kc, w.k[0], nullptr, Q, w.m, w.m + 1, cmap,
                                cmap_cap, barrier);
    if (e != hipSuccess) return e;
    // stable sort by parent: digits of at most kRMaxBits bits, as few passes as the parent ids need
    int bits = 0;
    while (bits < 32 && ((uint64_t)1 << bits) < (uint64_t)P) ++bits;
    const int passes = bits == 0 ? 1 : (bits + kRMaxBits - 1) / kRMaxBits;   // one pass of width 0 copies
    const int64_t spans_cap = (Q + kRSpanLen - 1) / kRSpanLen > 0 ? (Q + kRSpanLen - 1) / kRSpanLen : 1;
    const int64_t gsort = spans_cap < (int64_t)L.num_cus * 4 ? spans_cap : (int64_t)L.num_cus * 4;
    int cur = 0;
    const uint64_t *vals = nullptr;          // built from the compaction in the first pass
    for (int pass = 0, shift = 0; pass < passes; ++pass) {
        const int width = (bits - shift) < kRMaxBits ? (bits - shift) : kRMaxBits;
        RO_LAUNCH(L, RO_K_PBATCH_SORT, k_rs_hist, dim3((unsigned)gsort), dim3(kBlock), 0, L.stream, w.k[cur], w.m,
                  shift, width, w.hist, spans_cap);
        e = launch_expand(L, w.hist, (int64_t)(1 << width) * spans_cap, w.hoff, nullptr, nullptr, 0);
        if (e != hipSuccess) return e;
        RO_LAUNCH(L, RO_K_PBATCH_SORT, k_rs_scatter, dim3((unsigned)gsort), dim3(kBlock), 0, L.stream, w.k[cur],
                  vals, w.kc, w.k[1 - cur], w.v[1 - cur], w.m, shift, width, w.hoff, spans_cap);
        vals = w.v[1 - cur];
        cur = 1 - cur;
        shift += width;
    }
    const uint32_t *keys = w.k[cur];
    const int64_t g = grid_for(L, Q, kBlock);
    RO_LAUNCH(L, RO_K_PBATCH, k_pb_bounds, dim3((unsigned)g), dim3(kBlock), 0, L.stream, keys, w.m, P, w.pstart,
              w.pend, w.fsize, L.ctl);
    RO_LAUNCH(L, RO_K_PBATCH, k_pb_firsts, dim3((unsigned)g), dim3(kBlock), 0, L.stream, keys, vals, w.m, P,
              w.pstart, w.pend, B, w.fsize, L.ctl);
    const int64_t ntiles = (Q + kTile - 1) / kTile > 0 ? (Q + kTile - 1) / kTile : 1;
    const int64_t gscan = ntiles < (int64_t)L.num_cus * 4 ? ntiles : (int64_t)L.num_cus * 4;
    if (2 * ntiles > L.desc_cap) return hipErrorInvalidValue;
    RO_LAUNCH(L, RO_K_PBATCH, k_pb_scan, dim3((unsigned)gscan), dim3(kBlock), 0, L.stream, w.fsize, w.m, out_cap,
              w.bidx, batch_off, batch_cap, n_out, n_batches, L.ctl, L.desc, L.desc + ntiles, L.desc_cap);
    RO_LAUNCH(L, RO_K_PBATCH, k_pb_place, dim3((unsigned)g), dim3(kBlock), 0, L.stream, keys, vals, w.m, P,
              w.pstart, B, w.bidx, batch_off, offsets, out_child, out_parent, out_ordinal, out_cap, L.ctl);
    return hipGetLastError();
}

}  // namespace ro
