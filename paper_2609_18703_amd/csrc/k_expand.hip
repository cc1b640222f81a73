// F.expand on gfx950: child counts -> Expansion offsets (decoupled look-back
// scan) and per-child lineage keys (load-balanced over children).
//
// RayOrch (arXiv 2609.18703), Sec. 4 "Lineage State and Parent Completion":
// each parent's Expansion is its ordered child set and every child carries
// (parent, immutable zero-based ordinal).
#include "ro_device.h"

namespace ro {

// Counts int32[P] -> offsets int64[P+1].  One tile = 4096 counts, 16 per
// thread.  Tiles come from the ticket; the exclusive prefix of each tile
// comes from the look-back.
__global__ __launch_bounds__(kBlock) void k_expand_scan(const int32_t *__restrict__ counts, int64_t P,
                                                        int64_t *__restrict__ offsets, int64_t child_cap,
                                                        int want_tags, Ctl *ctl, uint64_t *desc,
                                                        int64_t desc_cap, int64_t ntiles)
{
    const uint32_t epoch = scan_epoch(ctl);
    __shared__ int64_t s_wave[kBlock / 64];
    __shared__ uint64_t s_b;
    __shared__ int64_t s_t;
    __shared__ int32_t s_last;
    for (;;) {
        const int64_t t = next_ticket(ctl, &s_t);
        if (t >= ntiles) break;
        const int64_t i0 = t * kTile + (int64_t)threadIdx.x * kItems;
        int32_t v[kItems];
        int64_t sum = 0;
        bool bad = false;
#pragma unroll
        for (int k = 0; k < kItems; ++k) {
            const int64_t i = i0 + k;
            int32_t x = i < P ? counts[i] : 0;
            if (x < 0) { bad = true; x = 0; }
            v[k] = x;
            sum += x;
        }
        if (bad) raise_err(ctl, RO_EINVAL);
        int64_t tot;
        const int64_t ex = block_excl_scan(sum, s_wave, tot);
        const uint64_t pre = tile_prefix(desc, t, epoch, (uint64_t)tot, &s_b, ctl);
        int64_t run = (int64_t)pre + ex;
#pragma unroll
        for (int k = 0; k < kItems; ++k) {
            const int64_t i = i0 + k;
            if (i < P) offsets[i] = run;
            run += v[k];
        }
        if (t == ntiles - 1 && threadIdx.x == 0) {
            const int64_t n = (int64_t)pre + tot;
            offsets[P] = n;
            if (pre >= kSat || n >= ((int64_t)1 << 32)) raise_err(ctl, RO_EOVERFLOW);
            else if (want_tags && n > child_cap) raise_err(ctl, RO_ECAP);
        }
    }
    ticket_done(ctl, epoch, desc, desc_cap, &s_last);
}

// Lineage keys: child c -> (p, c - offsets[p]).  Each thread owns 16
// consecutive children, finds the parent of the first one by binary search
// and walks forward, so a huge parent is spread over as many threads as it
// has children/16 and never serialises a wave.
// Expansions of more children than this write their tags with
// non-temporal stores (32 MB per tag array, the size of all L2s).
constexpr int64_t kTagsNtChildren = (int64_t)8 << 20;

__global__ __launch_bounds__(kBlock) void k_expand_tags(const int64_t *__restrict__ offsets, int64_t P,
                                                        uint32_t *__restrict__ child_parent,
                                                        uint32_t *__restrict__ child_ordinal,
                                                        int64_t child_cap, int vec_ok)
{
    constexpr int kWaveSpan = 64 * kItems;            // children per wave and step
    __shared__ alignas(16) uint32_t s_stage[kBlock / 64][kWaveSpan];
    const int64_t N = offsets[P];
    if (N > child_cap || N >= ((int64_t)1 << 32)) return;     // reported by the scan
    const int lane = lane_id();
    const bool nt = N > kTagsNtChildren;
    uint32_t *stage = s_stage[threadIdx.x >> 6];
    const int64_t nwaves = (int64_t)gridDim.x * (kBlock / 64);
    for (int64_t wt = (int64_t)blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6); wt * kWaveSpan < N; wt += nwaves) {
        // the wave's parent range by two wave-wide searches, then each lane's
        // first parent by a search inside that range
        const int64_t cb = wt * kWaveSpan;
        const int64_t ce = cb + kWaveSpan < N ? cb + kWaveSpan : N;
        const int64_t pf = wave_last_le(offsets, 0, P + 1, cb);
        const int64_t pl = wave_last_le(offsets, 0, P + 1, ce - 1);
        const int64_t c0 = cb + (int64_t)lane * kItems;
        int64_t p = c0 < N ? upper_bound_g(offsets, pf, pl + 1, c0) - 1 : pl;
        int64_t start = offsets[p];
        int64_t next = offsets[p + 1];
        uint32_t par[kItems], ord[kItems];
#pragma unroll
        for (int k = 0; k < kItems; ++k) {
            const int64_t c = c0 + k;
            if (c < N && c >= next) {
                p = advance_parent(offsets, P, p, c);
                start = offsets[p];
                next = offsets[p + 1];
            }
            par[k] = (uint32_t)p;
            ord[k] = (uint32_t)(c - start);
        }
        if (vec_ok && ce - cb == kWaveSpan) {
            // staged in LDS, then written 1 KiB per store instruction
#pragma unroll 1
            for (int which = 0; which < 2; ++which) {
                uint32_t *dst = which == 0 ? child_parent : child_ordinal;
                if (dst == nullptr) continue;
                const uint32_t *v = which == 0 ? par : ord;
#pragma unroll
                for (int k = 0; k < kItems / 4; ++k)
                    *reinterpret_cast<uint4 *>(&stage[lane * kItems + 4 * k]) =
                        make_uint4(v[4 * k], v[4 * k + 1], v[4 * k + 2], v[4 * k + 3]);
                __builtin_amdgcn_wave_barrier();
                if (nt) {
                    // non-temporal: an expansion this large is not read back
                    // soon, and its tags would only push other data out of L2
                    typedef uint32_t t4 __attribute__((ext_vector_type(4)));
                    t4 *out = reinterpret_cast<t4 *>(dst + cb);
#pragma unroll
                    for (int k = 0; k < kItems / 4; ++k)
                        __builtin_nontemporal_store(*reinterpret_cast<const t4 *>(&stage[(k * 64 + lane) * 4]),
                                                    out + k * 64 + lane);
                } else {
                    uint4 *out = reinterpret_cast<uint4 *>(dst + cb);
#pragma unroll
                    for (int k = 0; k < kItems / 4; ++k)
                        out[k * 64 + lane] = *reinterpret_cast<const uint4 *>(&stage[(k * 64 + lane) * 4]);
                }
                __builtin_amdgcn_wave_barrier();
            }
        } else {
#pragma unroll
            for (int k = 0; k < kItems; ++k) {
                if (c0 + k < N) {
                    if (child_parent) child_parent[c0 + k] = par[k];
                    if (child_ordinal) child_ordinal[c0 + k] = ord[k];
                }
            }
        }
    }
}

hipError_t launch_expand(const Launch &L, const int32_t *counts, int64_t P,
                         int64_t *offsets, uint32_t *child_parent, uint32_t *child_ordinal,
                         int64_t child_cap)
{
    const int64_t ntiles = P > 0 ? (P + kTile - 1) / kTile : 1;
    const int want = (child_parent != nullptr || child_ordinal != nullptr);
    const int64_t grid = ntiles < (int64_t)L.num_cus * 4 ? ntiles : (int64_t)L.num_cus * 4;
    RO_LAUNCH(L, RO_K_EXPAND_SCAN, k_expand_scan, dim3((unsigned)grid), dim3(kBlock), 0, L.stream, counts, P,
                       offsets, child_cap, want, L.ctl, L.desc, L.desc_cap, ntiles);
    if (want) {
        const bool aligned = ((reinterpret_cast<uintptr_t>(child_parent) |
                               reinterpret_cast<uintptr_t>(child_ordinal)) & 15u) == 0;
        const int64_t grid2 = (int64_t)L.num_cus * 8;
        RO_LAUNCH(L, RO_K_EXPAND_TAGS, k_expand_tags, dim3((unsigned)grid2), dim3(kBlock), 0, L.stream, offsets,
                           P, child_parent, child_ordinal, child_cap, aligned ? 1 : 0);
    }
    return hipGetLastError();
}

hipError_t launch_expand_tags(const Launch &L, const int64_t *offsets, int64_t P, uint32_t *child_parent,
                              uint32_t *child_ordinal, int64_t child_cap)
{
    const bool aligned = ((reinterpret_cast<uintptr_t>(child_parent) |
                           reinterpret_cast<uintptr_t>(child_ordinal)) & 15u) == 0;
    const int64_t grid2 = (int64_t)L.num_cus * 8;
    RO_LAUNCH(L, RO_K_EXPAND_TAGS, k_expand_tags, dim3((unsigned)grid2), dim3(kBlock), 0, L.stream, offsets, P,
              child_parent, child_ordinal, child_cap, aligned ? 1 : 0);
    return hipGetLastError();
}

}  // namespace ro
