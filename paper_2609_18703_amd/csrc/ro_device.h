// Device helpers: wave64 scans, decoupled look-back, searches, error word.
#pragma once

#include "ro_internal.h"

namespace ro {

__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & 63); }

__device__ __forceinline__ void raise_err(Ctl *ctl, int code)
{
    atomicCAS(&ctl->err, 0, code);
}

__device__ __forceinline__ int32_t read_err(Ctl *ctl)
{
    return __hip_atomic_load(&ctl->err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// A value every lane of the wave holds alike, moved to a scalar register
// (the compiler cannot see that results of shuffles or LDS reads are
// wave-uniform, and would keep them in vector registers).
__device__ __forceinline__ int32_t uni32(int32_t v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ int64_t uni64(int64_t v)
{
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int32_t)(uint32_t)v);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int32_t)(uint32_t)((uint64_t)v >> 32));
    return (int64_t)((uint64_t)hi << 32 | lo);
}

// ---- wave64 reductions / scans -------------------------------------------
template <typename T>
__device__ __forceinline__ T wave_incl_sum(T v)
{
    const int lane = lane_id();
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        T t = __shfl_up(v, d, 64);
        if (lane >= d) v += t;
    }
    return v;
}

template <typename T>
__device__ __forceinline__ T wave_sum(T v)
{
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) v += __shfl_xor(v, d, 64);
    return v;
}

// Exclusive scan over the kBlock threads of a workgroup.  `s_wave` holds
// kBlock/64 entries of LDS.  Every thread gets its exclusive prefix and the
// workgroup total.
__device__ __forceinline__ int64_t block_excl_scan(int64_t v, int64_t *s_wave, int64_t &total)
{
    const int lane = lane_id(), w = (int)(threadIdx.x >> 6);
    int64_t inc = wave_incl_sum(v);
    if (lane == 63) s_wave[w] = inc;
    __syncthreads();
    int64_t off = 0, tot = 0;
#pragma unroll
    for (int i = 0; i < kBlock / 64; ++i) {
        int64_t x = s_wave[i];
        off += (i < w) ? x : 0;
        tot += x;
    }
    __syncthreads();
    total = tot;
    return off + inc - v;
}

__device__ __forceinline__ int64_t block_sum(int64_t v, int64_t *s_wave)
{
    int64_t t;
    (void)block_excl_scan(v, s_wave, t);
    return t;
}

// ---- tile tickets ---------------------------------------------------------
// Tiles are handed out in increasing order from an atomic ticket, so a tile
// only ever waits on tiles already owned by running workgroups.  The last
// workgroup to finish resets the ticket for the next launch.
__device__ __forceinline__ int64_t next_ticket(Ctl *ctl, int64_t *s_t)
{
    if (threadIdx.x == 0)
        *s_t = (int64_t)__hip_atomic_fetch_add(&ctl->ticket, (uint64_t)1, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    int64_t t = *s_t;
    __syncthreads();
    return t;
}

// Epoch of this ticketed launch: every workgroup reads it at its start; the
// last workgroup to finish advances it, after all others are done with it.
__device__ __forceinline__ uint32_t scan_epoch(Ctl *ctl)
{
    return __hip_atomic_load(&ctl->scan_epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void desc_put_raw(uint64_t *d, uint64_t w)
{
    __hip_atomic_store(d, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Called once by every workgroup that takes part, after its last tile: the
// first `parts` workgroups of the grid (ticket_done: all of them; the others
// return without drawing a ticket).  The last one resets the ticket and
// advances the epoch; when the 16-bit epoch would wrap it first clears every
// descriptor, so an old descriptor can never carry the epoch of a later
// launch.
__device__ __forceinline__ void ticket_done_n(Ctl *ctl, uint32_t epoch, uint64_t *desc, int64_t desc_cap,
                                              int32_t *s_last, uint32_t parts)
{
    if (threadIdx.x == 0) {
        const uint32_t d = __hip_atomic_fetch_add(&ctl->done, 1u, __ATOMIC_RELAXED,
                                                  __HIP_MEMORY_SCOPE_AGENT);
        *s_last = (d == parts - 1) ? 1 : 0;
    }
    __syncthreads();
    if (*s_last) {
        const bool wrap = epoch + 1 > kMaxScanEpoch;
        if (wrap)
            for (int64_t i = threadIdx.x; i < desc_cap; i += blockDim.x) desc_put_raw(&desc[i], 0);
        __syncthreads();
        if (threadIdx.x == 0) {
            __hip_atomic_store(&ctl->ticket, (uint64_t)0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(&ctl->done, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(&ctl->scan_epoch, wrap ? 1u : epoch + 1, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

__device__ __forceinline__ void ticket_done(Ctl *ctl, uint32_t epoch, uint64_t *desc, int64_t desc_cap,
                                            int32_t *s_last)
{
    ticket_done_n(ctl, epoch, desc, desc_cap, s_last, gridDim.x);
}

// ---- decoupled look-back --------------------------------------------------
// Descriptor word: [63:48] launch epoch, [47:46] flag, [45:0] value.  The
// value saturates at kSat, so prefix sums never wrap; a saturated result is
// reported as an overflow by the caller.  Flag and value travel in one
// 64-bit word, so relaxed agent-scope atomics are enough on every XCD.
constexpr uint64_t kSat = 1ull << 45;
constexpr uint64_t kValMask = (1ull << 46) - 1;
constexpr uint32_t kFlagAgg = 1, kFlagInc = 2;

__device__ __forceinline__ uint64_t desc_word(uint32_t epoch, uint32_t flag, uint64_t v)
{
    return ((uint64_t)epoch << 48) | ((uint64_t)flag << 46) | (v & kValMask);
}

__device__ __forceinline__ void desc_put(uint64_t *d, uint64_t w)
{
    __hip_atomic_store(d, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Polls of one predecessor descriptor before the look-back gives up (about
// a second): a predecessor tile always belongs to a running workgroup, so
// this bound is only a guard that turns a protocol bug into an error
// instead of a hung device.
constexpr uint32_t kSpinLimit = 1u << 24;

// The look-back of tile t by one wave (all 64 lanes call it): posts the
// tile's aggregate, sums the predecessors' values back to the nearest
// inclusive one (64 descriptors a round), posts the tile's inclusive value
// and returns the exclusive prefix to every lane.
__device__ __forceinline__ uint64_t lookback_wave(uint64_t *desc, int64_t t, uint32_t epoch, uint64_t agg, Ctl *ctl)
{
    const int lane = lane_id();
    agg = agg < kSat ? agg : kSat;
    if (t == 0) {
        if (lane == 0) desc_put(&desc[0], desc_word(epoch, kFlagInc, agg));
        return 0;
    }
    if (lane == 0) desc_put(&desc[t], desc_word(epoch, kFlagAgg, agg));
    uint64_t excl = 0;
    int64_t base = t - 1;
    for (;;) {
        const int64_t j = base - lane;
        uint32_t flag = kFlagInc;
        uint64_t val = 0;
        if (j >= 0) {
            uint64_t d = 0;
            bool ready = false;
            for (uint32_t spin = 0; spin < kSpinLimit; ++spin) {
                d = __hip_atomic_load(&desc[j], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                if ((uint32_t)(d >> 48) == epoch && ((d >> 46) & 3u) != 0) {
                    ready = true;
                    break;
                }
                __builtin_amdgcn_s_sleep(1);
            }
            if (ready) {
                flag = (uint32_t)((d >> 46) & 3u);
                val = d & kValMask;
            } else {
                raise_err(ctl, RO_EHIP);     // treated as an inclusive zero
            }
        }
        const uint64_t incm = __ballot(flag == kFlagInc);
        const int first = incm ? (__ffsll((unsigned long long)incm) - 1) : 64;
        excl += wave_sum<uint64_t>(lane <= first ? val : 0);
        if (incm) break;
        base -= 64;
    }
    excl = excl < kSat ? excl : kSat;
    if (lane == 0) {
        const uint64_t inc = excl + agg;
        desc_put(&desc[t], desc_word(epoch, kFlagInc, inc < kSat ? inc : kSat));
    }
    return excl;
}

// Exclusive prefix of tile t given its aggregate; called by every thread of
// the workgroup, returns the same value to all of them.
__device__ __forceinline__ uint64_t tile_prefix_inl(uint64_t *desc, int64_t t, uint32_t epoch,
                                                   uint64_t agg, uint64_t *s_b, Ctl *ctl)
{
    if (threadIdx.x < 64) {
        const uint64_t r = lookback_wave(desc, t, epoch, agg, ctl);
        if (threadIdx.x == 0) *s_b = r;
    }
    __syncthreads();
    uint64_t r = *s_b;
    __syncthreads();
    return r;
}

// The same out of line, so that the look-back's registers do not add to the
// caller's (a call waits for every load the caller has in flight; the inline
// form above does not).
__device__ __noinline__ uint64_t tile_prefix(uint64_t *desc, int64_t t, uint32_t epoch,
                                             uint64_t agg, uint64_t *s_b, Ctl *ctl)
{
    return tile_prefix_inl(desc, t, epoch, agg, s_b, ctl);
}

// Two independent look-back chains of tile t at once, one wave each;
// s_b2 holds two entries of LDS.
__device__ __noinline__ void tile_prefix2(uint64_t *desc_a, uint64_t agg_a, uint64_t *desc_b, uint64_t agg_b,
                                          int64_t t, uint32_t epoch, uint64_t *s_b2, uint64_t &pa, uint64_t &pb,
                                          Ctl *ctl)
{
    const int w = (int)(threadIdx.x >> 6);
    if (w < 2) {
        const uint64_t r = w == 0 ? lookback_wave(desc_a, t, epoch, agg_a, ctl)
                                  : lookback_wave(desc_b, t, epoch, agg_b, ctl);
        if (lane_id() == 0) s_b2[w] = r;
    }
    __syncthreads();
    pa = s_b2[0];
    pb = s_b2[1];
    __syncthreads();
}

// ---- searches ---------------------------------------------------------------
// First index i in [lo, hi) with a[i] > x (hi if none).
__device__ __forceinline__ int64_t upper_bound_g(const int64_t *a, int64_t lo, int64_t hi, int64_t x)
{
    while (lo < hi) {
        int64_t mid = (lo + hi) >> 1;
        if (a[mid] <= x) lo = mid + 1; else hi = mid;
    }
    return lo;
}

// First index i in [lo, hi) with a[i] >= x (hi if none).
__device__ __forceinline__ int64_t lower_bound_g(const int64_t *a, int64_t lo, int64_t hi, int64_t x)
{
    while (lo < hi) {
        int64_t mid = (lo + hi) >> 1;
        if (a[mid] < x) lo = mid + 1; else hi = mid;
    }
    return lo;
}

// Parent of child c (largest p with offsets[p] <= c) when p is known to be
// >= p; walks a few steps, then falls back to a binary search so that long
// runs of empty parents cost a logarithm.
__device__ __forceinline__ int64_t advance_parent(const int64_t *offsets, int64_t P, int64_t p, int64_t c)
{
#pragma unroll 1
    for (int s = 0; s < 4; ++s) {
        if (offsets[p + 1] > c) return p;
        ++p;
    }
    return upper_bound_g(offsets, p, P + 1, c) - 1;
}

// Largest i in [lo, hi) with a[i] <= x, for nondecreasing a with a[lo] <= x.
// Called by all 64 lanes of a wave, which get the same result.  Each round
// the lanes probe 64 evenly spaced entries of the remaining range and a
// ballot keeps the gap holding the answer, so n entries take about
// log_65(n) rounds of one load each.
__device__ __forceinline__ int64_t wave_last_le(const int64_t *a, int64_t lo, int64_t hi, int64_t x)
{
    const int lane = lane_id();
    int64_t l = lo, h = hi;
    while (h - l > 1) {
        const int64_t idx = l + ((h - l) * (int64_t)(lane + 1)) / 65;
        const uint64_t m = __ballot(a[idx] <= x);
        const int k = __popcll(m);                 // the true probes form a prefix
        const int64_t nl = k > 0 ? __shfl(idx, k - 1, 64) : l;
        const int64_t nh = k < 64 ? __shfl(idx, k, 64) : h;
        l = nl;
        h = nh;
    }
    return l;
}

// Searches over tile-relative parent offsets held in LDS.
// Largest i in [lo, hi) with a[i] <= x, given a[lo] <= x.
__device__ __forceinline__ int lds_last_le(const int16_t *a, int lo, int hi, int x)
{
    while (hi - lo > 1) {
        const int m = (lo + hi) >> 1;
        if (a[m] <= x) lo = m; else hi = m;
    }
    return lo;
}

// First i in [lo, hi) with a[i] >= x (hi if none).
__device__ __forceinline__ int lds_first_ge(const int16_t *a, int lo, int hi, int x)
{
    while (lo < hi) {
        const int m = (lo + hi) >> 1;
        if (a[m] < x) lo = m + 1; else hi = m;
    }
    return lo;
}

// Group-failure commit rule (Sec. 4 "Commit, Failure, and Recovery"), for
// report i of parent p in a call whose first group failure per parent is
// recorded in gkey as (epoch << 32 | ~index): the report is rejected if p was
// barred before this call or if p's first group failure comes earlier in
// this call's report order.
__device__ __forceinline__ bool gf_rejected(const uint8_t *barrier, const uint64_t *gkey, uint32_t epoch,
                                            uint32_t p, int64_t i)
{
    if (barrier == nullptr) return false;
    if (barrier[p]) return true;
    const uint64_t k = gkey[p];
    if ((uint32_t)(k >> 32) != epoch) return false;
    return i > (int64_t)(0xffffffffu - (uint32_t)k);
}

__device__ __forceinline__ uint64_t gf_key(uint32_t epoch, int64_t i)
{
    return ((uint64_t)epoch << 32) | (uint64_t)(0xffffffffu - (uint32_t)i);
}

__device__ __forceinline__ int64_t min64(int64_t a, int64_t b) { return a < b ? a : b; }
__device__ __forceinline__ int64_t max64(int64_t a, int64_t b) { return a > b ? a : b; }

}  // namespace ro
