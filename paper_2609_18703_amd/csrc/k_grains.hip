// Grain phases and the generation fence on gfx950.
//
// RayOrch (arXiv 2609.18703), Sec. 4: a Grain goes WAITING -> READY ->
// IN-FLIGHT -> SEALED, and a retry takes IN-FLIGHT back to READY (Eq.
// grain-phase); a report commits only while its Grain is in flight at the
// report's generation (Eq. generation-fence); a repeat of a committed fact is
// idempotent and a conflicting one is rejected (publication rules).
//
// One 16-byte record per Grain: a word with the phase (READY or IN-FLIGHT)
// and the generation, and the fence key, so that each report or reservation
// touches one random line.  Reservation and retry change the word by one
// 64-bit compare-and-swap, so a child named twice in one call is caught.  A
// commit call is two passes over its reports.  The first records, per Grain,
// the first report (in report order) that passes the fence, as the largest
// key epoch << 32 | ~index, and tags every report that met another one of the
// call at the same Grain.  The second accepts the report the key names and
// classifies every other one as stale, duplicate or conflict; it reads a
// Grain's record only for tagged reports.  Every key the first pass sets
// belongs to a report the second accepts, so a Grain is SEALED exactly when
// its key is not zero, and the second pass writes nothing to the records.
// The bytes of a same-length repeat are compared by the whole wave.  Each
// thread takes kGItems reports (or children) per round, loads first, so that
// their random accesses overlap.
#include "ro_device.h"

namespace ro {

constexpr int kGItems = 4;

__device__ __forceinline__ uint32_t word_phase(uint64_t w) { return (uint32_t)w; }
__device__ __forceinline__ uint32_t word_gen(uint64_t w) { return (uint32_t)(w >> 32); }
__device__ __forceinline__ uint64_t make_word(uint32_t phase, uint32_t gen)
{
    return (uint64_t)phase | ((uint64_t)gen << 32);
}

__global__ void k_grains_fill(Grain *__restrict__ g, int64_t n)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        g[i].word = make_word(RO_READY, 0);
        g[i].key = 0;
    }
}

// Before commit epochs start again at 1: a sealed Grain keeps a key of epoch
// 0 (no call has it), an unsealed one keeps 0.
__global__ void k_grains_rekey(Grain *__restrict__ g, int64_t n)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        if (g[i].key != 0) g[i].key = 1;
}

// Phase and generation of every Grain, for inspection.
__global__ void k_grains_read(const Grain *__restrict__ g, int64_t n, uint32_t *__restrict__ phase,
                              uint32_t *__restrict__ gen)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        const Grain r = g[i];
        if (phase) phase[i] = r.key != 0 ? (uint32_t)RO_SEALED : word_phase(r.word);
        if (gen) gen[i] = word_gen(r.word);
    }
}

// READY -> IN-FLIGHT; the attempt's generation goes out.
__global__ __launch_bounds__(kBlock) void k_grains_dispatch(const uint32_t *__restrict__ child, int64_t n, int64_t N,
                                                            Grain *g, uint32_t *__restrict__ out_gen, Ctl *ctl)
{
    int err = 0;
    const int64_t span = (int64_t)kBlock * kGItems;
    for (int64_t base = (int64_t)blockIdx.x * span; base < n; base += (int64_t)gridDim.x * span) {
        uint32_t c[kGItems];
        Grain r[kGItems];
#pragma unroll
        for (int k = 0; k < kGItems; ++k) {
            const int64_t i = base + k * kBlock + threadIdx.x;
            c[k] = i < n ? child[i] : 0xffffffffu;
        }
#pragma unroll
        for (int k = 0; k < kGItems; ++k) r[k] = (int64_t)c[k] < N ? g[c[k]] : Grain{0, 0};
#pragma unroll
        for (int k = 0; k < kGItems; ++k) {
            const int64_t i = base + k * kBlock + threadIdx.x;
            if (i >= n) continue;
            if ((int64_t)c[k] >= N) { err = RO_ERANGE; continue; }
            const uint64_t w = r[k].word;
            if (r[k].key != 0 || word_phase(w) != RO_READY) { err = RO_ESTATE; continue; }
            const uint64_t nw = make_word(RO_IN_FLIGHT, word_gen(w));
            if (atomicCAS((unsigned long long *)&g[c[k]].word, (unsigned long long)w, (unsigned long long)nw) != w) {
                err = RO_ESTATE;                 // named twice in this call
                continue;
            }
            if (out_gen) out_gen[i] = word_gen(w);
        }
    }
    if (err) raise_err(ctl, err);
}

// IN-FLIGHT (not sealed) -> READY at the next generation.
__global__ __launch_bounds__(kBlock) void k_grains_retry(const uint32_t *__restrict__ child, int64_t n, int64_t N,
                                                         Grain *g, Ctl *ctl)
{
    int err = 0;
    const int64_t span = (int64_t)kBlock * kGItems;
    for (int64_t base = (int64_t)blockIdx.x * span; base < n; base += (int64_t)gridDim.x * span) {
        uint32_t c[kGItems];
        Grain r[kGItems];
#pragma unroll
        for (int k = 0; k < kGItems; ++k) {
            const int64_t i = base + k * kBlock + threadIdx.x;
            c[k] = i < n ? child[i] : 0xffffffffu;
        }
#pragma unroll
        for (int k = 0; k < kGItems; ++k) r[k] = (int64_t)c[k] < N ? g[c[k]] : Grain{0, 0};
#pragma unroll
        for (int k = 0; k < kGItems; ++k) {
            const int64_t i = base + k * kBlock + threadIdx.x;
            if (i >= n) continue;
            if ((int64_t)c[k] >= N) { err = RO_ERANGE; continue; }
            const uint64_t w = r[k].word;
            if (r[k].key != 0 || word_phase(w) != RO_IN_FLIGHT) { err = RO_ESTATE; continue; }
            const uint64_t nw = make_word(RO_READY, word_gen(w) + 1);
            if (atomicCAS((unsigned long long *)&g[c[k]].word, (unsigned long long)w, (unsigned long long)nw) != w)
                err = RO_ESTATE;
        }
    }
    if (err) raise_err(ctl, err);
}

// Pass 1: validation; the first report per Grain that passes the fence (the
// largest key); the provisional outcome of every report in state_out (its
// state if it passed the fence, RO_PENDING if not); and the reports that met
// another one of this call at the same Grain, tagged with the epoch in tag[]
// (the later of two tags itself and the one it found).
__global__ __launch_bounds__(kBlock) void k_grains_first(
    const uint32_t *__restrict__ rp, const uint32_t *__restrict__ ro_, const uint8_t *__restrict__ rs,
    const int64_t *__restrict__ roff, const uint32_t *__restrict__ rgen, int64_t n,
    const int64_t *__restrict__ offsets, int64_t P, int64_t N, Grain *g, uint32_t epoch, uint32_t *tag,
    uint8_t *__restrict__ state_out, int64_t *counts, Ctl *ctl)
{
    if (blockIdx.x == 0 && threadIdx.x < 4 && counts) counts[threadIdx.x] = 0;
    int err = 0;
    const int64_t span = (int64_t)kBlock * kGItems;
    for (int64_t base = (int64_t)blockIdx.x * span; base < n; base += (int64_t)gridDim.x * span) {
        int64_t c[kGItems];
        uint32_t gen[kGItems], s[kGItems];
        Grain r[kGItems];
#pragma unroll
        for (int k = 0; k < kGItems; ++k) {
            const int64_t i = base + k * kBlock + threadIdx.x;
            c[k] = -1;
            s[k] = RO_PENDING;
            if (i >= n) continue;
            const uint32_t st = rs[i];
            if (roff[i + 1] < roff[i]) { err = RO_EINVAL; continue; }
            if (st > RO_GROUP_FAILED) { err = RO_ESTATE; continue; }
            if (st == RO_PENDING) continue;
            const uint32_t p = rp[i];
            if ((int64_t)p >= P) { err = RO_ERANGE; continue; }
            const int64_t o = offsets[p];
            if ((int64_t)ro_[i] >= offsets[p + 1] - o) { err = RO_ERANGE; continue; }
            const int64_t ch = o + (int64_t)ro_[i];
            if (o < 0) { err = RO_EINVAL; continue; }      // offsets not an Expansion
            if (ch >= N) { err = RO_ERANGE; continue; }
            c[k] = ch;
            s[k] = st;
            gen[k] = rgen[i];
        }
#pragma unroll
        for (int k = 0; k < kGItems; ++k) r[k] = c[k] >= 0 ? g[c[k]] : Grain{0, 0};
#pragma unroll
        for (int k = 0; k < kGItems; ++k) {
            const int64_t i = base + k * kBlock + threadIdx.x;
            if (i >= n) continue;
            // unsealed before this call: no key, or one set in this pass
            const bool open = r[k].key == 0 || (uint32_t)(r[k].key >> 32) == epoch;
            const bool pass = c[k] >= 0 && open && word_phase(r[k].word) == RO_IN_FLIGHT &&
                              word_gen(r[k].word) == gen[k];
            state_out[i] = pass ? (uint8_t)s[k] : (uint8_t)RO_PENDING;
            if (pass) {
                const uint64_t old = __hip_atomic_fetch_max(&g[c[k]].key, gf_key(epoch, i), __ATOMIC_RELAXED,
                                                            __HIP_MEMORY_SCOPE_AGENT);
                if ((uint32_t)(old >> 32) == epoch) {
                    tag[i] = epoch;
                    tag[0xffffffffu - (uint32_t)old] = epoch;
                }
            }
        }
    }
    if (err) raise_err(ctl, err);
}

// Pass 2: an untagged report keeps its provisional outcome (accepted if it
// passed the fence, stale if not); among tagged ones, the report the key
// names is accepted and every other one repeats it: a duplicate if state and
// bytes are the same, a conflict otherwise.  The wave compares the bytes of
// its lanes' same-length repeats one repeat at a time, 16 bytes a lane.
__global__ __launch_bounds__(kBlock) void k_grains_decide(
    const uint32_t *__restrict__ rp, const uint32_t *__restrict__ ro_, const uint8_t *__restrict__ rs,
    const int64_t *__restrict__ roff, const uint8_t *__restrict__ data, int64_t n,
    const int64_t *__restrict__ offsets, const Grain *__restrict__ g, uint32_t epoch,
    const uint32_t *__restrict__ tag, uint8_t *__restrict__ state_out, int64_t *counts, Ctl *ctl)
{
    __shared__ int64_t s_wave[kBlock / 64];
    if (read_err(ctl) != 0) return;                  // the first pass found a bad report
    const int lane = lane_id();
    int64_t cnt[4] = {0, 0, 0, 0};                   // accepted, stale, duplicate, conflict
    const int64_t span = (int64_t)kBlock * kGItems;
    for (int64_t base = (int64_t)blockIdx.x * span; base < n; base += (int64_t)gridDim.x * span) {
#pragma unroll
        for (int k = 0; k < kGItems; ++k) {
            const int64_t i = base + k * kBlock + threadIdx.x;
            int kind = -1;
            int64_t a = 0, b = 0, len = 0;           // a same-length repeat to compare
            if (i < n && rs[i] != RO_PENDING) {
                const uint32_t s = rs[i];
                if (tag[i] != epoch) {
                    kind = state_out[i] == RO_PENDING ? 1 : 0;
                } else {
                    const uint64_t key = g[offsets[rp[i]] + (int64_t)ro_[i]].key;
                    if (key == gf_key(epoch, i)) {
                        kind = 0;
                    } else {
                        const int64_t v = (int64_t)(0xffffffffu - (uint32_t)key);
                        bool same = rs[v] == s;
                        if (same && s == RO_SUCCESS) {
                            const int64_t lv = roff[v + 1] - roff[v];
                            same = lv == roff[i + 1] - roff[i];
                            if (same && data != nullptr && lv > 0) {
                                a = roff[v];
                                b = roff[i];
                                len = lv;
                            }
                        }
                        kind = same ? 2 : 3;
                        state_out[i] = RO_PENDING;
                    }
                }
            }
            uint64_t jobs = __ballot(len > 0);
            while (jobs) {
                const int l = __ffsll((unsigned long long)jobs) - 1;
                jobs &= jobs - 1;
                const int64_t pa = __shfl((long long)a, l), pb = __shfl((long long)b, l);
                const int64_t pl = __shfl((long long)len, l);
                uint32_t diff = 0;
                for (int64_t o = (int64_t)lane * 16; o < pl; o += 64 * 16) {
#pragma unroll
                    for (int q = 0; q < 16; ++q)
                        if (o + q < pl) diff |= (uint32_t)(data[pa + o + q] ^ data[pb + o + q]);
                }
                if (__ballot(diff != 0) != 0 && lane == l) kind = 3;
            }
            if (kind >= 0) ++cnt[kind];
        }
    }
    if (counts) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t t = block_sum(cnt[j], s_wave);
            if (threadIdx.x == 0 && t)
                __hip_atomic_fetch_add(&counts[j], t, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

__global__ void k_grains_zero_tags(uint32_t *__restrict__ tag, int64_t n)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        tag[i] = 0;
}

static int64_t grid_for(const Launch &L, int64_t n, int64_t per_block)
{
    int64_t grid = (n + per_block - 1) / per_block;
    return grid < 1 ? 1 : (grid > (int64_t)L.num_cus * 8 ? (int64_t)L.num_cus * 8 : grid);
}

hipError_t launch_grains_fill(const Launch &L, Grain *g, int64_t n)
{
    RO_LAUNCH(L, RO_K_GRAINS, k_grains_fill, dim3((unsigned)grid_for(L, n, kBlock)), dim3(kBlock), 0, L.stream, g,
              n);
    return hipGetLastError();
}

hipError_t launch_grains_rekey(const Launch &L, Grain *g, int64_t n)
{
    RO_LAUNCH(L, RO_K_GRAINS, k_grains_rekey, dim3((unsigned)grid_for(L, n, kBlock)), dim3(kBlock), 0, L.stream, g,
              n);
    return hipGetLastError();
}

hipError_t launch_grains_read(const Launch &L, const Grain *g, int64_t n, uint32_t *phase, uint32_t *gen)
{
    RO_LAUNCH(L, RO_K_GRAINS, k_grains_read, dim3((unsigned)grid_for(L, n, kBlock)), dim3(kBlock), 0, L.stream, g, n,
              phase, gen);
    return hipGetLastError();
}

hipError_t launch_grains_dispatch(const Launch &L, const uint32_t *child, int64_t n, int64_t N, Grain *g,
                                  uint32_t *out_gen)
{
    RO_LAUNCH(L, RO_K_GRAINS, k_grains_dispatch, dim3((unsigned)grid_for(L, n, kBlock * kGItems)), dim3(kBlock), 0,
              L.stream, child, n, N, g, out_gen, L.ctl);
    return hipGetLastError();
}

hipError_t launch_grains_retry(const Launch &L, const uint32_t *child, int64_t n, int64_t N, Grain *g)
{
    RO_LAUNCH(L, RO_K_GRAINS, k_grains_retry, dim3((unsigned)grid_for(L, n, kBlock * kGItems)), dim3(kBlock), 0,
              L.stream, child, n, N, g, L.ctl);
    return hipGetLastError();
}

hipError_t launch_grains_zero_tags(const Launch &L, uint32_t *tag, int64_t n)
{
    RO_LAUNCH(L, RO_K_GRAINS, k_grains_zero_tags, dim3((unsigned)grid_for(L, n, kBlock)), dim3(kBlock), 0, L.stream,
              tag, n);
    return hipGetLastError();
}

hipError_t launch_grains_commit(const Launch &L, const uint32_t *rp, const uint32_t *ro, const uint8_t *rs,
                                const int64_t *roff, const uint8_t *data, const uint32_t *rgen, int64_t n,
                                const int64_t *offsets, int64_t P, int64_t N, Grain *g, uint32_t epoch, uint32_t *tag,
                                uint8_t *state_out, int64_t *counts)
{
    const int64_t grid = grid_for(L, n, kBlock * kGItems);
    RO_LAUNCH(L, RO_K_FENCE_FIRST, k_grains_first, dim3((unsigned)grid), dim3(kBlock), 0, L.stream, rp, ro, rs, roff,
              rgen, n, offsets, P, N, g, epoch, tag, state_out, counts, L.ctl);
    RO_LAUNCH(L, RO_K_FENCE_DECIDE, k_grains_decide, dim3((unsigned)grid), dim3(kBlock), 0, L.stream, rp, ro, rs,
              roff, data, n, offsets, g, epoch, tag, state_out, counts, L.ctl);
    return hipGetLastError();
}

}  // namespace ro
