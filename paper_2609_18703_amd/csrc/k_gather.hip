// F.reduce on gfx950: ordered gather of variable-length child reports into
// parent slots, with per-parent counts and completion.
//
// RayOrch (arXiv 2609.18703), Sec. 4, Reduce rule: a parent resolves once its
// Expansion and every member outcome are terminal; dropped members are left
// out, failed members suppress the parent, present values appear in immutable
// ordinal order, and zero survivors give an empty list.  The publication
// rules of the same section reject a second, conflicting report.
//
// Four kernels:
//   scatter  : report i -> canonical slot c = offsets[p] + o (validation, one
//              16-byte store per report; the only random-access pass).
//   scan     : canonical order, decoupled look-back over the surviving byte
//              lengths -> every parent's slot offset, per-parent counts (LDS
//              aggregated), per-sub-tile output bases.
//   finalize : per parent: complete / state, trailing slot offsets, duplicate
//              and capacity checks.
//   copy     : the output is cut into byte ranges of equal size; per range,
//              a wave rebuilds the destination offsets of the canonical
//              sub-tiles it overlaps and writes the range as aligned 16-byte
//              stores; sources are byte-aligned records read as aligned
//              16-byte pairs and realigned in registers.
#include "ro_copy.h"

namespace ro {

// ---------------------------------------------------------------- group failure
__global__ void k_first_gf(const uint8_t *__restrict__ rs, const uint32_t *__restrict__ rp, int64_t n,
                           int64_t P, const uint8_t *__restrict__ barrier, uint64_t *__restrict__ gkey,
                           uint32_t epoch)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        if (rs[i] != RO_GROUP_FAILED) continue;
        const uint32_t p = rp[i];
        if ((int64_t)p >= P || barrier[p]) continue;
        __hip_atomic_fetch_max(&gkey[p], gf_key(epoch, i), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

__global__ void k_gf_fold(const uint8_t *__restrict__ rs, const uint32_t *__restrict__ rp, int64_t n, int64_t P,
                          uint8_t *__restrict__ barrier, const uint64_t *__restrict__ gkey, uint32_t epoch)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        if (rs[i] != RO_GROUP_FAILED) continue;
        const uint32_t p = rp[i];
        if ((int64_t)p < P && gkey[p] == gf_key(epoch, i)) barrier[p] = 1;
    }
}

hipError_t launch_first_gf(const Launch &L, const uint8_t *rs, const uint32_t *rp, int64_t n, int64_t P,
                           const uint8_t *barrier, uint64_t *gkey, uint32_t epoch)
{
    int64_t grid = (n + kBlock - 1) / kBlock;
    grid = grid < 1 ? 1 : (grid > (int64_t)L.num_cus * 8 ? (int64_t)L.num_cus * 8 : grid);
    RO_LAUNCH(L, RO_K_GATHER_SCATTER, k_first_gf, dim3((unsigned)grid), dim3(kBlock), 0, L.stream, rs, rp, n, P,
              barrier, gkey, epoch);
    return hipGetLastError();
}

hipError_t launch_gf_fold(const Launch &L, const uint8_t *rs, const uint32_t *rp, int64_t n, int64_t P,
                          uint8_t *barrier, const uint64_t *gkey, uint32_t epoch)
{
    int64_t grid = (n + kBlock - 1) / kBlock;
    grid = grid < 1 ? 1 : (grid > (int64_t)L.num_cus * 8 ? (int64_t)L.num_cus * 8 : grid);
    RO_LAUNCH(L, RO_K_STREAM_REPORT, k_gf_fold, dim3((unsigned)grid), dim3(kBlock), 0, L.stream, rs, rp, n, P,
              barrier, gkey, epoch);
    return hipGetLastError();
}

// ---------------------------------------------------------------- scatter
#ifndef RO_SCATTER_ITEMS
#define RO_SCATTER_ITEMS 2
#endif
constexpr int kScatterItems = RO_SCATTER_ITEMS;   // reports per thread and step
// With a group-failure barrier, reports commit in report order: one of a
// barred parent, or one after its parent's first group failure in this
// call, is rejected; an accepted group failure is a failed member.
__global__ __launch_bounds__(kBlock) void k_gather_scatter(
    const uint32_t *__restrict__ rp, const uint32_t *__restrict__ ro_, const uint8_t *__restrict__ rs,
    const int64_t *__restrict__ roff, const uint8_t *data, int64_t n,
    const int64_t *__restrict__ offsets, int64_t P, Canon *__restrict__ canon, int64_t canon_cap,
    int32_t *__restrict__ ns, int32_t *__restrict__ nf, int32_t *__restrict__ nk,
    const uint8_t *__restrict__ barrier, const uint64_t *__restrict__ gkey, uint32_t epoch, Ctl *ctl)
{
    __shared__ int64_t s_wave[kBlock / 64];
    const int64_t N = offsets[P];
    const bool cap_ok = N <= canon_cap;
    const int64_t gtid = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    const int64_t gstride = (int64_t)gridDim.x * kBlock;
    if (gtid == 0) {
        if (!cap_ok) raise_err(ctl, RO_ECAP);
        if (n > 0 && roff[0] < 0) raise_err(ctl, RO_EINVAL);
    }
    int err = 0;
    // the Expansion must be an exclusive scan: offsets[0] = 0, nondecreasing
    if (gtid == 0 && offsets[0] != 0) err = RO_EINVAL;
    for (int64_t p = gtid; p < P; p += gstride) {
        if (ns) ns[p] = 0;
        if (nf) nf[p] = 0;
        if (nk) nk[p] = 0;
        if (offsets[p + 1] < offsets[p]) err = RO_EINVAL;
    }
    int64_t cnt = 0, rej = 0;
    constexpr int U = kScatterItems;
    // U reports per thread and step, their loads and lookups all in flight
    // before any is validated or stored
    for (int64_t b = gtid; b < n; b += U * gstride) {
        uint32_t sv[U], pv[U], ov[U];
        int64_t o0v[U], o1v[U], stv[U], env[U];
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const int64_t i = b + k * gstride;
            const bool in = i < n;
            // the report columns are read once: non-temporal loads leave L2
            // to the slots being written (workload 2's scatter 1.53 -> 1.45 ms)
            sv[k] = in ? __builtin_nontemporal_load(rs + i) : RO_PENDING;
            pv[k] = in ? __builtin_nontemporal_load(rp + i) : 0xffffffffu;
            ov[k] = in ? __builtin_nontemporal_load(ro_ + i) : 0u;
            o0v[k] = in ? __builtin_nontemporal_load(roff + i) : 0;
            o1v[k] = in ? __builtin_nontemporal_load(roff + i + 1) : 0;
        }
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const bool ok = (int64_t)pv[k] < P;
            stv[k] = ok ? offsets[pv[k]] : 0;
            env[k] = ok ? offsets[pv[k] + 1] : 0;
        }
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const int64_t i = b + k * gstride;
            if (i >= n) continue;
            uint32_t s = sv[k];
            const int64_t o0 = o0v[k], o1 = o1v[k];
            if (o1 < o0) { err = RO_EINVAL; continue; }
            if (s > RO_PENDING && !(s == RO_GROUP_FAILED && barrier)) { err = RO_ESTATE; continue; }
            if (s == RO_PENDING) continue;
            const uint32_t p = pv[k];
            if ((int64_t)p >= P) { err = RO_ERANGE; continue; }
            const int64_t st = stv[k];
            const uint32_t o = ov[k];
            if ((int64_t)o >= env[k] - st) { err = RO_ERANGE; continue; }
            const int64_t c = st + (int64_t)o;
            if (st < 0 || c >= N) { err = RO_EINVAL; continue; }
            const int64_t len = s == RO_SUCCESS ? o1 - o0 : 0;
            if (len >= ((int64_t)1 << 32)) { err = RO_EOVERFLOW; continue; }
            if (gf_rejected(barrier, gkey, epoch, p, i)) { ++rej; continue; }
            if (s == RO_GROUP_FAILED) s = RO_FAILED;
            ++cnt;
            if (cap_ok) {
                Canon e;
                e.src = reinterpret_cast<uint64_t>(data) + (uint64_t)o0;
                e.len = (uint32_t)len;
                e.tag = (epoch << 2) | s;
                canon[c] = e;
            }
        }
    }
    if (err) raise_err(ctl, err);
    const int64_t tot = block_sum(cnt, s_wave);
    if (threadIdx.x == 0 && tot)
        __hip_atomic_fetch_add(&ctl->n_valid, tot, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (barrier) {
        const int64_t r = block_sum(rej, s_wave);
        if (threadIdx.x == 0 && r)
            __hip_atomic_fetch_add(&ctl->n_rejected, r, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// ---------------------------------------------------------------- scan
#ifndef RO_SCAN_WG
#define RO_SCAN_WG 3                        // workgroups per CU
#endif
// One tile = 4096 canonical children, 16 consecutive per thread; every 16
// threads cover one copy sub-tile of 256 children and record its first output
// byte.  A workgroup holds one tile at a time, but as soon as the tile's
// look-back is done it draws the next ticket, finds the next tile's parents
// and issues the loads of its slots, which are then in flight while the
// current tile's pass 2 runs.  The current tile has posted its prefix before
// the workgroup waits on anything for the next one, so the smallest tile not
// yet posted always belongs to a workgroup that can post it.
//
// In place (the output is the report bytes themselves, as for an upper level
// whose slots are the level below's output): nothing is copied, and the scan
// checks that every surviving record already sits at its output position;
// any other would overwrite bytes still to be read (RO_EINVAL).
template <bool kInPlace>
__global__ __launch_bounds__(kBlock) void k_gather_scan(
    const int64_t *__restrict__ offsets, int64_t P, const Canon *__restrict__ canon, int64_t canon_cap,
    int64_t *__restrict__ out_off, int32_t *__restrict__ ns, int32_t *__restrict__ nf,
    int32_t *__restrict__ nk, int64_t *__restrict__ cdst, int64_t *__restrict__ sub_base, const uint8_t *out,
    uint32_t epoch, Ctl *ctl, uint64_t *desc, int64_t desc_cap)
{
    const uint32_t sepoch = scan_epoch(ctl);
    __shared__ int64_t s_wave[kBlock / 64];
    __shared__ uint64_t s_b;
    __shared__ int64_t s_t;
    __shared__ int32_t s_last;
    __shared__ int64_t s_p[2][3];
    __shared__ int32_t s_cnt[3][kCntLds];
    __shared__ int16_t s_off[2][kTile + 2];     // offsets[pf..pl+1] - ct0, clamped to [-1, kTile + 1]
    __shared__ uint32_t s_len[kTile + kTile / 16];
    __shared__ alignas(16) uint8_t s_st[kTile];
    const int64_t N0 = offsets[P];
    // over capacity, or an invalid Expansion found by the scatter: no tiles
    const int64_t N = (N0 <= canon_cap && read_err(ctl) == 0) ? N0 : 0;
    const int64_t ntiles = (N + kTile - 1) / kTile;
    int32_t *cnt_out[3] = {ns, nf, nk};
    int64_t filled_total = 0;
    const int wv = (int)(threadIdx.x >> 6), ln = lane_id();

    // Tile tt's parents, one wave-parallel search each: pf holds child a0,
    // pl holds child a1 - 1, q0 is the first parent starting at or after a0
    // (empty parents before pf may start exactly at a0).  With few enough
    // parents, a tile-relative copy of their offsets goes to s_off[b] for
    // pass 2 to search instead of global memory.
    auto prepare = [&](int64_t tt, int b) {
        const int64_t a0 = tt * kTile;
        const int64_t a1 = min64(a0 + kTile, N);
        if (threadIdx.x < 3 * 64) {
            int64_t r;
            if (wv == 0) r = wave_last_le(offsets, 0, P + 1, a0);
            else if (wv == 1) r = wave_last_le(offsets, 0, P + 1, a1 - 1);
            else r = a0 == 0 ? 0 : wave_last_le(offsets, 0, P + 1, a0 - 1) + 1;
            if (ln == 0) s_p[b][wv] = r;
        }
        __syncthreads();
        const int64_t pf = s_p[b][0];
        const int64_t Rp = s_p[b][1] - pf + 1;
        if (Rp <= kTile) {
            for (int64_t j = threadIdx.x; j <= Rp; j += kBlock) {
                const int64_t v = offsets[pf + j] - a0;
                s_off[b][j] = (int16_t)(v < -1 ? -1 : (v > kTile + 1 ? kTile + 1 : v));
            }
        }
    };
    // The length and tag words (8 of every 16 bytes) of tile tt's slots, each
    // wave lane-contiguously over its 1024, into ev: the loads are only
    // issued here.  A slot past the expansion re-reads the tile's first one
    // and is ignored.
    uint2 ev[kItems];
    auto load_slots = [&](int64_t tt) {
        const int64_t a0 = uni64(tt * kTile);
        const int nloc = (int)uni64(min64(a0 + kTile, N) - a0);
        // uniform base and 32-bit unsigned lane offsets: scalar-base loads
        const uint8_t *tb = reinterpret_cast<const uint8_t *>(canon + a0) + offsetof(Canon, len);
        const uint32_t jb = (uint32_t)(wv * (64 * kItems) + ln);
        if (nloc == kTile) {
#pragma unroll
            for (int k = 0; k < kItems; ++k)
                ev[k] = *reinterpret_cast<const uint2 *>(tb + (jb + 64u * k) * (uint32_t)sizeof(Canon));
        } else {
#pragma unroll
            for (int k = 0; k < kItems; ++k) {
                const uint32_t j = jb + 64u * k;
                ev[k] = *reinterpret_cast<const uint2 *>(tb + (j < (uint32_t)nloc ? j : 0u) *
                                                                  (uint32_t)sizeof(Canon));
            }
        }
    };

    for (int j = threadIdx.x; j < 3 * kCntLds; j += kBlock) (&s_cnt[0][0])[j] = 0;
    // a workgroup that sees no tiles draws no ticket, so every drawn ticket
    // is processed even if workgroups disagree about an error raised meanwhile
    int64_t t = ntiles > 0 ? next_ticket(ctl, &s_t) : ntiles;
    int buf = 0;
    if (t < ntiles) {
        prepare(t, 0);
        load_slots(t);
    }
    while (t < ntiles) {
        __syncthreads();                    // s_p / s_off of this tile, cleared counts
        const int64_t ct0 = t * kTile;
        const int64_t ct1 = min64(ct0 + kTile, N);
        const int64_t pf = s_p[buf][0], pl = s_p[buf][1], q0t = s_p[buf][2];
        const int64_t Rp = pl - pf + 1;
        const int64_t R = min64(Rp, kCntLds);
        const bool lds_ok = Rp <= kTile;
        const int16_t *so = s_off[buf];

        // pass 1: surviving lengths and filled slots into LDS; then every
        // thread takes its 16 consecutive children from there.  s_len is
        // padded by one word per 16 so that both access patterns are free of
        // bank conflicts.
        {
            const int nloc = (int)(ct1 - ct0);
            const int jb = wv * (64 * kItems) + ln;
            const int lb = jb + (jb >> 4);          // s_len index of child jb + 64 k is lb + 68 k
#pragma unroll
            for (int k = 0; k < kItems; ++k) {
                uint32_t L = 0, S = 4;        // state, or 4 = not reported in this call
                if (jb + k * 64 < nloc && (ev[k].y >> 2) == epoch) {
                    S = ev[k].y & 3u;
                    L = S == RO_SUCCESS ? ev[k].x : 0;
                }
                s_len[lb + 68 * k] = L;
                s_st[jb + 64 * k] = (uint8_t)S;
            }
        }
        __syncthreads();
        const int64_t c0 = ct0 + (int64_t)threadIdx.x * kItems;
        const int lj = (int)threadIdx.x * kItems + (int)threadIdx.x;      // s_len index of c0
        uint32_t sw[4];                     // the thread's 16 state bytes, four per word
        int64_t sum = 0, filled = 0;
        {
            const uint4 sv = *reinterpret_cast<const uint4 *>(&s_st[threadIdx.x * kItems]);
            sw[0] = sv.x;
            sw[1] = sv.y;
            sw[2] = sv.z;
            sw[3] = sv.w;
#pragma unroll
            for (int k = 0; k < kItems; ++k) {
                sum += s_len[lj + k];
                filled += ((sw[k >> 2] >> (8 * (k & 3))) & 0xffu) < 4 ? 1 : 0;
            }
        }
        filled_total += filled;
        int64_t tot;
        const int64_t ex = block_excl_scan(sum, s_wave, tot);
        const uint64_t pre = tile_prefix_inl(desc, t, sepoch, (uint64_t)tot, &s_b, ctl);
        const int64_t base = (int64_t)pre + ex;
        if ((threadIdx.x % (kSub / kItems)) == 0) {
            const int64_t sb = t * (kTile / kSub) + threadIdx.x / (kSub / kItems);
            sub_base[sb] = base;                    // first byte of each copy sub-tile
        }
        if (t == ntiles - 1 && threadIdx.x == 0) {
            ctl->total = (int64_t)pre + tot;
            if (pre >= kSat) raise_err(ctl, RO_EOVERFLOW);
        }

        // the next tile: ticket, parents, and its slot loads in flight
        const int64_t t_next = next_ticket(ctl, &s_t);
        if (t_next < ntiles) {
            prepare(t_next, buf ^ 1);
            load_slots(t_next);
        }

        // pass 2: parents -- slot offsets and run-length counts
        if (c0 < ct1) {
            uint64_t srcv[kInPlace ? kItems : 1];
            bool moved = false;
            if constexpr (kInPlace) {
#pragma unroll
                for (int k = 0; k < kItems; ++k) srcv[k] = canon[min64(c0 + k, ct1 - 1)].src;
            }
            const uint64_t outa = reinterpret_cast<uint64_t>(out);
            int32_t run[3] = {0, 0, 0};
            auto flush = [&](int64_t p) {
#pragma unroll
                for (int s = 0; s < 3; ++s) {
                    if (run[s]) {
                        if (p - pf < R) atomicAdd(&s_cnt[s][p - pf], run[s]);
                        else if (cnt_out[s]) atomicAdd(&cnt_out[s][p], run[s]);
                        run[s] = 0;
                    }
                }
            };
            int64_t pos = base;
            if (lds_ok) {
                const int r0 = (int)(c0 - ct0), rend = (int)(ct1 - ct0);
                int j = lds_last_le(so, 0, (int)Rp, r0);
                if (so[j] == r0 && out_off) {
                    // every parent whose first child is c0 (empty ones included)
                    const int64_t qa = r0 == 0 ? q0t : pf + lds_first_ge(so, 1, j + 1, r0);
                    for (int64_t q = qa; q <= pf + j; ++q) out_off[q] = pos;
                }
                int next = so[j + 1];
                for (int k = 0; k < kItems; ++k) {
                    const int rc = r0 + k;
                    if (rc >= rend) break;
                    if (rc >= next) {
                        flush(pf + j);
                        const int jn = lds_last_le(so, j + 1, (int)Rp, rc);
                        if (out_off)
                            for (int64_t q = pf + j + 1; q <= pf + jn; ++q) out_off[q] = pos;
                        j = jn;
                        next = so[j + 1];
                    }
                    const uint32_t sk = (sw[k >> 2] >> (8 * (k & 3))) & 0xffu;
                    if (sk < 3) run[sk] += 1;
                    if (cdst) cdst[c0 + k] = pos;
                    if constexpr (kInPlace) moved |= s_len[lj + k] != 0 && srcv[k] != outa + (uint64_t)pos;
                    pos += s_len[lj + k];
                }
                flush(pf + j);
            } else {
                int64_t p = upper_bound_g(offsets, pf, pl + 1, c0) - 1;
                if (offsets[p] == c0) {
                    const int64_t q0 = c0 == ct0 ? q0t : lower_bound_g(offsets, pf, p + 1, c0);
                    if (out_off)
                        for (int64_t q = q0; q <= p; ++q) out_off[q] = pos;
                }
                int64_t next = offsets[p + 1];
                for (int k = 0; k < kItems; ++k) {
                    const int64_t c = c0 + k;
                    if (c >= ct1) break;
                    if (c >= next) {
                        flush(p);
                        const int64_t pn = advance_parent(offsets, P, p, c);
                        if (out_off)
                            for (int64_t q = p + 1; q <= pn; ++q) out_off[q] = pos;
                        p = pn;
                        next = offsets[p + 1];
                    }
                    const uint32_t sk = (sw[k >> 2] >> (8 * (k & 3))) & 0xffu;
                    if (sk < 3) run[sk] += 1;
                    if (cdst) cdst[c] = pos;
                    if constexpr (kInPlace) moved |= s_len[lj + k] != 0 && srcv[k] != outa + (uint64_t)pos;
                    pos += s_len[lj + k];
                }
                flush(p);
            }
            if (moved) raise_err(ctl, RO_EINVAL);
        }
        __syncthreads();
        for (int64_t j = threadIdx.x; j < R; j += kBlock) {
#pragma unroll
            for (int s = 0; s < 3; ++s) {
                const int32_t v = s_cnt[s][j];
                if (v && cnt_out[s]) atomicAdd(&cnt_out[s][pf + j], v);
            }
        }
        __syncthreads();
        for (int j = threadIdx.x; j < 3 * kCntLds; j += kBlock) (&s_cnt[0][0])[j] = 0;
        t = t_next;
        buf ^= 1;
    }
    const int64_t f = block_sum(filled_total, s_wave);
    if (threadIdx.x == 0 && f)
        __hip_atomic_fetch_add(&ctl->n_filled, f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    ticket_done(ctl, sepoch, desc, desc_cap, &s_last);
}

// ---------------------------------------------------------------- finalize
__global__ __launch_bounds__(kBlock) void k_gather_finalize(
    const int64_t *__restrict__ offsets, int64_t P, int64_t canon_cap, int64_t *__restrict__ out_off,
    int64_t out_cap, int has_data, const int32_t *__restrict__ ns, const int32_t *__restrict__ nf,
    const int32_t *__restrict__ nk, uint8_t *__restrict__ complete, uint8_t *__restrict__ pstate,
    int64_t *__restrict__ cdst, uint8_t *__restrict__ barrier, const uint64_t *__restrict__ gkey,
    int64_t *n_rejected, uint32_t epoch, Ctl *ctl)
{
    const int64_t N0 = offsets[P];
    const int64_t N = N0 <= canon_cap ? N0 : 0;
    const int64_t total = N > 0 ? ctl->total : 0;
    const int64_t gtid = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (gtid == 0) {
        if (out_off) out_off[P] = total;
        if (cdst && N0 <= canon_cap) cdst[N0] = total;
        if (n_rejected) *n_rejected = ctl->n_rejected;
        if (ctl->n_filled != ctl->n_valid) raise_err(ctl, RO_EDUP);
        if (has_data && total > out_cap) raise_err(ctl, RO_ECAP);
        // the call's counters are read only here: cleared for the next
        // gather (the byte total is rewritten by every scan with children)
        ctl->n_valid = 0;
        ctl->n_filled = 0;
        ctl->n_rejected = 0;
    }
    for (int64_t p = gtid; p < P; p += (int64_t)gridDim.x * kBlock) {
        const int64_t st = offsets[p];
        const int64_t k = offsets[p + 1] - st;
        if (st >= N && out_off) out_off[p] = total;       // no child at or after its start
        const int64_t a = ns ? ns[p] : 0, b = nf ? nf[p] : 0, c = nk ? nk[p] : 0;
        // a barred parent's uncommitted children are suppressed: it is done
        bool barred = false;
        if (barrier) {
            barred = barrier[p] || (uint32_t)(gkey[p] >> 32) == epoch;
            if (barred) barrier[p] = 1;
        }
        const bool done = barred || (a + b + c) == k;
        if (complete) complete[p] = done ? 1 : 0;
        if (pstate) pstate[p] = !done ? RO_PENDING : ((barred || b > 0) ? RO_FAILED : RO_SUCCESS);
    }
}

// finalize needs all three counters even if the caller wants none of them;
// the runtime passes workspace arrays in that case.

// ---------------------------------------------------------------- copy
// First sub-tile whose output holds byte `lo`: the largest s in [0, nsub)
// with sub_base[s] <= lo (sub_base[0] = 0).
__device__ __forceinline__ int64_t find_sub_tile(const int64_t *__restrict__ sub_base, int64_t nsub, int64_t lo)
{
    return wave_last_le(sub_base, 0, nsub, lo);
}

// Each wave works alone on its units of output bytes, with no workgroup
// barrier.  For each sub-tile of kSub canonical children that a unit touches,
// it rebuilds the destination offsets with a wave scan, clips every record to
// the unit's byte range (shifting the source start of a record that begins
// before it), and writes that range with aligned 16-byte stores.  Byte-sized
// units keep the chip busy whether the records are a few bytes or megabytes
// long, and few parents or many.
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(RO_COPY_WAVES))) void k_gather_copy(
    const int64_t *__restrict__ offsets, int64_t P, const Canon *__restrict__ canon, int64_t canon_cap,
    const int64_t *__restrict__ sub_base, uint8_t *__restrict__ out, uint32_t epoch, Ctl *ctl)
{
    constexpr int kWaves = kBlock / 64;
    __shared__ int32_t s_dst_all[kWaves][kSub + 1];     // clipped destination offset of each record
    __shared__ uint64_t s_src_all[kWaves][kSub];        // source address of its first clipped byte
    __shared__ int32_t s_edge_all[kWaves][kEdgeCap];    // edge chunks of the window
    __shared__ int16_t s_edger_all[kWaves][kEdgeCap];   // the record holding each one's first byte
    if (read_err(ctl) != 0) return;                      // any recorded error: copy nothing
    const int64_t N0 = offsets[P];
    const int64_t N = N0 <= canon_cap ? N0 : 0;
    const int64_t T = N > 0 ? ctl->total : 0;           // output bytes, from the scan
    if (T <= 0) return;
    const int64_t nsub = (N + kSub - 1) / kSub;
    const uint64_t outa = reinterpret_cast<uint64_t>(out);
    const int64_t mis = (int64_t)(outa & 15);
    const int64_t nwaves = (int64_t)gridDim.x * kWaves;
    int64_t G, nunits;
    copy_units(T, nwaves, mis, G, nunits);
    const int wave = uni32((int)(threadIdx.x >> 6)), lane = lane_id();
    int32_t *s_dst = s_dst_all[wave];
    uint64_t *s_src = s_src_all[wave];
    int32_t *s_edge = s_edge_all[wave];
    int16_t *s_edger = s_edger_all[wave];
    for (int64_t u = (int64_t)blockIdx.x * kWaves + wave; u < nunits; u += nwaves) {
        const int64_t lo = max64(u * G - mis, 0);
        const int64_t hi = min64((u + 1) * G - mis, T);
        for (int64_t sb = uni64(find_sub_tile(sub_base, nsub, lo)); sb < nsub; ++sb) {
            const int64_t D0 = sub_base[sb];
            if (D0 >= hi) break;
            const int64_t c0 = sb * kSub;
            const int64_t cnt = min64(kSub, N - c0);
            // surviving lengths -> destination offsets relative to the sub-tile
            int64_t lsum = 0;
            uint32_t l[kCopyPer];
            uint64_t s[kCopyPer];
            // whole 16-byte slots, all four loads in flight together (a
            // slot past the expansion re-reads the last one and is ignored)
            uint4 ev[kCopyPer];
#pragma unroll
            for (int k = 0; k < kCopyPer; ++k) {
                const int64_t r = (int64_t)lane * kCopyPer + k;
                ev[k] = ld16(reinterpret_cast<uint64_t>(&canon[c0 + (r < cnt ? r : cnt - 1)]));
            }
#pragma unroll
            for (int k = 0; k < kCopyPer; ++k) {
                const int64_t r = (int64_t)lane * kCopyPer + k;
                const bool ok = r < cnt && ev[k].w == ((epoch << 2) | RO_SUCCESS);
                l[k] = ok ? ev[k].z : 0u;
                s[k] = ok ? ((uint64_t)ev[k].y << 32 | ev[k].x) : 0ull;
                lsum += l[k];
            }
            const int64_t inc = wave_incl_sum(lsum);
            const int64_t tot = uni64(__shfl(inc, 63, 64));
            // this unit's part of the sub-tile: [ws, we), relative to D0
            const int64_t ws = max64(lo - D0, 0), we = min64(hi - D0, tot);
            if (we > ws) {
                int64_t run = inc - lsum;
#pragma unroll
                for (int k = 0; k < kCopyPer; ++k) {
                    const int r = lane * kCopyPer + k;
                    const int64_t cs = min64(max64(run, ws), we);
                    s_dst[r] = (int32_t)(cs - ws);
                    s_src[r] = s[k] + (uint64_t)(cs - run);
                    run += l[k];
                }
                if (lane == 0) s_dst[kSub] = (int32_t)(we - ws);
                __builtin_amdgcn_wave_barrier();
                copy_window_nb<RO_COPY_STEPS>(s_dst, s_src, s_edge, s_edger, (int)(we - ws), outa, D0 + ws, lane);
                __builtin_amdgcn_wave_barrier();
            }
        }
    }
}

hipError_t launch_gather(const Launch &L, const GatherArgs &a, const GatherWs &w, uint32_t epoch)
{
    if (a.barrier != nullptr && a.n > 0) {
        const hipError_t e = launch_first_gf(L, a.rs, a.rp, a.n, a.P, a.barrier, w.gkey, epoch);
        if (e != hipSuccess) return e;
    }
    const int64_t grid_r = (int64_t)L.num_cus * 8;
    RO_LAUNCH(L, RO_K_GATHER_SCATTER, k_gather_scatter, dim3((unsigned)grid_r), dim3(kBlock), 0, L.stream,
              a.rp, a.ro, a.rs, a.roff, a.data, a.n, a.offsets, a.P, w.canon, w.canon_cap, a.ns, a.nf,
              a.nk, a.barrier, w.gkey, epoch, L.ctl);
    // three workgroups per CU drew tickets faster than four (fewer waiting
    // on the look-back at once) and two left the largest scans short of work
    const int64_t grid_s = (int64_t)L.num_cus * RO_SCAN_WG;
    // output aliasing the report bytes: the scan checks that nothing moves,
    // and there is nothing to copy
    const bool in_place = a.out_data != nullptr && a.out_data == a.data;
    if (in_place) {
        RO_LAUNCH(L, RO_K_GATHER_SCAN, k_gather_scan<true>, dim3((unsigned)grid_s), dim3(kBlock), 0, L.stream,
                  a.offsets, a.P, w.canon, w.canon_cap, a.out_off, a.ns, a.nf, a.nk, a.cdst, w.sub_base, a.out_data,
                  epoch, L.ctl, L.desc, L.desc_cap);
    } else {
        RO_LAUNCH(L, RO_K_GATHER_SCAN, k_gather_scan<false>, dim3((unsigned)grid_s), dim3(kBlock), 0, L.stream,
                  a.offsets, a.P, w.canon, w.canon_cap, a.out_off, a.ns, a.nf, a.nk, a.cdst, w.sub_base, nullptr,
                  epoch, L.ctl, L.desc, L.desc_cap);
    }
    int64_t grid_f = (a.P + kBlock - 1) / kBlock;
    grid_f = grid_f < 1 ? 1 : (grid_f > (int64_t)L.num_cus * 8 ? (int64_t)L.num_cus * 8 : grid_f);
    RO_LAUNCH(L, RO_K_GATHER_FINALIZE, k_gather_finalize, dim3((unsigned)grid_f), dim3(kBlock), 0, L.stream, a.offsets,
                       a.P, w.canon_cap, a.out_off, a.out_cap, a.out_data != nullptr ? 1 : 0, a.ns, a.nf,
                       a.nk, a.complete, a.pstate, a.cdst, a.barrier, w.gkey, a.n_rejected, epoch, L.ctl);
    if (a.out_data != nullptr && !in_place) {
        // many small workgroups: a unit's cost varies with the records it
        // meets, and a deep queue of workgroups evens out the tail
        const int64_t grid_c = (int64_t)L.num_cus * RO_COPY_GRID;
        RO_LAUNCH(L, RO_K_GATHER_COPY, k_gather_copy, dim3((unsigned)grid_c), dim3(kBlock), 0, L.stream, a.offsets,
                  a.P, w.canon, w.canon_cap, w.sub_base, a.out_data, epoch, L.ctl);
    }
    return hipGetLastError();
}

}  // namespace ro
