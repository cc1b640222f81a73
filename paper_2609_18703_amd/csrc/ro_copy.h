// Byte-copy building blocks shared by the gather and the streaming emission:
// 16-byte aligned stores of byte-aligned records, assembled in registers.
#pragma once

#include "ro_device.h"

namespace ro {

// Payload accesses use explicit global-address-space pointers so they compile
// to global_load/global_store (flat accesses would also hold up every LDS
// read of the record search behind outstanding memory traffic).
#define RO_GLOBAL __attribute__((address_space(1)))

typedef uint32_t v4u32 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint4 ld16(uint64_t a)
{
    const v4u32 t = *(const RO_GLOBAL v4u32 *)a;
    return make_uint4(t.x, t.y, t.z, t.w);
}
__device__ __forceinline__ void st16(uint64_t a, uint4 v)
{
    const v4u32 t = {v.x, v.y, v.z, v.w};
    *(RO_GLOBAL v4u32 *)a = t;
}
__device__ __forceinline__ void st8(uint64_t a, uint8_t v) { *(RO_GLOBAL uint8_t *)a = v; }

// Bytes sh..sh+15 of the 32-byte pair (lo, hi), with selects only (sh
// differs between lanes, so a branch on it would split the wave).
__device__ __forceinline__ uint4 shift16(const uint4 &lo, const uint4 &hi, uint32_t sh)
{
    const bool b3 = (sh & 8u) != 0, b2 = (sh & 4u) != 0;
    const uint32_t bs = sh & 3u;
    const uint32_t t0 = b3 ? lo.z : lo.x, t1 = b3 ? lo.w : lo.y, t2 = b3 ? hi.x : lo.z;
    const uint32_t t3 = b3 ? hi.y : lo.w, t4 = b3 ? hi.z : hi.x, t5 = b3 ? hi.w : hi.y;
    const uint32_t w0 = b2 ? t1 : t0, w1 = b2 ? t2 : t1, w2 = b2 ? t3 : t2, w3 = b2 ? t4 : t3, w4 = b2 ? t5 : t4;
    uint4 r;
    r.x = __builtin_amdgcn_alignbyte(w1, w0, bs);
    r.y = __builtin_amdgcn_alignbyte(w2, w1, bs);
    r.z = __builtin_amdgcn_alignbyte(w3, w2, bs);
    r.w = __builtin_amdgcn_alignbyte(w4, w3, bs);
    return r;
}

// One record's share of an output chunk: output bytes fv..lv (0..15) come
// from source addresses S+fv .. S+lv.  Only the aligned 16-byte source
// chunks holding some of those bytes are read, so no load leaves a page the
// record occupies.
struct Piece {
    uint4 lo, hi;
    uint32_t sh;
    int fv, lv;
};

__device__ __forceinline__ void piece_load(Piece &p, uint64_t S, int fv, int lv)
{
    const uint64_t c0 = S & ~(uint64_t)15;
    p.sh = (uint32_t)(S & 15);
    p.fv = fv;
    p.lv = lv;
    const bool need0 = S + (uint64_t)fv < c0 + 16;
    const bool need1 = S + (uint64_t)lv >= c0 + 16;
    // Both loads are unconditional (a conditional load makes the compiler
    // zero its destination first, which waits for every outstanding memory
    // operation); a half that is not needed re-reads the one that is, and
    // its bytes are masked off by piece_merge.
    p.lo = ld16(need0 ? c0 : c0 + 16);
    p.hi = ld16(need1 ? c0 + 16 : c0);
}

// Byte mask of output bytes fv..lv that fall in dword j.
__device__ __forceinline__ uint32_t byte_mask(int j, int fv, int lv)
{
    const int a = fv - 4 * j > 0 ? fv - 4 * j : 0;
    const int b = lv - 4 * j < 3 ? lv - 4 * j : 3;
    if (a > b) return 0u;
    return (0xffffffffu >> (8 * (3 - b))) & (0xffffffffu << (8 * a));
}

__device__ __forceinline__ void piece_merge(uint4 &acc, const Piece &p)
{
    const uint4 v = shift16(p.lo, p.hi, p.sh);
    uint32_t m;
    m = byte_mask(0, p.fv, p.lv); acc.x = (acc.x & ~m) | (v.x & m);
    m = byte_mask(1, p.fv, p.lv); acc.y = (acc.y & ~m) | (v.y & m);
    m = byte_mask(2, p.fv, p.lv); acc.z = (acc.z & ~m) | (v.z & m);
    m = byte_mask(3, p.fv, p.lv); acc.w = (acc.w & ~m) | (v.w & m);
}

__device__ __forceinline__ uint32_t dword_of(const uint4 &v, int j)
{
    return j == 0 ? v.x : (j == 1 ? v.y : (j == 2 ? v.z : v.w));
}

constexpr int kCopyPer = kSub / 64;       // records per lane in a wave's copy prologue

// Largest r in [r, kSub] with s_dst[r] <= pos, given s_dst[r] <= pos: a few
// linear steps (the usual distance between neighbouring chunks), then a
// binary search.  Zero-length records are stepped over.
__device__ __forceinline__ int advance_record(const int32_t *s_dst, int r, int pos)
{
#pragma unroll 1
    for (int step = 0; step < 6; ++step) {
        if (s_dst[r + 1] > pos) return r;
        ++r;
    }
    int rl = r, rh = kSub + 1;
    while (rh - rl > 1) {
        const int mid = (rl + rh) >> 1;
        if (s_dst[mid] <= pos) rl = mid; else rh = mid;
    }
    return rl;
}

// Store the bytes [b0, b1) (0..16) of a 16-byte chunk value at A.
__device__ __forceinline__ void store_partial(uint64_t A, const uint4 &v, int b0, int b1)
{
    for (int b = b0; b < b1; ++b) st8(A + (uint64_t)b, (uint8_t)(dword_of(v, b >> 2) >> (8 * (b & 3))));
}

// The rest of one chunk at x (output bytes [lo, hi) of the window) once the
// piece of its first record r has been loaded: the pieces of any further
// records it holds, the merge and the store.  r moves to the chunk's last
// record.
__device__ __forceinline__ void copy_one_chunk(const int32_t *s_dst, const uint64_t *s_src, uint64_t outa, int64_t D0,
                                               int x, int lo, int hi, int &r, const Piece &p, int e1)
{
    uint4 acc = make_uint4(0u, 0u, 0u, 0u);
    if (e1 < hi) {
        int q = advance_record(s_dst, r, e1);
        int e = e1;
        while (e < hi) {
            const int dq = s_dst[q + 1];
            const int e2 = hi < dq ? hi : dq;
            Piece pq;
            piece_load(pq, s_src[q] + (uint64_t)(int64_t)(x - s_dst[q]), e - x, e2 - 1 - x);
            piece_merge(acc, pq);
            e = e2;
            if (e < hi) q = advance_record(s_dst, q, e);
        }
        r = q;
    }
    piece_merge(acc, p);
    const uint64_t A = outa + (uint64_t)(D0 + x);
    if (lo == x && hi == x + 16) st16(A, acc);
    else store_partial(A, acc, lo - x, hi - x);     // first or last chunk of the window
}

// One unit's window of a sub-tile (at most 1 GiB): positions relative to the
// window start fit in 32 bits.  The wave sweeps its window 1 KiB at a time,
// lane `lane` taking chunk 64*g + lane, so the record each lane reads from
// only moves forward.  Every chunk strictly inside the window is written with
// one aligned 16-byte store; chunks that straddle records are assembled from
// their pieces first, with all of their loads in flight together.
__device__ __forceinline__ void copy_window32(const int32_t *s_dst, const uint64_t *s_src, int tot,
                                              uint64_t outa, int64_t D0, int lane)
{
    const uint64_t a0 = (outa + (uint64_t)D0) & ~(uint64_t)15;
    const uint64_t a1 = (outa + (uint64_t)(D0 + tot) - 1) & ~(uint64_t)15;
    const int nchunks = (int)((a1 - a0) >> 4) + 1;
    const int xbase = (int)((int64_t)(a0 - outa) - D0);     // -15..0
    int r = 0;
    for (int ch = lane; ch < nchunks; ch += 64) {
        const int x = xbase + ch * 16;
        const int lo = x > 0 ? x : 0;
        const int hi = x + 16 < tot ? x + 16 : tot;
        r = advance_record(s_dst, r, lo);
        const int d1 = s_dst[r + 1];
        const int e1 = hi < d1 ? hi : d1;
        Piece p;
        piece_load(p, s_src[r] + (uint64_t)(int64_t)(x - s_dst[r]), lo - x, e1 - 1 - x);
        copy_one_chunk(s_dst, s_src, outa, D0, x, lo, hi, r, p, e1);
    }
}

// Lane i receives lane i + 1's value (a wave-wide DPP shift); lane 63
// receives `old`.  All 64 lanes must be active.
__device__ __forceinline__ uint32_t from_next_lane(uint32_t v, uint32_t old)
{
    return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)v, 0x130, 0xf, 0xf, false);
}

// Chunks a window can list for the edge pass: at most one per record end in
// the window plus its first and last chunk.
constexpr int kEdgeCap = kSub + 4;

// The edge chunks listed by copy_window_nb, 64 at a time, byte by byte: the
// source of every byte of the chunk is found among the window's records and
// all sixteen byte loads are in flight together (a byte outside the window
// re-reads the chunk's last byte inside it and is not stored).  Few chunks
// take this path (the two ends of a window, and chunks holding three or more
// records), so it is written for few registers rather than speed.
__device__ __forceinline__ void copy_edges(const int32_t *s_dst, const uint64_t *s_src, const int32_t *s_edge,
                                           const int16_t *s_edger, int nedge, int xbase, int tot, uint64_t outa,
                                           int64_t D0, int lane)
{
    for (int j = lane; j < nedge; j += 64) {
        const int x = xbase + s_edge[j] * 16;
        int q = s_edger[j];
        const int lo = x > 0 ? x : 0;
        const int hi = x + 16 < tot ? x + 16 : tot;
        uint32_t bv[16];
#pragma unroll
        for (int b = 0; b < 16; ++b) {
            const int pos = x + b < lo ? lo : (x + b >= hi ? hi - 1 : x + b);
            q = advance_record(s_dst, q, pos);
            bv[b] = *(const RO_GLOBAL uint8_t *)(s_src[q] + (uint64_t)(int64_t)(pos - s_dst[q]));
        }
        const uint64_t A = outa + (uint64_t)(D0 + x);
        if (lo == x && hi == x + 16) {
            v4u32 v;
#pragma unroll
            for (int d = 0; d < 4; ++d)
                v[d] = bv[4 * d] | bv[4 * d + 1] << 8 | bv[4 * d + 2] << 16 | bv[4 * d + 3] << 24;
            *(RO_GLOBAL v4u32 *)A = v;
        } else {
#pragma unroll
            for (int b = 0; b < 16; ++b)
                if (x + b >= lo && x + b < hi) st8(A + (uint64_t)b, (uint8_t)bv[b]);
        }
    }
}

// The same on native 4-dword vectors (kept in registers even in arrays
// written under a condition).
__device__ __forceinline__ v4u32 ld16v(uint64_t a) { return *(const RO_GLOBAL v4u32 *)a; }
__device__ __forceinline__ void st16v(uint64_t a, v4u32 v) { *(RO_GLOBAL v4u32 *)a = v; }

__device__ __forceinline__ v4u32 shift16v(v4u32 lo, v4u32 hi, uint32_t sh)
{
    const bool b3 = (sh & 8u) != 0, b2 = (sh & 4u) != 0;
    const uint32_t bs = sh & 3u;
    const uint32_t t0 = b3 ? lo.z : lo.x, t1 = b3 ? lo.w : lo.y, t2 = b3 ? hi.x : lo.z;
    const uint32_t t3 = b3 ? hi.y : lo.w, t4 = b3 ? hi.z : hi.x, t5 = b3 ? hi.w : hi.y;
    const uint32_t w0 = b2 ? t1 : t0, w1 = b2 ? t2 : t1, w2 = b2 ? t3 : t2, w3 = b2 ? t4 : t3, w4 = b2 ? t5 : t4;
    v4u32 r;
    r.x = __builtin_amdgcn_alignbyte(w1, w0, bs);
    r.y = __builtin_amdgcn_alignbyte(w2, w1, bs);
    r.z = __builtin_amdgcn_alignbyte(w3, w2, bs);
    r.w = __builtin_amdgcn_alignbyte(w4, w3, bs);
    return r;
}

// Bytes [0, n) of a, bytes [n, 16) of b (0 <= n <= 16).
__device__ __forceinline__ v4u32 merge_at(v4u32 a, v4u32 b, int n)
{
    v4u32 m;
#pragma unroll
    for (int d = 0; d < 4; ++d) {
        const int k = n - 4 * d;
        m[d] = k >= 4 ? 0xffffffffu : (k <= 0 ? 0u : (0xffffffffu >> (8 * (4 - k))));
    }
    return (a & m) | (b & ~m);
}

// One unit's window of a sub-tile, with about one aligned 16-byte source load
// per output chunk.  A step of the wave covers 64 consecutive output chunks,
// one per lane, and every lane loads the aligned source chunk holding the
// first byte its chunk needs.  Inside a record, lane i's chunk needs source
// bytes [s, s + 16), which lie in its own load and the aligned chunk after
// it: the one lane i + 1 loaded whenever lane i + 1 sits in the same record,
// so the pair is completed with a cross-lane move.  A chunk that holds the
// end of one record and the start of the next takes its second piece's
// upper half the same way (lane i + 1 loaded the chunk after the one holding
// the piece's start) and loads what else it needs itself, in the same step:
// every store of a step is whole when the step ends, so no cache line is
// left half written.  U steps are in flight per lane, their loads issued
// together.  Chunks at the window's two ends, chunks holding three or more
// records (records under 16 bytes) and two-record chunks whose second
// record does not go on into lane i + 1's chunk (it ends with the chunk, or
// the chunk is lane 63's) are listed in LDS and written after the sweep,
// byte by byte.
template <int U>
__device__ __forceinline__ void copy_window_nb(const int32_t *s_dst, const uint64_t *s_src, int32_t *s_edge,
                                               int16_t *s_edger, int tot, uint64_t outa, int64_t D0, int lane)
{
    const uint64_t a0 = (outa + (uint64_t)D0) & ~(uint64_t)15;
    const uint64_t a1 = (outa + (uint64_t)(D0 + tot) - 1) & ~(uint64_t)15;
    const int nchunks = (int)((a1 - a0) >> 4) + 1;
    const int xbase = (int)((int64_t)(a0 - outa) - D0);     // -15..0
    const uint64_t dbase = outa + (uint64_t)D0;             // destination of window byte 0
    // a chunk every lane may load: the one holding the window's first byte
    const uint64_t safe = (uint64_t)uni64((int64_t)(s_src[advance_record(s_dst, 0, 0)] & ~(uint64_t)15));
    int r = 0, nedge = 0;
    for (int s0 = 0; s0 * 64 < nchunks; s0 += U) {
        // info: bits 0-1 kind (0 nothing to write, 1 one record, 2 two
        // records, 3 listed), bit 2 first piece completed by lane i + 1,
        // bit 3 second piece completed by lane i + 1, bits 4-7 shift of the
        // first piece, 8-11 of the second, 12-16 length of the first piece
        uint32_t info[U];
        int rr[U];
        v4u32 L0[U], X1[U], X2[U];
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const int ch = (s0 + k) * 64 + lane;
            const int x = xbase + ch * 16;
            uint32_t f = 0;
            int q = -1;
            rr[k] = -1;
            uint64_t A0 = safe, C2 = safe;
            if (ch < nchunks) {
                const int b0 = x > 0 ? x : 0;
                r = advance_record(s_dst, r, b0);
                rr[k] = r;
                const int d1 = s_dst[r + 1];
                // source address of window byte 0, extended linearly through r
                const uint64_t vb = s_src[r] - (uint64_t)(int64_t)s_dst[r];
                A0 = (vb + (uint64_t)(int64_t)b0) & ~(uint64_t)15;
                f = 3;
                if (x >= 0 && x + 16 <= tot) {
                    const uint32_t sh1 = (uint32_t)(vb + (uint64_t)(int64_t)x) & 15u;
                    if (d1 >= x + 16) {
                        f = 1 | sh1 << 4 | 16u << 12;
                    } else {
                        const int qq = advance_record(s_dst, r, d1);
                        if (s_dst[qq + 1] > x + 16) {
                            q = qq;
                            const uint64_t V2 = s_src[q] - (uint64_t)(int64_t)s_dst[q] + (uint64_t)(int64_t)x;
                            f = 2 | sh1 << 4 | ((uint32_t)V2 & 15u) << 8 | (uint32_t)(d1 - x) << 12;
                            C2 = V2 & ~(uint64_t)15;
                        }
                    }
                }
            }
            // the record holding lane i + 1's first byte (-1 past the window)
            const int rn = (int)from_next_lane((uint32_t)rr[k], 0xffffffffu);
            // a second piece whose upper half lane i + 1 does not hold (lane
            // 63) is listed
            if ((f & 3u) == 2u && rn != q) f = 3;
            const v4u32 z = {0u, 0u, 0u, 0u};
            X1[k] = z;
            X2[k] = z;
            L0[k] = ld16v(A0);
            const uint32_t kd = f & 3u, sh1 = (f >> 4) & 15u, sh2 = (f >> 8) & 15u;
            const int n1 = (int)(f >> 12);
            // second source chunk of the first piece, unless lane i + 1 has it
            const bool n_x1 = (kd == 1 && sh1 != 0 && rn != rr[k]) || (kd == 2 && (int)sh1 + n1 > 16);
            // first source chunk of the second piece, if it holds any of it
            // (its second chunk is lane i + 1's)
            const bool n_x2 = kd == 2 && n1 + (int)sh2 < 16;
            f |= rn == rr[k] ? 4u : 0u;
            f |= (kd == 2) ? 8u : 0u;
            info[k] = f;
            if (n_x1) X1[k] = ld16v(A0 + 16);
            if (n_x2) X2[k] = ld16v(C2);
        }
#pragma unroll
        for (int k = 0; k < U; ++k) {
            v4u32 nb;
            nb.x = from_next_lane(L0[k].x, 0u);
            nb.y = from_next_lane(L0[k].y, 0u);
            nb.z = from_next_lane(L0[k].z, 0u);
            nb.w = from_next_lane(L0[k].w, 0u);
            const uint32_t f = info[k];
            // one record: the first piece is the whole chunk
            const v4u32 h1 = (f & 4u) ? nb : X1[k];
            const v4u32 v = merge_at(shift16v(L0[k], h1, (f >> 4) & 15u), shift16v(X2[k], nb, (f >> 8) & 15u),
                                     (int)(f >> 12));
            const uint32_t kd = f & 3u;
            const int x = xbase + ((s0 + k) * 64 + lane) * 16;
            if (kd == 1 || kd == 2) st16v(dbase + (uint64_t)x, v);
            const bool listed = kd == 3;
            const uint64_t m = __ballot(listed);
            if (listed) {
                const int pos = nedge + __popcll(m & ((1ull << lane) - 1ull));
                s_edge[pos] = (s0 + k) * 64 + lane;
                s_edger[pos] = (int16_t)rr[k];
            }
            nedge += __popcll(m);
        }
    }
    __builtin_amdgcn_wave_barrier();
    copy_edges(s_dst, s_src, s_edge, s_edger, nedge, xbase, tot, outa, D0, lane);
}

// Output bytes are split into units of G bytes (the last one shorter), cut
// where the destination address is 16-byte aligned, so that unit edges need
// no partial stores.  G is chosen from the total so that every wave of the
// grid gets about kCopyUnits units, but never under kCopyMinUnit bytes (a
// unit re-reads the slot descriptors of the sub-tiles it touches) nor over
// 1 GiB (positions inside a unit are 32-bit).
// Copy kernels trade per-wave registers for occupancy: the compiler keeps
// register use low enough for at least this many waves per SIMD.
#ifndef RO_COPY_WAVES
#define RO_COPY_WAVES 5
#endif
#ifndef RO_COPY_STEPS
#define RO_COPY_STEPS 2
#endif
#ifndef RO_COPY_UNITS
#define RO_COPY_UNITS 2
#endif
#ifndef RO_COPY_MIN_UNIT
#define RO_COPY_MIN_UNIT (128 << 10)
#endif
constexpr int64_t kCopyUnits = RO_COPY_UNITS;
constexpr int64_t kCopyMinUnit = RO_COPY_MIN_UNIT;

// Unit size G and unit count for T output bytes copied by nwaves waves into
// a buffer whose address is `mis` bytes past a 16-byte boundary.
__device__ __forceinline__ void copy_units(int64_t T, int64_t nwaves, int64_t mis, int64_t &G, int64_t &nunits)
{
    G = (T + nwaves * kCopyUnits - 1) / (nwaves * kCopyUnits);
    G = (G + 1023) & ~(int64_t)1023;
    G = G < kCopyMinUnit ? kCopyMinUnit : (G > ((int64_t)1 << 30) ? ((int64_t)1 << 30) : G);
    nunits = (T + mis + G - 1) / G;
}

}  // namespace ro
