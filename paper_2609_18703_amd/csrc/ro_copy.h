// Byte-copy building blocks shared by the gather and the streaming emission:
// byte-aligned records written with aligned 16-byte stores, read with
// 16-byte loads from their exact source addresses.
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
__device__ __forceinline__ void st8(uint64_t a, uint8_t v) { *(RO_GLOBAL uint8_t *)a = v; }

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

// Loads and stores on native 4-dword vectors (kept in registers even in
// arrays written under a condition).  ld16v takes any byte address: gfx950
// serves a misaligned 16-byte global load as one load returning the 16 bytes
// at that address, at the speed of an aligned one (the type tells the
// compiler to assume no alignment).
typedef uint32_t v4u32_u1 __attribute__((ext_vector_type(4), aligned(1)));
__device__ __forceinline__ v4u32 ld16v(uint64_t a) { return *(const RO_GLOBAL v4u32_u1 *)a; }
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

// One unit's window of a sub-tile.  A step of the wave covers 64
// consecutive output chunks, one per lane, each written with one aligned
// 16-byte store.  A chunk inside one record takes one 16-byte load from its
// exact (byte-aligned) source address: a misaligned 16-byte global load
// returns the 16 bytes at that address, at the speed of an aligned one, and
// all of them are bytes of the record.  A chunk holding the end of record r
// and the start of record q takes two: the 16 bytes that end where r ends
// and the 16 that start where q starts (both inside their records); the
// chunk is bytes 16 - n1 .. 31 - n1 of the two side by side, n1 being r's
// share of it.  Every store of a step is whole when the step ends, so no
// cache line is left half written.  U steps are in flight per lane, their
// loads issued together.  Chunks at the window's two ends, chunks holding
// three or more records, and two-record chunks with a side shorter than 16
// bytes in the window (records under 16 bytes) are listed in LDS and
// written after the sweep, byte by byte.
template <int U>
__device__ __forceinline__ void copy_window_nb(const int32_t *s_dst, const uint64_t *s_src, int32_t *s_edge,
                                               int16_t *s_edger, int tot, uint64_t outa, int64_t D0, int lane)
{
    const uint64_t a0 = (outa + (uint64_t)D0) & ~(uint64_t)15;
    const uint64_t a1 = (outa + (uint64_t)(D0 + tot) - 1) & ~(uint64_t)15;
    const int nchunks = (int)((a1 - a0) >> 4) + 1;
    const int xbase = (int)((int64_t)(a0 - outa) - D0);     // -15..0
    const uint64_t dbase = outa + (uint64_t)D0;             // destination of window byte 0
    // an address every lane may load from: the window's first source byte
    // (its record holds at least one byte, and 16 bytes from it stay in the
    // record or in the aligned 16-byte chunks next to it only when the
    // record is that long, so lanes with nothing to do load from its aligned
    // chunk instead)
    const uint64_t safe = (uint64_t)uni64((int64_t)(s_src[advance_record(s_dst, 0, 0)] & ~(uint64_t)15));
    int r = 0, nedge = 0;
    for (int s0 = 0; s0 * 64 < nchunks; s0 += U) {
        // kind: 0 nothing, 1 one record, 2 two records, 3 listed
        int kind[U], n1[U], rr[U];
        v4u32 L[U], X[U];
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const int ch = (s0 + k) * 64 + lane;
            const int x = xbase + ch * 16;
            uint64_t A = safe, B = safe;
            kind[k] = 0;
            n1[k] = 16;
            rr[k] = -1;
            if (ch < nchunks) {
                const int b0 = x > 0 ? x : 0;
                r = advance_record(s_dst, r, b0);
                rr[k] = r;
                kind[k] = 3;
                if (x >= 0 && x + 16 <= tot) {
                    const int d0 = s_dst[r], d1 = s_dst[r + 1];
                    // source of window byte 0, extended linearly through r
                    const uint64_t vb = s_src[r] - (uint64_t)(int64_t)d0;
                    if (d1 >= x + 16) {
                        kind[k] = 1;
                        A = vb + (uint64_t)(int64_t)x;
                    } else if (d1 - d0 >= 16) {
                        const int q = advance_record(s_dst, r, d1);
                        const int e0 = s_dst[q], e1 = s_dst[q + 1];
                        if (e1 > x + 16 && e1 - e0 >= 16) {
                            kind[k] = 2;
                            n1[k] = d1 - x;
                            A = vb + (uint64_t)(int64_t)(d1 - 16);                  // ends where r ends
                            B = s_src[q] + (uint64_t)(int64_t)(d1 - e0);            // starts where q starts
                        }
                    }
                }
            }
            const v4u32 z = {0u, 0u, 0u, 0u};
            X[k] = z;
            L[k] = ld16v(A);
            if (kind[k] == 2) X[k] = ld16v(B);
        }
#pragma unroll
        for (int k = 0; k < U; ++k) {
            v4u32 v = L[k];
            if (__ballot(kind[k] == 2) != 0) {
                const v4u32 w = shift16v(L[k], X[k], (uint32_t)(16 - n1[k]) & 15u);
                if (kind[k] == 2) v = w;
            }
            const int x = xbase + ((s0 + k) * 64 + lane) * 16;
            if (kind[k] == 1 || kind[k] == 2) st16v(dbase + (uint64_t)x, v);
            const bool listed = kind[k] == 3;
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
#define RO_COPY_WAVES 4
#endif
#ifndef RO_COPY_STEPS
#define RO_COPY_STEPS 6
#endif
#ifndef RO_COPY_GRID
#define RO_COPY_GRID 32                     // gather copy workgroups per CU
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
