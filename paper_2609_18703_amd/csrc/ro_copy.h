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

// Bytes sh..sh+15 of the 32-byte pair (lo, hi).
__device__ __forceinline__ uint4 shift16(const uint4 &lo, const uint4 &hi, uint32_t sh)
{
    const uint32_t dw = sh >> 2, bs = sh & 3;
    uint32_t w0, w1, w2, w3, w4;
    if (dw == 0)      { w0 = lo.x; w1 = lo.y; w2 = lo.z; w3 = lo.w; w4 = hi.x; }
    else if (dw == 1) { w0 = lo.y; w1 = lo.z; w2 = lo.w; w3 = hi.x; w4 = hi.y; }
    else if (dw == 2) { w0 = lo.z; w1 = lo.w; w2 = hi.x; w3 = hi.y; w4 = hi.z; }
    else              { w0 = lo.w; w1 = hi.x; w2 = hi.y; w3 = hi.z; w4 = hi.w; }
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

// copy_window32 with two chunks per lane and step (the lane's chunk and the
// one 1 KiB further), the first pieces of both in flight together: twice
// the loads outstanding per wave at the same occupancy.  Used where a unit's
// window spans many KiB (the gather); small windows keep the one-chunk loop.
__device__ __forceinline__ void copy_window32_x2(const int32_t *s_dst, const uint64_t *s_src, int tot,
                                                 uint64_t outa, int64_t D0, int lane)
{
    const uint64_t a0 = (outa + (uint64_t)D0) & ~(uint64_t)15;
    const uint64_t a1 = (outa + (uint64_t)(D0 + tot) - 1) & ~(uint64_t)15;
    const int nchunks = (int)((a1 - a0) >> 4) + 1;
    const int xbase = (int)((int64_t)(a0 - outa) - D0);     // -15..0
    int r = 0;
    for (int ch = lane; ch < nchunks; ch += 128) {
        // two chunks 1 KiB apart, the first pieces of both loaded together
        const int xA = xbase + ch * 16;
        const int loA = xA > 0 ? xA : 0;
        const int hiA = xA + 16 < tot ? xA + 16 : tot;
        r = advance_record(s_dst, r, loA);
        int rA = r;
        const int d1A = s_dst[rA + 1];
        const int e1A = hiA < d1A ? hiA : d1A;
        Piece pA;
        piece_load(pA, s_src[rA] + (uint64_t)(int64_t)(xA - s_dst[rA]), loA - xA, e1A - 1 - xA);
        const bool two = ch + 64 < nchunks;
        const int xB = xA + 1024;
        const int loB = xB;
        const int hiB = xB + 16 < tot ? xB + 16 : tot;
        int rB = r;
        int e1B = hiB;
        Piece pB;
        if (two) {
            rB = advance_record(s_dst, r, loB);
            const int d1B = s_dst[rB + 1];
            e1B = hiB < d1B ? hiB : d1B;
            piece_load(pB, s_src[rB] + (uint64_t)(int64_t)(xB - s_dst[rB]), loB - xB, e1B - 1 - xB);
        }
        copy_one_chunk(s_dst, s_src, outa, D0, xA, loA, hiA, rA, pA, e1A);
        if (two) {
            copy_one_chunk(s_dst, s_src, outa, D0, xB, loB, hiB, rB, pB, e1B);
            r = rB;
        } else {
            r = rA;
        }
    }
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
