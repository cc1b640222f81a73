// F.filter and F.broadcast on gfx950.
//
// RayOrch (arXiv 2609.18703), Table "primitives" and Sec. 4 input
// propagation: filter keeps or drops an Item within its Domain, broadcast
// makes an ancestor's Item available in a descendant Domain; both derive the
// output state by the same precedence (a failed or suppressed input
// suppresses, an unresolved one waits, a dropped required one drops,
// otherwise the output is ready).  Both are one pass over the output Domain:
// the filter takes 16 states per thread and load; the broadcast one
// descendant per thread, whose chained map lookups mostly hit in cache.
#include "ro_device.h"

namespace ro {

// Precedence over two states, FAILED before PENDING before SKIPPED before
// SUCCESS; anything above PENDING is a bad state (returned as 0xff).
__device__ __forceinline__ uint32_t propagate2(uint32_t a, uint32_t b)
{
    if (a > RO_PENDING || b > RO_PENDING) return 0xffu;
    if (a == RO_FAILED || b == RO_FAILED) return RO_FAILED;
    if (a == RO_PENDING || b == RO_PENDING) return RO_PENDING;
    if (a == RO_SKIPPED || b == RO_SKIPPED) return RO_SKIPPED;
    return RO_SUCCESS;
}

__global__ __launch_bounds__(kBlock) void k_filter(const uint8_t *__restrict__ xs, const uint8_t *__restrict__ ms,
                                                   const uint8_t *__restrict__ mv, int64_t n, uint8_t *__restrict__ out,
                                                   int vec, Ctl *ctl)
{
    const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    bool bad = false;
    if (vec) {
        // 16 items per thread: one 16-byte load per input, one store
        for (int64_t i0 = g * 16; i0 < n; i0 += stride * 16) {
            if (i0 + 16 <= n) {
                const uint4 x = *reinterpret_cast<const uint4 *>(xs + i0);
                const uint4 m = ms ? *reinterpret_cast<const uint4 *>(ms + i0) : make_uint4(0, 0, 0, 0);
                const uint4 v = *reinterpret_cast<const uint4 *>(mv + i0);
                const uint32_t xw[4] = {x.x, x.y, x.z, x.w}, mw[4] = {m.x, m.y, m.z, m.w}, vw[4] = {v.x, v.y, v.z, v.w};
                uint32_t ow[4];
#pragma unroll
                for (int w = 0; w < 4; ++w) {
                    uint32_t o = 0;
#pragma unroll
                    for (int b = 0; b < 4; ++b) {
                        uint32_t s = propagate2((xw[w] >> (8 * b)) & 0xffu, (mw[w] >> (8 * b)) & 0xffu);
                        bad |= s == 0xffu;
                        if (s == RO_SUCCESS && ((vw[w] >> (8 * b)) & 0xffu) == 0) s = RO_SKIPPED;
                        o |= (s & 0xffu) << (8 * b);
                    }
                    ow[w] = o;
                }
                *reinterpret_cast<uint4 *>(out + i0) = make_uint4(ow[0], ow[1], ow[2], ow[3]);
            } else {
                for (int64_t i = i0; i < n; ++i) {
                    uint32_t s = propagate2(xs[i], ms ? ms[i] : RO_SUCCESS);
                    bad |= s == 0xffu;
                    if (s == RO_SUCCESS && mv[i] == 0) s = RO_SKIPPED;
                    out[i] = (uint8_t)s;
                }
            }
        }
    } else {
        for (int64_t i = g; i < n; i += stride) {
            uint32_t s = propagate2(xs[i], ms ? ms[i] : RO_SUCCESS);
            bad |= s == 0xffu;
            if (s == RO_SUCCESS && mv[i] == 0) s = RO_SKIPPED;
            out[i] = (uint8_t)s;
        }
    }
    if (bad) raise_err(ctl, RO_ESTATE);
}

struct Maps {
    const uint32_t *m[kMaxBroadcastLevels];
    int64_t len[kMaxBroadcastLevels];       // entries of each map
};

__global__ __launch_bounds__(kBlock) void k_broadcast(Maps maps, int32_t levels, int64_t n,
                                                      const uint8_t *__restrict__ xs, int64_t n_anc,
                                                      const uint8_t *__restrict__ ls, uint32_t *__restrict__ anc,
                                                      uint8_t *__restrict__ out, Ctl *ctl)
{
    const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    int err = 0;
    for (int64_t d = g; d < n; d += stride) {
        uint32_t a = (uint32_t)d;
        bool in_range = true;
        for (int32_t l = 0; l < levels; ++l) {
            if ((int64_t)a >= maps.len[l]) {
                in_range = false;
                break;
            }
            a = maps.m[l][a];
        }
        if (!in_range || (int64_t)a >= n_anc) {
            err = RO_ERANGE;
            continue;
        }
        const uint32_t s = propagate2(xs[a], ls ? ls[d] : RO_SUCCESS);
        if (s == 0xffu) {
            err = RO_ESTATE;
            continue;
        }
        if (anc) anc[d] = a;
        out[d] = (uint8_t)s;
    }
    if (err) raise_err(ctl, err);
}

hipError_t launch_filter(const Launch &L, const uint8_t *xs, const uint8_t *ms, const uint8_t *mv, int64_t n,
                         uint8_t *out)
{
    const bool vec = ((reinterpret_cast<uintptr_t>(xs) | reinterpret_cast<uintptr_t>(ms) |
                       reinterpret_cast<uintptr_t>(mv) | reinterpret_cast<uintptr_t>(out)) & 15u) == 0;
    int64_t grid = (n + kBlock * 16 - 1) / (kBlock * 16);
    grid = grid < 1 ? 1 : (grid > (int64_t)L.num_cus * 8 ? (int64_t)L.num_cus * 8 : grid);
    RO_LAUNCH(L, RO_K_FILTER, k_filter, dim3((unsigned)grid), dim3(kBlock), 0, L.stream, xs, ms, mv, n, out,
              vec ? 1 : 0, L.ctl);
    return hipGetLastError();
}

hipError_t launch_broadcast(const Launch &L, const uint32_t *const *maps, const int64_t *map_len, int32_t levels,
                            int64_t n, const uint8_t *xs, int64_t n_anc, const uint8_t *ls, uint32_t *anc,
                            uint8_t *out)
{
    Maps m{};
    for (int32_t l = 0; l < levels; ++l) {
        m.m[l] = maps[l];
        m.len[l] = map_len[l];
    }
    int64_t grid = (n + kBlock - 1) / kBlock;
    grid = grid < 1 ? 1 : (grid > (int64_t)L.num_cus * 8 ? (int64_t)L.num_cus * 8 : grid);
    RO_LAUNCH(L, RO_K_BROADCAST, k_broadcast, dim3((unsigned)grid), dim3(kBlock), 0, L.stream, m, levels, n, xs, n_anc,
              ls, anc, out, L.ctl);
    return hipGetLastError();
}

}  // namespace ro
