// Per-Call FIFO Ready Queue with elastic reservation on gfx950.
//
// RayOrch (arXiv 2609.18703), Sec. 4 "Scheduling Ready Grains": ready Grains
// sit in one FIFO queue in enqueue order; each elastic reservation removes at
// most B entries from the head and may mix parents.  Taking the reservations
// one after another until the queue is empty is a stable compaction of the
// ready entries cut into consecutive chunks of B, which is what this kernel
// computes in one pass: ballot ranks inside a wave, a workgroup scan, and a
// decoupled look-back across tiles keep every ready entry in queue order.
#include "ro_device.h"

namespace ro {

// Samples of the offsets array: samp[j] = offsets[min(j << shift, P)].
__global__ void k_batch_samples(const int64_t *__restrict__ offsets, int64_t P, int shift,
                                int64_t nsamp, int64_t *__restrict__ samp)
{
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (j < nsamp) {
        const int64_t i = j << shift;
        samp[j] = offsets[i < P ? i : P];
    }
}

// Parent of child c: the LDS samples narrow the search to 2^shift offsets,
// a short global binary search finishes it.
__device__ __forceinline__ int64_t find_parent(const int64_t *s_samp, int64_t nsamp, int shift,
                                               const int64_t *offsets, int64_t P, int64_t c)
{
    int64_t lo = 0, hi = nsamp;
    while (lo < hi) {
        int64_t mid = (lo + hi) >> 1;
        if (s_samp[mid] <= c) lo = mid + 1; else hi = mid;
    }
    const int64_t j = lo - 1;                    // s_samp[0] = 0 <= c
    const int64_t b = j << shift;
    int64_t e = b + ((int64_t)1 << shift);
    e = e < P + 1 ? e : P + 1;
    return upper_bound_g(offsets, b, e, c) - 1;
}

__global__ __launch_bounds__(kBlock) void k_batch(
    const uint32_t *__restrict__ queue, const uint8_t *__restrict__ keep, int64_t Q,
    const int64_t *__restrict__ offsets, int64_t P, const int64_t *__restrict__ samp, int64_t nsamp,
    int shift, int32_t B, uint32_t *__restrict__ out_child, uint32_t *__restrict__ out_parent,
    uint32_t *__restrict__ out_ordinal, int64_t out_cap, int64_t *n_out, int64_t *n_batches,
    Ctl *ctl, uint64_t *desc, int64_t desc_cap, int64_t ntiles, int vec_ok)
{
    const uint32_t epoch = scan_epoch(ctl);
    __shared__ int64_t s_samp[kMaxSamples];
    __shared__ int64_t s_wave[kBlock / 64];
    __shared__ uint64_t s_b;
    __shared__ int64_t s_t;
    __shared__ int32_t s_last;
    for (int64_t j = threadIdx.x; j < nsamp; j += kBlock) s_samp[j] = samp[j];
    __syncthreads();
    const int64_t N = offsets[P];
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
        const int64_t cnt = __popc(kmask);
        int64_t tot;
        const int64_t ex = block_excl_scan(cnt, s_wave, tot);
        const uint64_t pre = tile_prefix(desc, t, epoch, (uint64_t)tot, &s_b, ctl);
        int64_t slot = (int64_t)pre + ex;
        bool bad_range = false, bad_cap = false;
#pragma unroll
        for (int k = 0; k < kItems; ++k) {
            if (!(kmask & (1u << k))) continue;
            const int64_t c = q[k];
            uint32_t p = 0xffffffffu, o = 0xffffffffu;
            if (c >= N) {
                bad_range = true;
            } else if (want_tags) {
                const int64_t pp = find_parent(s_samp, nsamp, shift, offsets, P, c);
                p = (uint32_t)pp;
                o = (uint32_t)(c - offsets[pp]);
            }
            if (slot < out_cap) {
                if (out_child) out_child[slot] = (uint32_t)c;
                if (out_parent) out_parent[slot] = p;
                if (out_ordinal) out_ordinal[slot] = o;
            } else {
                bad_cap = true;
            }
            ++slot;
        }
        if (bad_range) raise_err(ctl, RO_ERANGE);
        if (bad_cap) raise_err(ctl, RO_ECAP);
        if (t == ntiles - 1 && threadIdx.x == 0) {
            const int64_t m = (int64_t)pre + tot;
            if (n_out) *n_out = m;
            if (n_batches) *n_batches = (m + B - 1) / B;
        }
    }
    ticket_done(ctl, epoch, desc, desc_cap, &s_last);
}

hipError_t launch_batch(const Launch &L, const uint32_t *queue, const uint8_t *keep,
                        int64_t Q, const int64_t *offsets, int64_t P, int32_t B,
                        uint32_t *out_child, uint32_t *out_parent, uint32_t *out_ordinal,
                        int64_t out_cap, int64_t *n_out, int64_t *n_batches, int64_t *samples)
{
    int shift = 0;
    while ((((P + 1) + ((int64_t)1 << shift) - 1) >> shift) > kMaxSamples) ++shift;
    const int64_t nsamp = ((P + 1) + ((int64_t)1 << shift) - 1) >> shift;
    RO_LAUNCH(L, RO_K_BATCH_SAMPLES, k_batch_samples, dim3((unsigned)((nsamp + 255) / 256)), dim3(256), 0, L.stream,
                       offsets, P, shift, nsamp, samples);
    const int64_t ntiles = Q > 0 ? (Q + kTile - 1) / kTile : 1;
    const int64_t cap_grid = (int64_t)L.num_cus * 4;
    const int64_t grid = ntiles < cap_grid ? ntiles : cap_grid;
    const bool aligned = ((reinterpret_cast<uintptr_t>(queue) | reinterpret_cast<uintptr_t>(keep)) & 15u) == 0;
    RO_LAUNCH(L, RO_K_BATCH, k_batch, dim3((unsigned)grid), dim3(kBlock), 0, L.stream, queue, keep, Q, offsets,
                       P, samples, nsamp, shift, B, out_child, out_parent, out_ordinal, out_cap, n_out,
                       n_batches, L.ctl, L.desc, L.desc_cap, ntiles, aligned ? 1 : 0);
    return hipGetLastError();
}

}  // namespace ro
