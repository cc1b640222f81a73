// Device-side record fill for the synthetic workloads (generator side; not
// part of the expand/batch/gather library).  Record r is the little-endian
// byte stream of splitmix64 (Steele, Lea and Flood, OOPSLA 2014) started from
// seeds[r], truncated to off[r+1] - off[r] bytes, written at data + off[r].
#include <hip/hip_runtime.h>
#include <stdint.h>

__device__ __forceinline__ uint64_t sm64_output(uint64_t seed, uint64_t k)
{
    uint64_t z = seed + (k + 1) * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// One wave per record, one 8-byte output word per lane.
__global__ void k_fill(const uint64_t *__restrict__ seeds, const int64_t *__restrict__ off, int64_t n,
                       uint8_t *__restrict__ data)
{
    const int lane = threadIdx.x & 63;
    const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
    for (int64_t r = wave; r < n; r += nwaves) {
        const int64_t o0 = off[r];
        const int64_t len = off[r + 1] - o0;
        const uint64_t seed = seeds[r];
        for (int64_t k = lane; k * 8 < len; k += 64) {
            const uint64_t z = sm64_output(seed, (uint64_t)k);
            const int64_t b0 = k * 8;
            uint8_t *dst = data + o0 + b0;
            if (b0 + 8 <= len && (((uintptr_t)dst) & 7) == 0) {
                *reinterpret_cast<uint64_t *>(dst) = z;
            } else {
#pragma unroll
                for (int b = 0; b < 8; ++b)
                    if (b0 + b < len) dst[b] = (uint8_t)(z >> (8 * b));
            }
        }
    }
}

extern "C" int synth_fill_records(const uint64_t *seeds, const int64_t *off, int64_t n, uint8_t *data,
                                  void *stream)
{
    if (n <= 0) return 0;
    int64_t blocks = (n + 3) / 4;
    if (blocks > 65536) blocks = 65536;
    hipLaunchKernelGGL(k_fill, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, seeds, off, n,
                       data);
    return hipGetLastError() == hipSuccess ? 0 : -7;
}
