// ro_expand_noalloc: F.expand for callers that cannot allocate device memory
// (code under stream capture, tight serving loops, harnesses that forbid
// hipMalloc).  The scan's workspace -- control words (ticket, completion
// count, look-back epoch, error word) and the look-back descriptors -- lives
// in one file-scope device array per GPU instead of a context.
#include <mutex>

#include "ro_device.h"

namespace ro {

// Workspace bound: expansions of up to kNoAllocMaxParents parents.
constexpr int64_t kNoAllocMaxParents = (int64_t)1 << 24;
constexpr int64_t kNoAllocDesc = kNoAllocMaxParents / kTile + 2;     // look-back descriptors
constexpr int64_t kNoAllocCtlBytes = 256;                            // Ctl, padded
static_assert(sizeof(Ctl) <= kNoAllocCtlBytes, "control words fit their slot");
constexpr int64_t kNoAllocWords = (kNoAllocCtlBytes + 8 * kNoAllocDesc) / 8;

// One copy per GPU, held until the process ends.  In host code this name is
// a host-side stand-in, never a device address: the device address comes
// from hipGetSymbolAddress, once per device.
static __device__ __align__(256) uint64_t scratch[kNoAllocWords];

// Start of a call: a clean error word; on a device's first call also the
// control words and every descriptor (the array's load-time contents are
// not relied on).
__global__ void k_noalloc_begin(uint64_t *ws, int first)
{
    Ctl *ctl = reinterpret_cast<Ctl *>(ws);
    uint64_t *desc = ws + kNoAllocCtlBytes / 8;
    if (first) {
        for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < kNoAllocDesc;
             i += (int64_t)gridDim.x * blockDim.x)
            desc[i] = 0;
        if (blockIdx.x == 0 && threadIdx.x == 0) {
            ctl->done = 0;
            ctl->ticket = 0;
            ctl->scan_epoch = 1;
        }
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) ctl->err = 0;
}

// End of a call: the first device-detected error (RO_OK if none).
__global__ void k_noalloc_end(uint64_t *ws, int32_t *status)
{
    if (threadIdx.x == 0 && status) *status = reinterpret_cast<Ctl *>(ws)->err;
}

namespace {

constexpr int kMaxDevices = 64;

struct NoAllocDevice {
    uint64_t *ptr = nullptr;     // device address of this GPU's copy of `scratch`
    int num_cus = 0;
    bool initialised = false;    // the begin kernel has cleared it once
};

std::mutex g_mu;
NoAllocDevice g_dev[kMaxDevices];

// The device address of the current GPU's workspace, looked up once per
// device with that device current.
int noalloc_device(NoAllocDevice **out)
{
    int d = 0;
    if (hipGetDevice(&d) != hipSuccess) return RO_EHIP;
    if (d < 0 || d >= kMaxDevices) return RO_EINVAL;
    std::lock_guard<std::mutex> lk(g_mu);
    NoAllocDevice &s = g_dev[d];
    if (s.ptr == nullptr) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return RO_EHIP;
        int cus = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, d) != hipSuccess) return RO_EHIP;
        s.ptr = static_cast<uint64_t *>(p);
        s.num_cus = cus > 0 ? cus : 1;
    }
    *out = &s;
    return RO_OK;
}

}  // namespace

}  // namespace ro

extern "C" int ro_expand_noalloc(void *hip_stream, const int32_t *counts, int64_t n_parents, int64_t *offsets,
                                 uint32_t *child_parent, uint32_t *child_ordinal, int64_t child_cap,
                                 int32_t *status_dev)
{
    using namespace ro;
    if (!offsets || n_parents < 0 || child_cap < 0 || (n_parents > 0 && !counts)) return RO_EINVAL;
    if (n_parents > kNoAllocMaxParents) return RO_ECAP;
    NoAllocDevice *dev = nullptr;
    const int rc = noalloc_device(&dev);
    if (rc != RO_OK) return rc;
    const hipStream_t stream = (hipStream_t)hip_stream;
    bool first;
    {
        std::lock_guard<std::mutex> lk(g_mu);
        first = !dev->initialised;
        dev->initialised = true;
    }
    hipLaunchKernelGGL(k_noalloc_begin, dim3(first ? 16 : 1), dim3(kBlock), 0, stream, dev->ptr, first ? 1 : 0);
    if (hipGetLastError() != hipSuccess) return RO_EHIP;
    Launch L;
    L.stream = stream;
    L.num_cus = dev->num_cus;
    L.ctl = reinterpret_cast<Ctl *>(dev->ptr);
    L.desc = dev->ptr + kNoAllocCtlBytes / 8;
    L.desc_cap = kNoAllocDesc;
    L.tracer = nullptr;
    if (launch_expand(L, counts, n_parents, offsets, child_parent, child_ordinal, child_cap) != hipSuccess)
        return RO_EHIP;
    hipLaunchKernelGGL(k_noalloc_end, dim3(1), dim3(64), 0, stream, dev->ptr, status_dev);
    return hipGetLastError() == hipSuccess ? RO_OK : RO_EHIP;
}
