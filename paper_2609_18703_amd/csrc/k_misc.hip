// Context bookkeeping kernels: control-word initialisation, epoch resets and
// fills.  (The look-back epoch wraps on the device: see ticket_done_n.)
#include "ro_device.h"

namespace ro {

__global__ void k_ctl_init(Ctl *ctl)
{
    if (threadIdx.x == 0) ctl->scan_epoch = 1;
}

// Clears the error word (after the host has read it), in stream order.
__global__ void k_clear_err(Ctl *ctl)
{
    if (threadIdx.x == 0) ctl->err = 0;
}

// Zero-fill (a kernel, so that a captured graph holds no memset node).
__global__ void k_fill_u64(uint64_t *p, int64_t n)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = 0;
}

// Clears canonical slot tags: a context's when its canonical epoch wraps, a
// stream's when its run epoch wraps.
__global__ void k_clear_tags(Canon *canon, int64_t n)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        canon[i].tag = 0;
}

hipError_t launch_zero_u64(const Launch &L, uint64_t *p, int64_t n)
{
    RO_LAUNCH(L, RO_K_MISC, k_fill_u64, dim3((unsigned)L.num_cus * 4), dim3(256), 0, L.stream, p, n);
    return hipGetLastError();
}

hipError_t launch_clear_tags(const Launch &L, Canon *canon, int64_t n)
{
    RO_LAUNCH(L, RO_K_MISC, k_clear_tags, dim3((unsigned)L.num_cus * 4), dim3(256), 0, L.stream, canon, n);
    return hipGetLastError();
}

hipError_t launch_ctl_init(const Launch &L)
{
    RO_LAUNCH(L, RO_K_MISC, k_ctl_init, dim3(1), dim3(64), 0, L.stream, L.ctl);
    return hipGetLastError();
}

hipError_t launch_clear_err(const Launch &L)
{
    RO_LAUNCH(L, RO_K_MISC, k_clear_err, dim3(1), dim3(64), 0, L.stream, L.ctl);
    return hipGetLastError();
}

}  // namespace ro
