"""Stage generated workloads in GPU memory (generator side).

Uploads the seeded arrays as torch tensors and fills the record bytes, either
from the host copy (small workloads) or with the device splitmix64 fill in
``libsynth.so`` (large ones).  Nothing here runs a step of the method.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SYNTH_SRC = os.path.join(HERE, "synth.hip")
SYNTH_LIB = os.path.join(HERE, "libsynth.so")

_synth = None


def build_synth():
    cmd = ["/opt/rocm/bin/hipcc", "--offload-arch=gfx950", "-O3", "-fPIC", "-shared",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-o", SYNTH_LIB + ".tmp", SYNTH_SRC]
    subprocess.run(cmd, check=True, capture_output=True)
    os.replace(SYNTH_LIB + ".tmp", SYNTH_LIB)
    return SYNTH_LIB


def synth():
    global _synth
    if _synth is None:
        if not os.path.exists(SYNTH_LIB):
            raise RuntimeError(f"{SYNTH_LIB} missing: run workloads.device.build_synth()")
        L = C.CDLL(SYNTH_LIB)
        L.synth_fill_records.argtypes = [C.c_void_p, C.c_void_p, C.c_int64, C.c_void_p, C.c_void_p]
        L.synth_fill_records.restype = C.c_int
        _synth = L
    return _synth


def to_dev(a, dtype=None):
    import torch
    a = np.ascontiguousarray(a)
    if not a.flags.writeable:          # torch.from_numpy wants a writable array
        a = a.copy()
    t = torch.from_numpy(a)
    if dtype is not None:
        t = t.to(dtype)
    return t.cuda()


def fill_records_dev(seeds, off, data, stream=None):
    """Fill data[off[r]:off[r+1]] with splitmix64(seeds[r]) bytes on the GPU."""
    import torch
    stream = stream or torch.cuda.current_stream()
    n = seeds.numel()
    rc = synth().synth_fill_records(C.c_void_p(seeds.data_ptr()), C.c_void_p(off.data_ptr()), n,
                                    C.c_void_p(data.data_ptr()), C.c_void_p(stream.cuda_stream))
    if rc != 0:
        raise RuntimeError(f"synth fill failed: {rc}")


def reports_data_dev(rep, host_limit=64 << 20):
    """Device bytes of a Reports layout (host generation when small)."""
    import torch
    total = int(rep.off[-1])
    if total - rep.base <= host_limit:
        host = np.zeros(total, np.uint8)
        host[rep.base:] = rep.data()
        return to_dev(host)
    data = torch.empty(max(total, 1), dtype=torch.uint8, device="cuda")
    fill_records_dev(to_dev(rep.seed), to_dev(rep.off), data)
    return data
