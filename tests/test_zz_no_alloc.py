"""ro_expand_noalloc (no context, no device allocation) against ro_expand
through the C ABI: two calls in a row, the second smaller, bit-exact in
every output; the size limit; a device-detected error and a clean call
after it."""
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _counts(n, seed):
    rng = np.random.default_rng(seed)
    c = rng.integers(0, 60, n).astype(np.int32)
    c[rng.random(n) < 0.1] = 0          # empty parents
    return c


def _run_both(R, ctx, counts):
    dev = torch.from_numpy(counts).cuda()
    P = counts.size
    N = int(counts.astype(np.int64).sum())
    ref = [torch.full((P + 1,), -1, dtype=torch.int64, device="cuda"),
           torch.full((max(N, 1),), 7, dtype=torch.int32, device="cuda"),
           torch.full((max(N, 1),), 7, dtype=torch.int32, device="cuda")]
    got = [torch.full((P + 1,), -2, dtype=torch.int64, device="cuda"),
           torch.full((max(N, 1),), 9, dtype=torch.int32, device="cuda"),
           torch.full((max(N, 1),), 9, dtype=torch.int32, device="cuda")]
    status = torch.full((1,), 12345, dtype=torch.int32, device="cuda")
    ctx.expand(dev, *ref)
    ctx.check("ro_expand")
    R.expand_noalloc(dev, *got, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == R.OK
    for a, b in zip(ref, got):
        assert torch.equal(a, b)
    return N


def test_noalloc_matches_expand_twice():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_18703_amd as R
    ctx = R.Context()
    try:
        # several tiles and a ragged tail, then a smaller expansion that
        # leaves the first call's workspace contents behind
        for P, seed in ((3 * 4096 + 1234, 1), (517, 2)):
            _say(f"noalloc case P={P} seed={seed}")
            N = _run_both(R, ctx, _counts(P, seed))
            _say(f"  N={N} matches ro_expand")
    finally:
        ctx.close()


def test_noalloc_limits_and_errors():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import ctypes as C
    import paper_2609_18703_amd as R
    L = R.load()
    off = torch.empty(8, dtype=torch.int64, device="cuda")
    cnt = torch.zeros(7, dtype=torch.int32, device="cuda")
    # above the workspace bound: refused on the host, nothing launched
    _say("noalloc size limit")
    rc = L.ro_expand_noalloc(None, C.c_void_p(cnt.data_ptr()), R.EXPAND_NOALLOC_MAX_PARENTS + 1,
                             C.c_void_p(off.data_ptr()), None, None, 0, None)
    assert rc == R.ECAP
    rc = L.ro_expand_noalloc(None, C.c_void_p(cnt.data_ptr()), -1, C.c_void_p(off.data_ptr()), None, None, 0, None)
    assert rc == R.EINVAL
    # a negative count is found on the device and reported in the status
    _say("noalloc device error, then a clean call")
    bad = torch.tensor([3, -1, 2], dtype=torch.int32, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    R.expand_noalloc(bad, off[:4], status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == R.EINVAL
    good = torch.tensor([3, 0, 2], dtype=torch.int32, device="cuda")
    R.expand_noalloc(good, off[:4], status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == R.OK
    assert off[:4].cpu().tolist() == [0, 3, 3, 5]
    # more children than the tag arrays hold
    tags = torch.empty(4, dtype=torch.int32, device="cuda")
    R.expand_noalloc(good, off[:4], tags, tags.clone(), status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == R.ECAP
