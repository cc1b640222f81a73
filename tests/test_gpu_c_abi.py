"""The library from plain C: tests/c_abi_driver.c (built by
__graft_entry__.build()) allocates with the HIP runtime, runs expand, batch
and gather through the C ABI on seeded cases and compares every output with
the C oracle; one case plants an out-of-range ordinal and expects RO_ERANGE
from ro_ctx_status, and the context is used again afterwards."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_c_abi_from_plain_c():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    exe = os.path.join(ROOT, "tests", "c_abi_driver")
    if not os.path.exists(exe):
        pytest.fail("tests/c_abi_driver is missing: build it with __graft_entry__.build()")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=110)
    print(r.stdout, flush=True)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.strip().splitlines()[-1] == "c abi ok"
