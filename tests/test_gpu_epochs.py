"""The look-back descriptors carry a 16-bit launch epoch that wraps after
65,535 ticketed launches (every descriptor is cleared first).  This runs a
context through more than one wrap and checks every scan around it against
the oracle."""
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

import oracle as O  # noqa: E402
from workloads import device as D  # noqa: E402


def test_scan_epoch_wrap():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_18703_amd as R
    ctx = R.Context()
    try:
        rng = np.random.default_rng(3)
        inputs = []
        for k in range(3):
            counts = rng.integers(0, 50, 20_000 + 7_000 * k).astype(np.int32)   # 5 to 10 tiles
            inputs.append((D.to_dev(counts), O.expand(counts, tags=False)))
        outs = [torch.empty(len(w) + 0, dtype=torch.int64, device="cuda") for _, w in inputs]
        n_calls = 66_500
        print("ticketed launches:", n_calls, flush=True)
        for i in range(n_calls):
            j = i % 3
            ctx.expand(inputs[j][0], outs[j])
            near = 65_400 <= i <= 65_700
            if near or i % 5_000 == 4_999:
                ctx.check(f"call {i}")
                assert np.array_equal(outs[j].cpu().numpy(), inputs[j][1]), i
                outs[j].fill_(-1)
        ctx.check("end")
        print("ok", flush=True)
        sys.stdout.flush()
    finally:
        ctx.close()
