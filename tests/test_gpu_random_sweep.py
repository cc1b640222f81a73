"""Randomized parity sweep over valid inputs: 160 seeded cases drawn from
five count shapes (small uniform, mostly empty, heavy-tailed Zipf, wide
uniform, one huge parent among tiny ones), each run through one of: the
FIFO batch with a random keep mask and B, the gather with partial reports,
pending states and random record lengths and alignments, the parent-bound
batch with a random barrier, or a stream over 1-11 waves of random sizes.
Every output is compared with the oracle bit for bit (the checks are the
ones of the dedicated tests, reused)."""
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

import oracle as O  # noqa: E402
import test_gpu_kernels as TK  # noqa: E402
import test_gpu_pbatch as TP  # noqa: E402
import test_gpu_stream_nested as TS  # noqa: E402


@pytest.fixture(scope="module")
def ctx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_18703_amd as R
    c = R.Context()
    yield c
    c.close()


def _counts(rng):
    kind = int(rng.integers(0, 5))
    P = int(rng.integers(0, 2000))
    if kind == 0:
        c = rng.integers(0, 4, P)
    elif kind == 1:
        c = np.where(rng.random(P) < 0.7, 0, rng.integers(1, 12, P))
    elif kind == 2:
        c = np.minimum(rng.zipf(1.3, P), 20000)
    elif kind == 3:
        c = rng.integers(0, 40, P)
    else:
        c = rng.integers(0, 3, P)
        if P:
            c[rng.integers(0, P)] = int(rng.integers(5000, 40000))
    return np.asarray(c, np.int32)


@pytest.mark.parametrize("block", range(8))
def test_random_sweep(ctx, block):
    for case in range(20):
        seed = 7_000 + block * 20 + case
        rng = np.random.default_rng(seed)
        counts = _counts(rng)
        what = int(rng.integers(0, 4))
        if what == 1 and int(counts.sum()) > 40_000:
            counts = np.minimum(counts, 20)
        offs = O.expand(counts, tags=False)
        N = int(offs[-1])
        print(f"sweep seed {seed}: P {len(counts)} N {N} test {what}", flush=True)
        sys.stdout.flush()
        ctx.reserve(N, len(counts), N)
        if what == 0 and N:
            Q = int(rng.integers(0, N + 1))
            q = rng.permutation(N)[:Q].astype(np.uint32)
            keep = None if rng.random() < 0.3 else (rng.random(Q) < rng.random()).astype(np.uint8)
            TK._batch_case(ctx, counts, q, keep, int(rng.integers(1, 3000)))
        elif what == 1:
            lens = [np.array([0, 1, 3, 16, 17, 100], np.int64), np.arange(0, 2000, 7, dtype=np.int64),
                    TK.LENS][int(rng.integers(0, 3))]
            states = [(0, 0, 0, 1, 2), (0, 1, 2, 3), (0,), (2, 2, 0)][int(rng.integers(0, 4))]
            par, ordi, st, off, data = TK._make_reports(rng, counts, float(rng.choice([1.0, 0.9, 0.5])), states,
                                                        lens)
            TK._gather_case(ctx, counts, par, ordi, st, off, data, extra_lead=int(rng.integers(0, 16)))
        elif what == 2 and N:
            Q = int(rng.integers(0, N + 1))
            q = rng.permutation(N)[:Q].astype(np.uint32)
            keep = None if rng.random() < 0.5 else (rng.random(Q) < 0.8).astype(np.uint8)
            bar = None if rng.random() < 0.5 else (rng.random(len(counts)) < 0.2).astype(np.uint8)
            TP._check(ctx, q, keep, offs, int(rng.integers(1, 600)), barrier=bar, what=f"seed {seed}")
        elif what == 3 and 0 < N <= 300_000:
            nw = int(rng.integers(1, 12))
            perm = rng.permutation(N)
            cuts = np.sort(rng.integers(0, N + 1, nw - 1))
            waves = []
            for ids in np.split(perm, cuts):
                st = rng.choice(np.array([0, 0, 0, 1, 2], np.uint8), len(ids))
                waves.append((ids.astype(np.uint32), st, rng.integers(0, 300, len(ids))))
            TS._stream_case(ctx, counts, waves, B=int(rng.integers(1, 2000)))
