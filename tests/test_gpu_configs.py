"""GPU parity on the synthetic workloads: whole chains vs the oracle."""
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

import oracle as O  # noqa: E402
import workloads as W  # noqa: E402
from workloads import device as D  # noqa: E402
import gpu_common as G  # noqa: E402


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def ctx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_18703_amd as R
    c = R.Context()
    yield c
    c.close()


def _single(ctx, c):
    from paper_2609_18703_amd import pipeline as PL
    b = G.stage_single(c)
    ctx.reserve(c.n_children, c.n_parents, c.n_children)
    PL.single_level(ctx, b)
    ctx.check("single level")
    want = G.oracle_single(c)
    G.compare_single(b, want)
    return b


def test_config1_full(ctx):
    _say("config1 full")
    _single(ctx, W.config1())


def test_config1_canonical_order(ctx):
    _single(ctx, W.config1(canonical_order=True))


@pytest.mark.parametrize("P", [700, 5000])
def test_config2_scaled(ctx, P):
    _say("config2 P", P)
    _single(ctx, W.config2(n_parents=P))


def test_config2_twice_same_context(ctx):
    """Back-to-back runs of the whole chain on one context agree."""
    from paper_2609_18703_amd import pipeline as PL
    c = W.config2(n_parents=1200)
    b = G.stage_single(c)
    ctx.reserve(c.n_children, c.n_parents, c.n_children)
    PL.single_level(ctx, b)
    first = b.out_data.clone(), b.out_off.clone()
    PL.single_level(ctx, b)
    ctx.check("twice")
    assert torch.equal(first[0], b.out_data) and torch.equal(first[1], b.out_off)
