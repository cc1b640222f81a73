"""Contexts and streams: two contexts on two streams run whole single-level
pipelines at the same time; a context re-bound to another stream; the
per-kernel trace."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

import workloads as W  # noqa: E402
import gpu_common as G  # noqa: E402


def test_two_contexts_two_streams_and_rebinding():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_18703_amd as R
    from paper_2609_18703_amd import pipeline as PL
    cases = [W.config2(n_parents=3_000, seed=s) for s in (11, 12)]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    ctxs, bufs = [], []
    for c, s in zip(cases, streams):
        with torch.cuda.stream(s):
            ctxs.append(R.Context())
            bufs.append(G.stage_single(c))
    torch.cuda.synchronize()
    try:
        for rep in range(3):
            for ctx, b, s in zip(ctxs, bufs, streams):          # both in flight at once
                with torch.cuda.stream(s):
                    PL.single_level(ctx, b)
            for ctx in ctxs:
                ctx.check(f"round {rep}")
            torch.cuda.synchronize()
            for c, b in zip(cases, bufs):
                G.compare_single(b, G.oracle_single(c))
        # the first context moves to the second's stream
        ctxs[0].set_stream(streams[1])
        with torch.cuda.stream(streams[1]):
            PL.single_level(ctxs[0], bufs[0])
        ctxs[0].check("rebound")
        torch.cuda.synchronize()
        G.compare_single(bufs[0], G.oracle_single(cases[0]))
    finally:
        for ctx in ctxs:
            ctx.close()


def test_kernel_trace_counts_launches():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_18703_amd as R
    from paper_2609_18703_amd import pipeline as PL
    c = W.config1()
    ctx = R.Context()
    try:
        b = G.stage_single(c)
        ctx.trace(True)
        for _ in range(3):
            PL.single_level(ctx, b)
        kern = ctx.trace_read()
        ctx.trace(False)
        ctx.check("trace")
        assert kern["expand_scan"][0] == 3 and kern["gather_copy"][0] == 3
        assert all(ms > 0 for _, ms in kern.values())
        assert ctx.trace_read() == {}                             # the read cleared the record
        G.compare_single(b, G.oracle_single(c))
    finally:
        ctx.close()
