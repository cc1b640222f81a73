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


def test_binding_rejects_wrong_element_size_and_short_arrays():
    """The C calls see bare pointers, so the binding checks element sizes and
    lengths before anything is launched; nothing reaches the device here."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_18703_amd as R
    ctx = R.Context()
    dev = "cuda"
    try:
        offs = torch.zeros(11, dtype=torch.int64, device=dev)
        with pytest.raises(TypeError):
            ctx.expand(torch.ones(10, dtype=torch.int64, device=dev), offs)       # counts are int32
        with pytest.raises(ValueError):
            ctx.expand(torch.ones(10, dtype=torch.int32, device=dev), offs[:10])  # offsets need P + 1
        with pytest.raises(TypeError):
            ctx.expand(torch.ones(10, dtype=torch.int32, device=dev), offs.to(torch.int32))
        q = torch.zeros(8, dtype=torch.int32, device=dev)
        tag = torch.zeros(4, dtype=torch.int32, device=dev)
        with pytest.raises(ValueError):
            ctx.batch(q, None, offs, 2, tag, q_len=8, out_cap=8)                     # out_child too short
        with pytest.raises(ValueError):
            ctx.batch(q, torch.ones(4, dtype=torch.uint8, device=dev), offs, 2, q)  # keep too short
        with pytest.raises(ValueError):
            ctx.batch(q, None, offs, 2, q, barrier=torch.zeros(3, dtype=torch.uint8, device=dev))
        par = torch.zeros(5, dtype=torch.int32, device=dev)
        st = torch.zeros(5, dtype=torch.uint8, device=dev)
        off = torch.zeros(6, dtype=torch.int64, device=dev)
        data = torch.zeros(16, dtype=torch.uint8, device=dev)
        out_off = torch.zeros(11, dtype=torch.int64, device=dev)
        with pytest.raises(ValueError):
            ctx.gather(par, par, st, off[:5], data, offs, out_off)                   # report offsets need n + 1
        with pytest.raises(TypeError):
            ctx.gather(par, par, st.to(torch.int32), off, data, offs, out_off)      # states are bytes
        with pytest.raises(ValueError):
            ctx.gather(par, par, st, off, data, offs, out_off[:10])                 # out_off needs P + 1
        with pytest.raises(ValueError):
            ctx.gather(par, par, st, off, data, offs, out_off, data, out_cap=32)    # out_data under out_cap
        with pytest.raises(ValueError):
            ctx.filter(st, st[:4], st)
        with pytest.raises(ValueError):
            ctx.gather(par, par, st, off, data, offs.cpu(), out_off)                # host memory
        ctx.check("nothing launched")
    finally:
        ctx.close()
