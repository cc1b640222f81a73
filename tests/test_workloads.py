"""The seeded generators: content stream and distribution readings."""
import numpy as np

import workloads as W


def test_splitmix64_published_outputs():
    # first outputs of splitmix64 started from state 0, as published with
    # the generator's reference implementation
    w = W.splitmix64_words(np.zeros(3, np.uint64), np.arange(3))
    assert [int(x) for x in w] == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


def test_record_bytes_truncate_little_endian():
    seeds = np.array([5, 5, 9], np.uint64)
    b = W.record_bytes(seeds, [3, 11, 0])
    w0 = int(W.splitmix64_words(np.uint64(5), np.uint64(0)))
    w1 = int(W.splitmix64_words(np.uint64(5), np.uint64(1)))
    full = w0.to_bytes(8, "little") + w1.to_bytes(8, "little")
    assert bytes(b) == full[:3] + full[:11]


def test_configs_deterministic_and_shaped():
    a = W.config1()
    b = W.config1()
    assert np.array_equal(a.counts, b.counts) and np.array_equal(a.queue, b.queue)
    assert a.n_parents == 1000 and a.counts.min() >= 1 and a.counts.max() <= 500
    assert np.all(a.lengths == 64)
    c = W.config2(n_parents=5000)
    assert c.counts.min() >= 1 and c.counts.max() <= 10_000
    assert c.lengths.min() >= 16 and c.lengths.max() <= 4096
    # sealed children are exactly the SKIPPED ones; reports hold every child once
    assert np.array_equal(c.keep == 0, c.states[c.queue] == W.SKIPPED)
    assert np.array_equal(np.sort(c.reports.child), np.arange(c.n_children))
    assert np.all(np.diff(c.reports.off) == np.where(c.reports.state == W.SUCCESS,
                                                      c.lengths[c.reports.child], 0))


def test_rank_zipf_sums_exactly():
    rng = np.random.default_rng(0)
    k = W.rank_zipf_counts(rng, 20_000, 400_000, 1.1, 1, 4000)
    assert k.sum() == 400_000 and k.min() >= 1 and k.max() <= 4000


def test_streaming_waves_partition_children():
    s = W.config5(n_parents=2000, n_children=30_000, n_waves=7)
    allc = np.concatenate(s.waves)
    assert np.array_equal(np.sort(allc), np.arange(30_000))
    assert s.wave_reports[0].off[0] == 0
    for a, b in zip(s.wave_reports[:-1], s.wave_reports[1:]):
        assert a.off[-1] == b.off[0]
