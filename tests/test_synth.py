"""The seeded input generator: deterministic, prefix-consistent, and drawing
from the distributions it states."""
import numpy as np

import synth
from synth import workloads


def test_streams_are_seeded_and_prefix_consistent():
    a, ca = synth.workload_streams(2, L=3000, B=8)
    b, _ = synth.workload_streams(2, L=3000, B=8)
    c, _ = synth.workload_streams(2, L=1000, B=4)
    assert np.array_equal(a, b)
    assert np.array_equal(a[:4, :1000], c)
    assert a.dtype == np.uint8 and a.shape == (8, 3000)


def test_zipf_table_entropy():
    for s, H in ((1.1, 5.7664), (1.2, 5.2898)):
        q = synth.cdf_probs(synth.zipf_table(s, 7))
        assert abs(-(q * np.log2(q)).sum() - H) < 1e-3


def test_markov_rows_are_distributions_and_sampling_matches_them():
    cdf = synth.markov_table(1, 0.5, 11)
    q = synth.cdf_probs(cdf)
    assert q.shape == (256, 256)
    np.testing.assert_allclose(q.sum(1), 1.0, rtol=1e-6)
    s, _ = synth.generate([(synth.SRC_MARKOV, 1, cdf)], np.zeros((64, 1), np.int32), 1 << 14, 1 << 14,
                          np.arange(1, 65, dtype=np.uint64))
    prev, nxt = s[:, :-1].ravel(), s[:, 1:].ravel()
    row = 17
    sel = nxt[prev == row]
    emp = np.bincount(sel, minlength=256) / sel.size
    assert np.abs(emp - q[row]).sum() < 0.25


def test_runs_have_geometric_mean_64():
    s, bits = synth.generate([(synth.SRC_RUNS, 0, None)], np.zeros((16, 1), np.int32), 1 << 16, 1 << 16,
                             np.arange(1, 17, dtype=np.uint64))
    changes = (s[:, 1:] != s[:, :-1]).sum()
    mean_run = s.size / (changes + 16)
    assert 55 < mean_run < 75
    assert 0 < bits.mean() / s.shape[1] < 0.5


def test_workload_shapes_and_mix():
    w3 = workloads.WORKLOADS[3]
    assert (w3.T, w3.d) == (8, 256)
    s, bits = synth.workload_streams(3, L=2048, B=6)
    per = bits / 2048
    assert abs(per[2] - 8.0) < 1e-12 and abs(per[5] - 8.0) < 1e-12       # uniform streams
    assert per[0] < 6.0 and 4.5 < per[1] < 6.0                            # markov, zipf
    s4, _ = synth.workload_streams(4, L=4096, B=4)
    assert s4.shape == (4, 4096)
    s5, b5 = synth.workload_streams(5, L=1024, B=16)
    assert s5.shape == (16, 1024) and np.all(np.isfinite(b5))
