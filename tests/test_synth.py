"""The synthetic workload generators (input generation, not the method):
shapes, ranges, sortedness, counter-based reproducibility, distributions."""
import math

import numpy as np
import pytest

import synth


@pytest.mark.parametrize("k", [1, 2, 3])
def test_whole_streams_have_the_promised_shape(k):
    w = synth.workload(k)
    src, dst, t, neg = synth.host_links(w)
    assert len(src) == w.links
    assert (np.diff(t.astype(np.int64)) >= 0).all()
    assert t.max() < 2**30
    if w.kind == 0:
        assert src.min() >= 0 and src.max() < w.n_src
        assert dst.min() >= w.n_src and dst.max() < w.num_nodes
        assert neg.min() >= w.n_src and neg.max() < w.num_nodes
        assert t.max() < w.T
    else:
        assert min(src.min(), dst.min(), neg.min()) >= 0
        assert max(src.max(), dst.max(), neg.max()) < w.num_nodes
        assert not (src == dst).any()


def test_repeats_reuse_prior_partners():
    w = synth.workload(2)
    src, dst, _, _ = synth.host_links(w)
    seen = {}
    reused = 0
    for u, v in zip(src[:200000], dst[:200000]):
        s = seen.setdefault(int(u), set())
        reused += int(v) in s
        s.add(int(v))
    assert reused / 200000 > 0.3


@pytest.mark.parametrize("k", [4, 5])
def test_counter_based_chunks_agree(k):
    w = synth.workload(k)
    a = synth.host_links(w, 1000, 5000)
    b = synth.host_links(w, 3000, 9000, threads=1)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x[2000:], y[:2000])


def test_pair_set_workload_mixes_reuse_and_fresh_pairs():
    w = synth.workload(4)
    src, dst, t, _ = synth.host_links(w, 0, 400000)
    assert not (src == dst).any() and t.max() < w.T
    key = src.astype(np.int64) * w.num_nodes + dst
    _, counts = np.unique(key, return_counts=True)
    # 80% of the links draw one of the 2M fixed pairs (with replacement), the
    # rest are fresh uniform pairs (almost surely unique)
    L, P = 400000, w.n_pairs
    expect = P * (1 - math.exp(-w.p_pair * L / P)) + (1 - w.p_pair) * L
    assert abs(len(counts) - expect) < 0.01 * expect


def test_zipf_alias_matches_weights():
    n, a = 1000, 1.2
    prob, alias = synth.alias_table(n, a)
    w = (np.arange(1, n + 1, dtype=np.float64)) ** -a
    w /= w.sum()
    # exact distribution implied by the table
    implied = prob.astype(np.float64) / 2**32 / n
    np.add.at(implied, alias, (1 - prob.astype(np.float64) / 2**32) / n)
    assert np.abs(implied - w).max() < 1e-9


def test_bipartite_popularity_is_zipf():
    w = synth.workload(1)
    src, dst, _, _ = synth.host_links(w)
    counts = np.sort(np.bincount(src, minlength=w.n_src))[::-1]
    p = np.arange(1, w.n_src + 1, dtype=np.float64) ** -w.exponent
    p /= p.sum()
    assert abs(counts[0] / len(src) - p[0]) < 5 * math.sqrt(p[0] / len(src))


def test_feature_rows_are_standard_normal_and_reproducible():
    w = synth.workload(3)
    rows = np.arange(0, 200000, 7)
    a = synth.host_feature_rows(w, "edge", rows)
    b = synth.host_feature_rows(w, "edge", rows[::-1])[::-1]
    np.testing.assert_array_equal(a, b)
    import torch
    v = torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).float().numpy()
    assert abs(v.mean()) < 0.01 and abs(v.std() - 1.0) < 0.01
    w1 = synth.workload(1)
    f = synth.host_feature_rows(w1, "edge", np.arange(1000))
    assert f.dtype == np.float32 and abs(f.std() - 1) < 0.02


def test_blocked_layout():
    w = synth.scaled(synth.workload(1), 1050)     # ragged last batch of 50
    src, dst, t, neg = synth.host_links(w)
    nodes, ts = synth.blocked(w, src, dst, t, neg)
    for b in range(w.batches):
        s_, d_, t_, q, tq = synth.batch_views(w, nodes, ts, b)
        lo, hi = w.batch_range(b)
        np.testing.assert_array_equal(s_, src[lo:hi])
        np.testing.assert_array_equal(d_, dst[lo:hi])
        np.testing.assert_array_equal(q[2 * (hi - lo):], neg[lo:hi])
        np.testing.assert_array_equal(tq, np.concatenate([t[lo:hi]] * 3))


def test_time_params():
    f, p = synth.time_params(synth.workload(1))
    assert f.dtype == np.float32 and len(f) == 100 and f[0] == 1.0
    assert abs(f[-1] - 1e-9) < 1e-15 and (np.diff(f) < 0).all()
    assert (p >= -np.pi).all() and (p < np.pi).all()
