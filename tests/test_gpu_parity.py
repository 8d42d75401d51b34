"""GPU library vs CPU oracle, element by element, on seeded workloads.

Indices, timestamps, arrival indices and feature rows must be bit-exact;
the fp32 time encoding must be within 1e-5 absolute.
"""
import numpy as np
import pytest

import oracle
import synth
from tests.gpu_helpers import (compare_sample, compare_tables, feat_to_dev, make_gpu_table,
                               make_oracle, to_dev, u32)

pytestmark = pytest.mark.gpu

ALL = ("nbr", "eid", "ts", "tenc", "efeat", "nfeat", "self")


def _run_stream(w, full_batches, index_batches="all", check_every=None):
    """Drive GPU and oracle over workload w; compare the sample outputs of
    `full_batches` fully, the indices of `index_batches`, and the tables at
    the end (and every `check_every` batches)."""
    import torch
    src, dst, t, neg = synth.host_links(w)
    nodes, ts = synth.blocked(w, src, dst, t, neg)
    nodes_d, ts_d = to_dev(nodes), to_dev(ts)
    ef = synth.host_features(w, "edge") if w.edge_dim else None
    nf = synth.host_features(w, "node") if w.node_dim else None
    ef_d = feat_to_dev(ef, w.edge_dtype) if ef is not None else None
    nf_d = feat_to_dev(nf, w.node_dtype) if nf is not None else None
    g = make_gpu_table(w, ef_d, nf_d)
    o = make_oracle(w)
    fw, fb = synth.time_params(w)
    full = set(full_batches)
    checked = 0
    for b in range(w.batches):
        s_, d_, t_, q, tq = synth.batch_views(w, nodes_d, ts_d, b)
        lo, hi = w.batch_range(b)
        qh = np.concatenate([src[lo:hi], dst[lo:hi], neg[lo:hi]])
        tqh = np.concatenate([t[lo:hi]] * 3)
        if b in full:
            gout = g.sample(q, tq)
            oout = o.sample(qh, tqh, fw, fb, ef, nf)
            compare_sample(gout, oout, f"batch {b}")
            checked += 1
        elif index_batches == "all" or b in index_batches:
            gout = g.sample(q, tq, want=("nbr", "eid", "ts"))
            oout = o.sample(qh, tqh, want=("nbr", "eid", "ts"))
            compare_sample(gout, oout, f"batch {b}")
        g.insert(s_, d_, t_)
        o.insert(src[lo:hi], dst[lo:hi], t[lo:hi])
        if check_every and (b + 1) % check_every == 0:
            compare_tables(g, o)
    torch.cuda.synchronize()
    assert g.status() == 0
    compare_tables(g, o)
    assert g.info()["interactions"] == w.links
    return checked


def test_tiny_bipartite_full_stream():
    """Workload 1 at full size: every batch's outputs and the final table."""
    w = synth.workload(1)
    assert _run_stream(w, full_batches=range(w.batches), check_every=25) == w.batches


def test_small_bipartite_full_stream():
    """Workload 2 at full size: indices of every batch, all outputs on a
    subset of batches (first 5, every 97th, last 5), tables at checkpoints."""
    w = synth.workload(2)
    nb = w.batches
    full = set(range(5)) | set(range(0, nb, 97)) | set(range(nb - 5, nb))
    _run_stream(w, full_batches=full, check_every=300)


def test_medium_homogeneous_prefix():
    """Workload 3 shape (s=64, alpha=0.3, bf16 edge+node rows) on its first
    120 batches: tables at checkpoints and full outputs of some batches."""
    w = synth.scaled(synth.workload(3), 120 * 4000)
    _run_stream(w, full_batches={0, 1, 50, 119}, index_batches={10, 60, 100}, check_every=40)


def test_dense_repeated_prefix():
    """Workload 4 shape (bf16 186-dim edge rows = 372 B, 4-byte copy path)."""
    w = synth.scaled(synth.workload(4), 60 * 10000)
    _run_stream(w, full_batches={0, 30, 59}, index_batches={10, 20, 40, 50}, check_every=20)


def test_time_encoding_launch_paths_agree():
    """A large first-hop launch that also writes timestamps computes the time
    encoding in a separate streaming kernel; without the timestamp output
    (or in a small launch) sample_gather computes it.  Both paths give
    bit-identical values, and both match the oracle within 1e-5."""
    import torch
    w = synth.scaled(synth.workload(4), 20 * 10000)
    src, dst, t, neg = synth.host_links(w)
    g = make_gpu_table(w)
    g.insert(to_dev(src), to_dev(dst), to_dev(t))
    o = make_oracle(w)
    o.insert(src, dst, t)
    rng = np.random.default_rng(8)
    for nq in (30000, 500):                   # 7.5M and 125k float4 outputs
        q = np.concatenate([src, dst])[rng.integers(0, 2 * len(src), nq)].astype(np.int32)
        tq = rng.integers(0, int(t[-1]) + 2, nq).astype(np.uint32)
        a = g.sample(to_dev(q), to_dev(tq), want=("nbr", "eid", "ts", "tenc"))
        b = g.sample(to_dev(q), to_dev(tq), want=("tenc",))
        assert torch.equal(a["tenc"], b["tenc"]), nq
        fw, fb = synth.time_params(w)
        oo = o.sample(q[:400], tq[:400], fw, fb, None, None, want=("nbr", "ts", "tenc"))
        compare_sample({"nbr": a["nbr"][:400], "ts": a["ts"][:400], "tenc": a["tenc"][:400]},
                       {"nbr": oo["nbr"], "ts": oo["ts"], "tenc": oo["tenc"]}, f"nq={nq}")


def test_time_encoding_wide_arguments():
    """Frequencies scaled by 10^4 put w dt + b far beyond 2^33 for most
    slots, outside the fast cosine's range: both time-encoding launch paths
    of nlb_sample stay bit-identical and match the oracle within 1e-5, and
    the aggregation (whose per-query kernel then takes its general-cosine
    branch) matches the oracle within its tolerance."""
    import torch
    import paper_2402_01964_amd as nlb
    for k in (4, 1):
        base = synth.workload(k)
        w = synth.scaled(base, 20 * base.batch)
        src, dst, t, neg = synth.host_links(w)
        fw, fb = synth.time_params(w)
        fw = (fw * 1.0e4).astype(np.float32)
        ef = synth.host_features(w, "edge") if w.edge_dim else None
        g = nlb.Table(w.num_nodes, w.s, w.alpha, w.table_seed, time_w=to_dev(fw), time_b=to_dev(fb),
                      edge_feat=feat_to_dev(ef, w.edge_dtype) if ef is not None else None)
        g.insert(to_dev(src), to_dev(dst), to_dev(t))
        o = make_oracle(w)
        o.insert(src, dst, t)
        rng = np.random.default_rng(9 + k)
        ends = np.concatenate([src, dst])
        for nq in (30000, 500):
            q = ends[rng.integers(0, len(ends), nq)].astype(np.int32)
            tq = rng.integers(0, int(t[-1]) + 2, nq).astype(np.uint32)
            a = g.sample(to_dev(q), to_dev(tq), want=("nbr", "eid", "ts", "tenc"))
            b = g.sample(to_dev(q), to_dev(tq), want=("tenc",))
            assert torch.equal(a["tenc"], b["tenc"]), (k, nq)
            oo = o.sample(q[:400], tq[:400], fw, fb, None, None, want=("nbr", "ts", "tenc"))
            compare_sample({"nbr": a["nbr"][:400], "ts": a["ts"][:400], "tenc": a["tenc"][:400]},
                           {"nbr": oo["nbr"], "ts": oo["ts"], "tenc": oo["tenc"]}, f"wide k={k} nq={nq}")
            W = synth.agg_weights(w)
            gz = g.aggregate(to_dev(q), to_dev(tq), _agg_dev(W)).cpu().numpy()
            oz = o.aggregate(q[:400], tq[:400], fw, fb, ef, None, W)
            err = agg_error(gz[:400], oz)
            print(f"aggregate wide arguments, workload {k}, {nq} queries: max scaled error {err:.3e}")
            assert err <= AGG_TOL
        assert g.status() == 0


# ----------------------------------------------------------------------------- invariance
def _insert_in_batches(w, src, dst, t, B, **kw):
    g = make_gpu_table(w, time=False, **kw)
    sd, dd, td = to_dev(src), to_dev(dst), to_dev(t)
    for lo in range(0, len(src), B):
        g.insert(sd[lo:lo + B], dd[lo:lo + B], td[lo:lo + B])
    return g


def test_batch_size_invariance_and_determinism():
    """The table equals sequential insertion for any batch size, and repeated
    runs give identical tables."""
    import torch
    w = synth.workload(2)
    src, dst, t, _ = synth.host_links(w)
    n = 200000
    src, dst, t = src[:n], dst[:n], t[:n]
    o = make_oracle(w)
    o.insert(src, dst, t)
    ref = None
    # batches below and above the size where insertion merges offers in LDS
    for B in (1, 7, 600, 2400, 65535, 65536, 100000, n):
        m = 3000 if B == 1 else (40000 if B == 7 else n)
        if m != n:
            o1 = make_oracle(w)
            o1.insert(src[:m], dst[:m], t[:m])
            compare_tables(_insert_in_batches(w, src[:m], dst[:m], t[:m], B), o1)
            continue
        g = _insert_in_batches(w, src, dst, t, B)
        compare_tables(g, o)
        cur = [x.cpu() for x in g.export()]
        if ref is not None:
            assert all(torch.equal(a, b) for a, b in zip(cur, ref))
        ref = cur


@pytest.mark.parametrize("alpha", [1.0, 1e-12, 0.3, 0.9])
def test_alpha_extremes(alpha):
    import dataclasses
    w = dataclasses.replace(synth.scaled(synth.workload(2), 30000), alpha=alpha)
    src, dst, t, _ = synth.host_links(dataclasses.replace(w, repeat=0.0))
    g = _insert_in_batches(w, src, dst, t, 600)
    o = make_oracle(w)
    o.insert(src, dst, t)
    compare_tables(g, o)


def test_single_hot_slot_batch():
    """Every offer of a batch lands on the same slot of one hub table (all
    links share the hub, the timestamp and a neighbour residue), plus
    self-loops, ties and a ragged batch."""
    N, s = 5000, 10
    import dataclasses
    w = dataclasses.replace(synth.workload(1), num_nodes=N, s=s)
    rng = np.random.default_rng(3)
    # neighbours congruent mod s, same t: eq. (2) gives one slot for all
    nb = (rng.integers(1, N // s, 140000) * s).astype(np.int32)
    src = np.zeros_like(nb)
    # self-loops, and timestamp ties throughout
    src[::97] = nb[::97]
    t = np.sort(np.concatenate([np.full(70000, 777, np.uint32), np.full(70000, 778, np.uint32)]))
    for B in (140000, 70000, 4096, 333):
        g = _insert_in_batches(w, src, nb, t, B)
        o = make_oracle(w)
        o.insert(src, nb, t)
        compare_tables(g, o)


@pytest.mark.parametrize("key_mode", [0, 1])
@pytest.mark.parametrize("s", [1, 3, 64, 100, 1024])
def test_slot_counts_and_key_modes(s, key_mode):
    """Table sizes across the layout classes (16-byte blocks up to multi-line
    blocks and more than 64 slots per query) and both key choices."""
    import dataclasses
    w = dataclasses.replace(synth.scaled(synth.workload(3), 40000, num_nodes=3000), s=s,
                            bursty=False, T=200000)
    src, dst, t, neg = synth.host_links(w)
    nf = synth.host_features(w, "node")
    nf_d = feat_to_dev(nf, w.node_dtype)
    g = make_gpu_table(w, None, nf_d, key_mode=key_mode)
    o = make_oracle(w, key_mode=key_mode)
    sd, dd, td = to_dev(src), to_dev(dst), to_dev(t)
    fw, fb = synth.time_params(w)
    nq = max(16, 20000 // s)   # keeps the oracle's cosine count bounded
    for lo in range(0, len(src), 8000):
        hi = lo + 8000
        q = np.concatenate([src[lo:lo + nq], neg[lo:lo + nq]])
        tq = np.concatenate([t[lo:lo + nq], t[lo:lo + nq] + 5])
        gout = g.sample(to_dev(q), to_dev(tq), want=("nbr", "eid", "ts", "tenc", "nfeat", "self"))
        oout = o.sample(q, tq, fw, fb, None, nf)
        compare_sample(gout, oout, f"s={s} lo={lo}")
        g.insert(sd[lo:hi], dd[lo:hi], td[lo:hi])
        o.insert(src[lo:hi], dst[lo:hi], t[lo:hi])
    compare_tables(g, o)


# ----------------------------------------------------------------------------- edge cases
def test_query_time_bounds_and_strictness():
    """tq = 0 sees nothing; tq = 2^32-1 sees every stored entry; entries at
    t' = tq are hidden (eq. (1) is strict)."""
    w = synth.scaled(synth.workload(1), 5000)
    src, dst, t, _ = synth.host_links(w)
    g = _insert_in_batches(w, src, dst, t, 200)
    o = make_oracle(w)
    o.insert(src, dst, t)
    nodes = np.arange(w.num_nodes, dtype=np.int32)
    nbr_o, ts_o, eid_o = o.export()
    for tq_val in (0, 2**32 - 1):
        tq = np.full(len(nodes), tq_val, np.uint32)
        gout = g.sample(to_dev(nodes), to_dev(tq), want=("nbr", "eid", "ts"))
        oout = o.sample(nodes, tq, want=("nbr", "eid", "ts"))
        compare_sample(gout, oout)
    assert (g.sample(to_dev(nodes), to_dev(np.full(len(nodes), 2**32 - 1, np.uint32)),
                     want=("nbr",))["nbr"].cpu().numpy() == nbr_o).all()
    # query each node at the timestamp of its first stored entry
    first_t = np.where(nbr_o[:, 0] >= 0, ts_o[:, 0], 0).astype(np.uint32)
    gout = g.sample(to_dev(nodes), to_dev(first_t), want=("nbr", "eid", "ts"))
    oout = o.sample(nodes, first_t, want=("nbr", "eid", "ts"))
    compare_sample(gout, oout)
    assert (gout["nbr"].cpu().numpy()[:, 0] == -1).all()


def test_feature_row_widths_and_time_dims():
    """Row sizes that take the 16-, 8- and 4-byte copy paths, a time
    encoding width that is not a multiple of 4, and offset output buffers."""
    import torch
    rng = np.random.default_rng(5)
    N, E, s = 300, 6000, 6
    src = rng.integers(0, N, E).astype(np.int32)
    dst = rng.integers(0, N, E).astype(np.int32)
    t = np.sort(rng.integers(0, 10**6, E)).astype(np.uint32)
    import paper_2402_01964_amd as nlb
    for erb_elems, nrb_elems, d_t in ((4, 6, 7), (2, 3, 100), (1, 1, 1), (93, 64, 12)):
        ef = rng.integers(0, 2**31, (E, erb_elems)).astype(np.int32)
        nf = rng.integers(0, 2**31, (N, nrb_elems)).astype(np.int32)
        fw = rng.uniform(0, 1, d_t).astype(np.float32)
        fb = rng.uniform(-3, 3, d_t).astype(np.float32)
        g = nlb.Table(N, s, 0.5, 9, time_w=to_dev(fw), time_b=to_dev(fb), edge_feat=to_dev(ef),
                      node_feat=to_dev(nf))
        o = oracle.Oracle(N, s, 0.5, 9)
        g.insert(to_dev(src), to_dev(dst), to_dev(t))
        o.insert(src, dst, t)
        q = rng.integers(0, N, 777).astype(np.int32)
        tq = rng.integers(0, 2 * 10**6, 777).astype(np.uint32)
        gout = g.sample(to_dev(q), to_dev(tq))
        compare_sample(gout, o.sample(q, tq, fw, fb, ef, nf), f"rows {erb_elems}/{nrb_elems}")
        # outputs at a 4-byte offset inside larger buffers
        big = torch.zeros(777 * s * erb_elems + 1, dtype=torch.int32, device="cuda")
        out = {"efeat": big[1:].view(777, s, erb_elems)}
        g.sample_into(to_dev(q), to_dev(tq), out)
        np.testing.assert_array_equal(out["efeat"].cpu().numpy(),
                                      o.sample(q, tq, None, None, ef, None)["efeat"])


def test_oversized_calls_are_rejected_before_launch():
    """Batch sizes whose 32-bit link or thread indices would wrap are refused
    on the host, and empty calls return at once: nothing is launched, so the
    tiny buffers are never read, and the table is unchanged."""
    import ctypes
    import torch
    import paper_2402_01964_amd as nlb
    g = nlb.Table(100, 4, 0.5, 1)
    z = torch.zeros(8, dtype=torch.int32, device="cuda")
    p = ctypes.c_void_p(z.data_ptr())
    lib = nlb.load_library()
    assert lib.nlb_insert_batch(g._h, p, p, p, 2**31, None) == nlb.NLB_EINVAL
    assert lib.nlb_insert_batch(g._h, p, p, p, 2**32 - 1, None) == nlb.NLB_EINVAL
    out = nlb._SampleOut()
    out.nbr = p
    # second hop: nq * s must stay below 2^32
    assert lib.nlb_sample_hop2(g._h, p, p, 2**30, ctypes.byref(out), None) == nlb.NLB_EINVAL
    # empty calls are no-ops that touch nothing
    assert lib.nlb_sample_hop2(g._h, p, p, 0, ctypes.byref(out), None) == nlb.NLB_OK
    aw = nlb._AggWeights()
    assert lib.nlb_aggregate(g._h, p, p, 0, ctypes.byref(aw), p, None) == nlb.NLB_OK
    torch.cuda.synchronize()
    assert g.info()["interactions"] == 0
    assert g.status() == nlb.NLB_OK
    assert not z.any()


def test_errors_are_reported_not_faulted():
    """Out-of-range ids, timestamps >= 2^30 and decreasing timestamps are
    skipped/flagged; the rest of the batch is applied as usual."""
    import paper_2402_01964_amd as nlb
    N, s = 100, 4
    g = nlb.Table(N, s, 0.5, 1)
    src = np.array([1, 2, 500, 3, -4], np.int32)
    dst = np.array([5, 6, 7, 8, 9], np.int32)
    t = np.array([10, 11, 12, 13, 14], np.uint32)
    g.insert(to_dev(src), to_dev(dst), to_dev(t))
    assert g.status() == nlb.NLB_ERANGE
    assert g.status() == nlb.NLB_OK  # cleared
    g.insert(to_dev(np.array([1], np.int32)), to_dev(np.array([2], np.int32)),
             to_dev(np.array([2**30], np.uint32)))
    assert g.status() == nlb.NLB_EORDER
    g.insert(to_dev(np.array([1], np.int32)), to_dev(np.array([2], np.int32)),
             to_dev(np.array([3], np.uint32)))
    assert g.status() == nlb.NLB_EORDER  # 3 < 14
    out = g.sample(to_dev(np.array([0, 5, 100, -1], np.int32)),
                   to_dev(np.array([99, 99, 99, 99], np.uint32)), want=("nbr",))
    assert g.status() == nlb.NLB_ERANGE
    nb = out["nbr"].cpu().numpy()
    assert (nb[2:] == -1).all()
    o = oracle.Oracle(N, s, 0.5, 1)
    o.insert_ids([0, 1, 3], src[[0, 1, 3]], dst[[0, 1, 3]], t[[0, 1, 3]])
    o.insert_ids([6], [1], [2], [3])
    nbr, ts, eid = g.export()
    on, ot, oe = o.export()
    np.testing.assert_array_equal(nbr.cpu().numpy(), on)
    np.testing.assert_array_equal(u32(eid), oe)
    # empty calls are no-ops
    g.insert(to_dev(np.zeros(0, np.int32)), to_dev(np.zeros(0, np.int32)),
             to_dev(np.zeros(0, np.uint32)))
    g.sample(to_dev(np.zeros(0, np.int32)), to_dev(np.zeros(0, np.uint32)), want=("nbr",))
    assert g.info()["interactions"] == 7   # flagged links still consume their index
    with pytest.raises(nlb.NLBError):  # no time encoding configured
        g.sample_into(to_dev(np.zeros(3, np.int32)), to_dev(np.zeros(3, np.uint32)),
                      {"tenc": to_dev(np.zeros(300, np.float32))})


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_second_hop_matches_oracle(k):
    """Sec. 4.4 second-hop retrieval on every workload shape: nlb_sample_hop2
    on the first-hop neighbours of a batch equals the oracle's second hop,
    rows and time encoding included, at several points of the stream (30
    batches of the workload's batch size, at most 200 000 nodes)."""
    base = synth.workload(k)
    w = synth.scaled(base, 30 * base.batch, num_nodes=min(base.num_nodes, 200000))
    src, dst, t, neg = synth.host_links(w)
    nodes, ts = synth.blocked(w, src, dst, t, neg)
    nodes_d, ts_d = to_dev(nodes), to_dev(ts)
    ef = synth.host_features(w, "edge") if w.edge_dim else None
    nf = synth.host_features(w, "node") if w.node_dim else None
    g = make_gpu_table(w, feat_to_dev(ef, w.edge_dtype) if ef is not None else None,
                       feat_to_dev(nf, w.node_dtype) if nf is not None else None)
    o = make_oracle(w)
    fw, fb = synth.time_params(w)
    for b in range(w.batches):
        s_, d_, t_, q, tq = synth.batch_views(w, nodes_d, ts_d, b)
        lo, hi = w.batch_range(b)
        if b in (3, 17, 29):
            qh = np.concatenate([src[lo:hi], dst[lo:hi], neg[lo:hi]])[:600]
            tqh = np.concatenate([t[lo:hi]] * 3)[:600]
            first = g.sample(q[:600], tq[:600], want=("nbr",))["nbr"]
            gout = g.sample_hop2(first, tq[:600])
            ofirst = o.sample(qh, tqh, want=("nbr",))["nbr"]
            np.testing.assert_array_equal(first.cpu().numpy(), ofirst)
            oout = o.sample_hop2(ofirst, tqh, fw, fb, ef, nf)
            compare_sample(gout, oout, f"hop2 batch {b}")
        g.insert(s_, d_, t_)
        o.insert(src[lo:hi], dst[lo:hi], t[lo:hi])
    assert g.status() == 0   # empty first-hop entries are not errors


def _agg_dev(W):
    import torch
    return {k: (to_dev(v.view(np.int16)) if v.dtype == np.uint16 else to_dev(v)) for k, v in W.items()}


def agg_error(gz, oz):
    """Max over elements of |z_gpu - z_oracle| / (|z_oracle| + rms(z_oracle))."""
    scale = np.sqrt(np.mean(oz ** 2))
    return float(np.max(np.abs(gz.astype(np.float64) - oz) / (np.abs(oz) + scale)))


AGG_TOL = 2e-4   # see nlb_aggregate in include/nlb.h for the derivation


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_aggregate_matches_oracle(k):
    """Eq. (4) forward on every workload shape (fp32 or bf16 rows, 372-byte
    unaligned rows, s = 10 / 20 / 64) at several points of a stream prefix,
    against the fp64 oracle; also queries with no valid slot."""
    base = synth.workload(k)
    w = synth.scaled(base, 12 * base.batch, num_nodes=min(base.num_nodes, 200000))
    src, dst, t, neg = synth.host_links(w)
    ef = synth.host_features(w, "edge") if w.edge_dim else None
    nf = synth.host_features(w, "node") if w.node_dim else None
    g = make_gpu_table(w, feat_to_dev(ef, w.edge_dtype) if ef is not None else None,
                       feat_to_dev(nf, w.node_dtype) if nf is not None else None)
    o = make_oracle(w)
    W = synth.agg_weights(w)
    Wd = _agg_dev(W)
    fw, fb = synth.time_params(w)
    worst = 0.0
    for b in range(w.batches):
        lo, hi = w.batch_range(b)
        if b in (2, 7, 11):
            q = np.concatenate([src[lo:hi], dst[lo:hi], neg[lo:hi]])[:3000]
            tq = np.concatenate([t[lo:hi]] * 3)[:3000]
            tq[::7] = 0                      # no valid slot for these
            gz = g.aggregate(to_dev(q), to_dev(tq), Wd).cpu().numpy()
            oz = o.aggregate(q, tq, fw, fb, ef, nf, W)
            worst = max(worst, agg_error(gz, oz))
        g.insert(to_dev(src[lo:hi]), to_dev(dst[lo:hi]), to_dev(t[lo:hi]))
        o.insert(src[lo:hi], dst[lo:hi], t[lo:hi])
    print(f"aggregate workload {k}: max scaled error {worst:.3e}")
    assert g.status() == 0
    assert worst <= AGG_TOL


# Input shapes that no wavefront-per-query instance covers (they take the
# tiled kernel): fp32 node rows 36 wide with bf16 link rows 90 wide and a
# 50-dim time encoding; bf16 node rows 200 wide (more than four k-steps).
TILED_SHAPES = {
    "f32node36-bf16edge90-t50": dict(node_dim=36, node_dtype="f32", edge_dim=90, edge_dtype="bf16", d_time=50),
    "bf16node200": dict(node_dim=200, node_dtype="bf16", edge_dim=0),
}


@pytest.mark.parametrize("shape", sorted(TILED_SHAPES))
def test_aggregate_tiled_shapes_match_oracle(shape):
    """Eq. (4) forward for input shapes outside the per-query kernel's
    instances, at 3 000 and 70 001 queries, against the fp64 oracle."""
    import dataclasses
    base = synth.workload(1)
    w = dataclasses.replace(synth.scaled(base, 12 * base.batch), **TILED_SHAPES[shape])
    src, dst, t, neg = synth.host_links(w)
    ef = synth.host_features(w, "edge") if w.edge_dim else None
    nf = synth.host_features(w, "node") if w.node_dim else None
    g = make_gpu_table(w, feat_to_dev(ef, w.edge_dtype) if ef is not None else None,
                       feat_to_dev(nf, w.node_dtype) if nf is not None else None)
    o = make_oracle(w)
    g.insert(to_dev(src), to_dev(dst), to_dev(t))
    o.insert(src, dst, t)
    W = synth.agg_weights(w)
    fw, fb = synth.time_params(w)
    rng = np.random.default_rng(7)
    ends = np.concatenate([src, dst, neg])
    worst = 0.0
    for nq in (3000, 70001):
        q = ends[rng.integers(0, len(ends), nq)].astype(np.int32)
        tq = rng.integers(0, int(t[-1]) + 2, nq).astype(np.uint32)
        tq[::9] = 0                                # no valid slot
        gz = g.aggregate(to_dev(q), to_dev(tq), _agg_dev(W)).cpu().numpy()
        pos = np.sort(rng.choice(nq, min(nq, 1500), replace=False))
        oz = o.aggregate(q[pos], tq[pos], fw, fb, ef, nf, W)
        worst = max(worst, agg_error(gz[pos], oz))
    print(f"aggregate tiled shape {shape}: max scaled error {worst:.3e}")
    assert g.status() == 0
    assert worst <= AGG_TOL


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_aggregate_large_launch_matches_oracle(k):
    """Launches of 70 001 queries (full groups of 16 queries in the
    wavefront-per-query kernel, with a partial last group) on every workload
    shape; 1 500 sampled queries are compared with the oracle,
    including queries without a valid slot and repeated query nodes."""
    import torch
    base = synth.workload(k)
    w = synth.scaled(base, 12 * base.batch, num_nodes=min(base.num_nodes, 200000))
    src, dst, t, _ = synth.host_links(w)
    ef = synth.host_features(w, "edge") if w.edge_dim else None
    nf = synth.host_features(w, "node") if w.node_dim else None
    g = make_gpu_table(w, feat_to_dev(ef, w.edge_dtype) if ef is not None else None,
                       feat_to_dev(nf, w.node_dtype) if nf is not None else None)
    o = make_oracle(w)
    lo, hi = 0, w.links
    g.insert(to_dev(src[lo:hi]), to_dev(dst[lo:hi]), to_dev(t[lo:hi]))
    o.insert(src[lo:hi], dst[lo:hi], t[lo:hi])
    rng = np.random.default_rng(70 + k)
    nq = 70001
    ends = np.concatenate([src, dst])
    q = ends[rng.integers(0, len(ends), nq)].astype(np.int32)
    tq = rng.integers(0, int(t[-1]) + 2, nq).astype(np.uint32)
    tq[::11] = 0                                   # no valid slot
    W = synth.agg_weights(w)
    gz = g.aggregate(to_dev(q), to_dev(tq), _agg_dev(W)).cpu().numpy()
    pos = np.sort(rng.choice(nq, 1500, replace=False))
    pos[-1] = nq - 1                               # the partial last group
    fw, fb = synth.time_params(w)
    oz = o.aggregate(q[pos], tq[pos], fw, fb, ef, nf, W)
    err = agg_error(gz[pos], oz)
    print(f"aggregate large launch, workload {k}: max scaled error {err:.3e}")
    assert g.status() == 0
    assert err <= AGG_TOL


@pytest.mark.parametrize("k,heads,shape", [(1, 2, None), (2, 2, None), (3, 2, None), (4, 2, None), (5, 2, None),
                                           (5, 4, None), (3, 8, None), (1, 2, "f32node36-bf16edge90-t50"),
                                           (1, 4, "bf16node200")])
def test_aggregate_heads_match_oracle(k, heads, shape):
    """Eq. (4) with several attention heads (App. E uses two), each over its
    own slice of the hidden width: two heads in the per-query kernel on
    every workload shape, four and eight in the tiled kernel, and the tiled
    shapes with two and four heads; launches of 3 000 and 70 001 queries,
    sampled queries against the fp64 oracle with the same heads."""
    import dataclasses
    base = synth.workload(k)
    w = synth.scaled(base, 12 * base.batch, num_nodes=min(base.num_nodes, 200000))
    if shape is not None:
        w = dataclasses.replace(w, **TILED_SHAPES[shape])
    src, dst, t, _ = synth.host_links(w)
    ef = synth.host_features(w, "edge") if w.edge_dim else None
    nf = synth.host_features(w, "node") if w.node_dim else None
    g = make_gpu_table(w, feat_to_dev(ef, w.edge_dtype) if ef is not None else None,
                       feat_to_dev(nf, w.node_dtype) if nf is not None else None)
    o = make_oracle(w)
    g.insert(to_dev(src), to_dev(dst), to_dev(t))
    o.insert(src, dst, t)
    W = synth.agg_weights(w)
    fw, fb = synth.time_params(w)
    rng = np.random.default_rng(40 + 3 * k + heads)
    ends = np.concatenate([src, dst])
    worst = 0.0
    for nq in (3000, 70001):
        q = ends[rng.integers(0, len(ends), nq)].astype(np.int32)
        tq = rng.integers(0, int(t[-1]) + 2, nq).astype(np.uint32)
        tq[::9] = 0
        gz = g.aggregate(to_dev(q), to_dev(tq), _agg_dev(W), heads=heads).cpu().numpy()
        pos = np.sort(rng.choice(nq, 800, replace=False))
        oz = o.aggregate(q[pos], tq[pos], fw, fb, ef, nf, W, heads=heads)
        worst = max(worst, agg_error(gz[pos], oz))
        if heads > 1:   # the heads change the result
            oz1 = o.aggregate(q[pos[:50]], tq[pos[:50]], fw, fb, ef, nf, W, heads=1)
            assert agg_error(gz[pos[:50]], oz1) > 10 * AGG_TOL
    print(f"aggregate, workload {k} shapes{'' if shape is None else ' ' + shape}, {heads} heads: "
          f"max scaled error {worst:.3e}")
    assert g.status() == 0
    assert worst <= AGG_TOL
