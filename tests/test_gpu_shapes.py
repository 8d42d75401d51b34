"""GPU parity at the edges of what nlb_create accepts, against the oracle.

* The widest sample tile: s = 1024 gives tiles of 1024 slot rows; with
  262 140-byte node and link rows (65 535 four-byte copy units per row) and
  a 65 535-wide time encoding the flat output index of a tile reaches
  1024 * 65535 (Sec. 4.4 row gathers, App. C time encoding).
* The time-encoding stream with a divisor of one: one slot per node (s = 1,
  the truncation case of Sec. 4.1) and four time dimensions (one float4
  per slot row), at launches large enough to take that kernel.
* Link rows past the link-feature table: a stored link without a row there
  gathers a zero row, in retrieval, the second hop and eq. (4).
"""
import numpy as np
import pytest

import oracle
import synth
from tests.gpu_helpers import compare_sample, feat_to_dev, make_gpu_table, make_oracle, to_dev

pytestmark = pytest.mark.gpu


def _log(*a):
    print("[shapes]", *a, flush=True)


def test_widest_tile_rows_and_time_encoding():
    import paper_2402_01964_amd as nlb
    import torch
    rng = np.random.default_rng(1024)
    N, s, E, units = 64, 1024, 6000, 65535
    d_time = units                                   # not a multiple of 4: one value per unit
    src = np.zeros(E, np.int32)                      # node 0 fills (nearly) all 1024 slots
    dst = (1 + np.arange(E) % (N - 1)).astype(np.int32)
    t = (10 * np.arange(E)).astype(np.uint32)
    nfeat = rng.integers(-2**31, 2**31 - 1, (N, units), dtype=np.int64).astype(np.int32)
    efeat = rng.integers(-2**31, 2**31 - 1, (E // 2, units), dtype=np.int64).astype(np.int32)
    fw = (10.0 ** -rng.uniform(0, 9, d_time)).astype(np.float32)
    fb = rng.uniform(-np.pi, np.pi, d_time).astype(np.float32)
    _log(f"s={s}, rows of {4 * units} B, d_time={d_time}: table on the GPU")
    # alpha = 0.3: about 40% of the first half's entries survive the second half
    g = nlb.Table(N, s, 0.3, 7, time_w=to_dev(fw), time_b=to_dev(fb), edge_feat=to_dev(efeat),
                  node_feat=to_dev(nfeat))
    g.insert(to_dev(src), to_dev(dst), to_dev(t))
    o = oracle.Oracle(N, s, 0.3, 7)
    o.insert(src, dst, t)
    q = np.array([0, 0, 5], np.int32)
    tq = np.array([10 * E + 1, 10 * E // 2, 10 * E + 1], np.uint32)
    gout = g.sample(to_dev(q), to_dev(tq))
    torch.cuda.synchronize()
    assert g.status() == 0
    _log("GPU done; oracle")
    oout = o.sample(q, tq, fw, fb, efeat, nfeat)
    valid = oout["nbr"] >= 0
    late = valid & (oout["eid"] >= E // 2)
    _log(f"valid slots per query {valid.sum(1).tolist()}, of them without a link row {int(late.sum())}")
    assert valid[0].sum() > 1000 and 300 < valid[1].sum() < 700 and late.sum() > 300
    assert (valid[0, 250:].sum() > 700)          # valid slots deep into the tile (rows >= 258)
    compare_sample(gout, oout, "widest tile")
    assert not oout["efeat"][late].any()


@pytest.mark.parametrize("d_time,nq", [(100, 50000), (4, 1_100_000)])
def test_time_encoding_stream_single_slot(d_time, nq):
    """s = 1: slot row j belongs to query j; d_time = 4: one float4 per slot
    row.  Both launches are large enough to compute the time encoding in
    its own streaming kernel (with the timestamp output requested); the
    same call without timestamps computes it in the sample kernel.  Both
    match the oracle everywhere."""
    import paper_2402_01964_amd as nlb
    import torch
    rng = np.random.default_rng(d_time)
    N, E = 1000, 20000
    src = rng.integers(0, N, E).astype(np.int32)
    dst = rng.integers(0, N, E).astype(np.int32)
    t = np.sort(rng.integers(0, 10**6, E)).astype(np.uint32)
    fw = (10.0 ** -np.linspace(0, 9, d_time)).astype(np.float32)
    fb = rng.uniform(-np.pi, np.pi, d_time).astype(np.float32)
    g = nlb.Table(N, 1, 0.5, 11, time_w=to_dev(fw), time_b=to_dev(fb))
    g.insert(to_dev(src), to_dev(dst), to_dev(t))
    o = oracle.Oracle(N, 1, 0.5, 11)
    o.insert(src, dst, t)
    q = rng.integers(0, N, nq).astype(np.int32)
    tq = rng.integers(int(t[-1]) - 10**5, int(t[-1]) + 2, nq).astype(np.uint32)
    a = g.sample(to_dev(q), to_dev(tq), want=("nbr", "eid", "ts", "tenc"))
    b = g.sample(to_dev(q), to_dev(tq), want=("tenc",))
    torch.cuda.synchronize()
    assert torch.equal(a["tenc"], b["tenc"])
    oout = o.sample(q, tq, fw, fb, want=("nbr", "eid", "ts", "tenc"))
    valid = oout["nbr"] >= 0
    assert 0.2 < valid.mean() < 0.9
    compare_sample(a, oout, f"s=1 d_time={d_time} nq={nq}")


def _agg_dev(W):
    return {k: (to_dev(v.view(np.int16)) if v.dtype == np.uint16 else to_dev(v)) for k, v in W.items()}


@pytest.mark.parametrize("k", [1, 4])
def test_link_rows_past_the_table(k):
    """The table is given the link rows of the first half of the stream
    only: stored links of the second half gather zero rows, exactly as the
    oracle with the same partial table answers, in retrieval, the second
    hop and eq. (4)."""
    base = synth.workload(k)
    w = synth.scaled(base, 20 * base.batch)
    src, dst, t, neg = synth.host_links(w)
    ef = synth.host_features(w, "edge")
    half = ef[: w.links // 2].copy()
    g = make_gpu_table(w, feat_to_dev(half, w.edge_dtype), None)
    o = make_oracle(w)
    g.insert(to_dev(src), to_dev(dst), to_dev(t))
    o.insert(src, dst, t)
    fw, fb = synth.time_params(w)
    rng = np.random.default_rng(k)
    ends = np.concatenate([src, dst])
    q = ends[rng.integers(0, len(ends), 3000)].astype(np.int32)
    tq = np.full(3000, int(t[-1]) + 1, np.uint32)
    gout = g.sample(to_dev(q), to_dev(tq))
    oout = o.sample(q, tq, fw, fb, half, None)
    late = (oout["nbr"] >= 0) & (oout["eid"] >= len(half))
    assert late.sum() > 1000 and ((oout["nbr"] >= 0) & ~late).sum() > 1000
    compare_sample(gout, oout, f"workload {k} partial link rows")
    g2 = g.sample_hop2(gout["nbr"][:300], to_dev(tq[:300]))
    compare_sample(g2, o.sample_hop2(oout["nbr"][:300], tq[:300], fw, fb, half, None),
                   f"workload {k} partial link rows, second hop")
    W = synth.agg_weights(w)
    gz = g.aggregate(to_dev(q), to_dev(tq), _agg_dev(W)).cpu().numpy()
    oz = o.aggregate(q[:500], tq[:500], fw, fb, half, None, W)
    scale = np.sqrt(np.mean(oz ** 2))
    err = float(np.max(np.abs(gz[:500].astype(np.float64) - oz) / (np.abs(oz) + scale)))
    _log(f"workload {k}: aggregate with partial link rows, scaled error {err:.2e}")
    assert err <= 2e-4
    assert g.status() == 0


@pytest.mark.parametrize("sweep", ["reduced-domain", "wide-arguments"])
def test_device_cosine_dense_sweep(sweep):
    """The library's fp32 cosine against the oracle's cosine in double of
    the same fp32 argument (App. C time encoding), through nlb_sample, by
    band of |x|: <= 5e-7 below 1e9; <= 2.5e-6 up to 2^33, where the double
    product x / (2 pi) is off by up to 2.7e-7 of a revolution; <= 1e-6
    beyond (the exact wide-argument route); <= 1e-5 (the interface's bound)
    everywhere.  reduced-domain: w = 0 and 65 532 phases b covering
    [-pi, pi] densely, so the argument is b itself (the whole reduced domain
    of [-1/2, 1/2] revolution); wide-arguments: log-spaced frequencies
    1e-9 .. 10 and 80 time gaps from 1 to 2^32 - 1, arguments up to 4e10
    (beyond 2^33 the wide-argument route).  Both launch paths: with the
    timestamp output (time-encoding stream, >= 2^20 float4 outputs) and
    without it (the sample kernel's own phase)."""
    import paper_2402_01964_amd as nlb
    import torch
    D, nq = 65532, 80                               # 80 x 16 383 float4 >= 2^20
    rng = np.random.default_rng(77)
    if sweep == "reduced-domain":
        fw = np.zeros(D, np.float32)
        fb = np.linspace(-np.pi, np.pi, D).astype(np.float32)
        dt = np.arange(1, nq + 1, dtype=np.uint64)
    else:
        fw = np.logspace(-9, 1, D).astype(np.float32)
        fb = rng.uniform(-np.pi, np.pi, D).astype(np.float32)
        dt = np.unique(np.concatenate([
            [1, 2, 3, 7, 1000, 65535, 65536, 65537, 10**6 + 3, 2**24 + 1, 10**8 - 1, 2**30 - 1, 2**31,
             2**32 - 1], rng.integers(1, 2**32, nq)]).astype(np.uint64))[:nq]
    assert len(dt) == nq
    g = nlb.Table(2, 1, 1.0, 5, time_w=to_dev(fw), time_b=to_dev(fb))
    g.insert(to_dev(np.zeros(1, np.int32)), to_dev(np.ones(1, np.int32)), to_dev(np.zeros(1, np.uint32)))
    q = np.zeros(nq, np.int32)
    tq = dt.astype(np.uint32)                      # the stored link has t' = 0
    a = g.sample(to_dev(q), to_dev(tq), want=("ts", "tenc"))
    b = g.sample(to_dev(q), to_dev(tq), want=("tenc",))
    torch.cuda.synchronize()
    o = oracle.Oracle(2, 1, 1.0, 5)
    o.insert([0], [1], [0])
    want = o.sample(q, tq, fw, fb, want=("nbr", "tenc"))
    assert (want["nbr"] >= 0).all()
    ref = want["tenc"].astype(np.float64)
    # |x| of each argument (w dt is exact in double for fp32 w and dt)
    x = np.abs(fw.astype(np.float64)[None, :] * dt.astype(np.float32).astype(np.float64)[:, None]
               + fb.astype(np.float64)[None, :]).reshape(nq, 1, D)
    bands = ((0.0, 1e9, 5e-7), (1e9, 2.0**33, 2.5e-6), (2.0**33, np.inf, 1e-6))
    for name, got in (("stream", a["tenc"]), ("sample kernel", b["tenc"])):
        err = np.abs(got.cpu().numpy().astype(np.float64) - ref)
        assert err.max() <= 1e-5, (sweep, name, float(err.max()))
        for lo, hi, tol in bands:
            sel = (x >= lo) & (x < hi)
            if sel.any():
                e = float(err[sel].max())
                _log(f"cosine sweep {sweep}, {name} path, {lo:.0e} <= |x| < {hi:.0e}: {int(sel.sum())} "
                     f"values, max abs error {e:.2e}")
                assert e <= tol, (sweep, name, lo, e)


@pytest.mark.parametrize("k,s", [(5, 100), (5, 1024), (1, 200)])
def test_aggregate_tables_wider_than_64_slots(k, s):
    """eq. (4) on tables of more than 64 slots, which the per-query kernel
    takes in ceil(s / 16) blocks per query, against the oracle on sampled
    queries of launches of 3 000 and 70 001 queries; a shape that only the
    tiled kernel serves is refused for such tables."""
    import dataclasses
    import paper_2402_01964_amd as nlb
    from tests.test_gpu_parity import AGG_TOL, _agg_dev, agg_error
    base = synth.workload(k)
    w = dataclasses.replace(synth.scaled(base, 8 * base.batch, num_nodes=min(base.num_nodes, 20000)), s=s)
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
    rng = np.random.default_rng(300 + s)
    ends = np.concatenate([src, dst])
    for nq in (3000, 70001):
        q = ends[rng.integers(0, len(ends), nq)].astype(np.int32)
        tq = rng.integers(0, int(t[-1]) + 2, nq).astype(np.uint32)
        tq[::9] = 0
        gz = g.aggregate(to_dev(q), to_dev(tq), _agg_dev(W)).cpu().numpy()
        pos = np.sort(rng.choice(nq, 400, replace=False))
        oz = o.aggregate(q[pos], tq[pos], fw, fb, ef, nf, W)
        err = agg_error(gz[pos], oz)
        _log(f"aggregate, workload {k} shapes, s={s}, {nq} queries: max scaled error {err:.3e}")
        assert err <= AGG_TOL, (nq, err)
    assert g.status() == nlb.NLB_OK
    g.close()
    # node rows 200 wide: no per-query instance, so s > 64 is refused
    w2 = dataclasses.replace(w, node_dim=200, node_dtype="bf16", edge_dim=0)
    nf2 = synth.host_features(w2, "node")
    g2 = make_gpu_table(w2, None, feat_to_dev(nf2, "bf16"))
    with pytest.raises(nlb.NLBError) as err:
        g2.aggregate(to_dev(q[:10]), to_dev(tq[:10]), _agg_dev(synth.agg_weights(w2)))
    assert err.value.code == nlb.NLB_EINVAL
    g2.close()
