"""Calls inside a HIP graph.

nlb_sample, nlb_aggregate and nlb_insert_batch enqueue kernels only (no
allocation, no memset, no synchronisation), and the insert keeps the stream's
link count on the device, as does nlb_rnn_update once its working memory is
sized; so a caller whose batches land in the same device buffers every step
can capture a whole step once and replay it: the launch-bound small
workloads then pay one graph launch per step.  Replays are checked against
eager calls and against the oracle."""
import numpy as np
import pytest

import synth
from tests.gpu_helpers import compare_sample, feat_to_dev, make_gpu_table, make_oracle, to_dev

pytestmark = pytest.mark.gpu


def _agg_dev(W):
    return {k: (to_dev(v.view(np.int16)) if v.dtype == np.uint16 else to_dev(v)) for k, v in W.items()}


def test_sample_and_aggregate_replay_in_a_hip_graph():
    import torch
    import paper_2402_01964_amd as nlb
    base = synth.workload(3)                        # bf16 link and node rows, s = 64
    w = synth.scaled(base, 6 * base.batch, num_nodes=min(base.num_nodes, 200000))
    src, dst, t, neg = synth.host_links(w)
    ef = synth.host_features(w, "edge")
    nf = synth.host_features(w, "node")
    g = make_gpu_table(w, feat_to_dev(ef, w.edge_dtype), feat_to_dev(nf, w.node_dtype))
    o = make_oracle(w)
    for b in range(4):
        lo, hi = w.batch_range(b)
        g.insert(to_dev(src[lo:hi]), to_dev(dst[lo:hi]), to_dev(t[lo:hi]))
        o.insert(src[lo:hi], dst[lo:hi], t[lo:hi])
    lo, hi = w.batch_range(4)
    qh = np.concatenate([src[lo:hi], dst[lo:hi], neg[lo:hi]])
    tqh = np.concatenate([t[lo:hi]] * 3)
    q, tq = to_dev(qh), to_dev(tqh)
    Wd = _agg_dev(synth.agg_weights(w))

    # Eager calls: the reference, and the first-call set-up of both paths.
    out = g.alloc_outputs(len(qh))
    z = torch.empty((len(qh), nlb.AGG_HIDDEN), dtype=torch.float32, device="cuda")
    g.sample_into(q, tq, out)
    g.aggregate(q, tq, Wd, out=z)
    torch.cuda.synchronize()
    ref = {k: v.clone() for k, v in out.items()}
    ref_z = z.clone()
    fw, fb = synth.time_params(w)
    compare_sample(ref, o.sample(qh, tqh, fw, fb, ef, nf), "eager sample")

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        g.sample_into(q, tq, out)
        g.aggregate(q, tq, Wd, out=z)
    for rep in range(3):
        for v in out.values():
            v.fill_(7)                              # eager work on the same buffers
        z.fill_(7.0)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for k, v in out.items():
            assert torch.equal(v, ref[k]), f"replay {rep}: {k}"
        assert torch.equal(z, ref_z), f"replay {rep}: z"
    del graph
    assert g.status() == nlb.NLB_OK
    g.close()


@pytest.mark.parametrize("k", [1, 2])
def test_whole_step_replays_against_the_oracle(k):
    """One whole step -- nlb_sample of the batch's queries (Sec. 4.4), then
    nlb_insert_batch of its links (Sec. 4.2), then the status update with
    the arrival indices of the links just inserted (NLB_EID_LAST_BATCH) --
    captured once and replayed for 40 consecutive batches, each copied into
    the captured input buffers before its replay.  Every replay's retrieval
    equals the oracle's at that point of the stream, the statuses its GRU
    update (within 1e-4, from the GPU's statuses before the step), and the
    tables and the device link count match at the end."""
    import torch
    import oracle
    import paper_2402_01964_amd as nlb
    from tests.gpu_helpers import compare_tables, host_np
    base = synth.workload(k)
    steps = 41
    w = synth.scaled(base, steps * base.batch)
    src, dst, t, neg = synth.host_links(w)
    nodes, ts = synth.blocked(w, src, dst, t, neg)
    ef = synth.host_features(w, "edge")
    g = make_gpu_table(w, feat_to_dev(ef, w.edge_dtype), None)
    o = make_oracle(w)
    fw, fb = synth.time_params(w)
    d, _ = synth.status_spec(w)                      # fp32 statuses (no node rows)
    status = to_dev(np.random.default_rng(k).standard_normal((w.num_nodes, d)).astype(np.float32))
    W = synth.gru_weights(w)
    Wd = _agg_dev(W)
    B, Q = w.batch, 3 * w.batch
    q_s = torch.empty(Q, dtype=torch.int32, device="cuda")
    tq_s = torch.empty(Q, dtype=torch.int32, device="cuda")
    out = g.alloc_outputs(Q)

    def run_step():
        g.sample_into(q_s, tq_s, out)
        g.insert(q_s[:B], q_s[B:2 * B], tq_s[:B])
        g.rnn_update(q_s[:B], q_s[B:2 * B], tq_s[:B], nlb.EID_LAST_BATCH, Wd, status)

    def check(b, pre):
        lo, hi = w.batch_range(b)
        compare_sample(out, o.sample(nodes[3 * lo:3 * hi], ts[3 * lo:3 * hi], fw, fb, ef, None),
                       f"workload {k} step {b}")
        o.insert(src[lo:hi], dst[lo:hi], t[lo:hi])
        want = oracle.gru_update(pre.copy(), src[lo:hi], dst[lo:hi], t[lo:hi], lo, fw, fb, ef, W)
        err = float(np.abs(host_np(status).astype(np.float64) - want.astype(np.float64)).max())
        assert err <= 1e-4, (k, b, err)

    def load(b):
        lo, hi = w.batch_range(b)
        q_s.copy_(to_dev(nodes[3 * lo:3 * hi]))
        tq_s.copy_(to_dev(ts[3 * lo:3 * hi]))

    load(0)                                          # eager step: sizes the update's memory
    pre = host_np(status).copy()
    run_step()
    torch.cuda.synchronize()
    check(0, pre)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        run_step()
    for b in range(1, steps):
        load(b)
        torch.cuda.synchronize()
        pre = host_np(status).copy()
        graph.replay()
        torch.cuda.synchronize()
        check(b, pre)
    del graph
    assert g.status() == nlb.NLB_OK
    assert g.info()["interactions"] == w.links       # the device count, refreshed by nlb_status
    compare_tables(g, o)
    g.close()


def test_packed_aggregation_replays_in_a_hip_graph():
    """The packed eq. (4) kernel (groups of at least 8 queries, s = 10) in a
    HIP graph: 30 000 queries captured once and replayed three times with
    eager work on the output between replays; every replay equals the eager
    result bit for bit, which matches the oracle on sampled queries."""
    import torch
    import paper_2402_01964_amd as nlb
    from tests.test_gpu_parity import AGG_TOL, agg_error
    base = synth.workload(5)
    w = synth.scaled(base, 4 * base.batch, num_nodes=200000)
    src, dst, t, neg = synth.host_links(w)
    nf = synth.host_features(w, "node")
    g = make_gpu_table(w, None, feat_to_dev(nf, w.node_dtype))
    o = make_oracle(w)
    lo, hi = w.batch_range(3)
    g.insert(to_dev(src[:lo]), to_dev(dst[:lo]), to_dev(t[:lo]))
    o.insert(src[:lo], dst[:lo], t[:lo])
    qh = np.concatenate([src[lo:hi], dst[lo:hi], neg[lo:hi]])[:30000]
    tqh = np.concatenate([t[lo:hi]] * 3)[:30000]
    q, tq = to_dev(qh), to_dev(tqh)
    W = synth.agg_weights(w)
    Wd = _agg_dev(W)
    z = torch.empty((len(qh), nlb.AGG_HIDDEN), dtype=torch.float32, device="cuda")
    g.aggregate(q, tq, Wd, out=z)
    torch.cuda.synchronize()
    ref = z.clone()
    fw, fb = synth.time_params(w)
    pos = np.sort(np.random.default_rng(5).choice(len(qh), 600, replace=False))
    assert agg_error(ref.cpu().numpy()[pos], o.aggregate(qh[pos], tqh[pos], fw, fb, None, nf, W)) <= AGG_TOL
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        g.aggregate(q, tq, Wd, out=z)
    for rep in range(3):
        z.fill_(7.0)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(z, ref), f"replay {rep}"
    del graph
    assert g.status() == nlb.NLB_OK
    g.close()
