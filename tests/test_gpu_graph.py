"""Retrieval and aggregation inside a HIP graph.

nlb_sample and nlb_aggregate enqueue kernels only (no allocation, no
memset, no synchronisation), so a caller whose queries land in the same
device buffers every step can capture them once and replay the graph: the
launch-bound small workloads then pay one graph launch per step.  Each
replay here follows eager work on the same buffers and is checked against
the eager call.  (nlb_insert_batch is not replayable: it assigns arrival
indices on the host.)"""
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
