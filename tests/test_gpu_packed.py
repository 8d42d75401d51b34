"""The packed form of the eq. (4) aggregation (Sec. 4.4).

Launches whose query groups hold at least 8 queries, on tables of at most 16
slots, pack the valid slots of each group of queries into full 16-row
blocks, each query's run padded to a multiple of four rows.  These cases
drive that form through the C ABI on every instantiated input shape (fp32
link rows, 4-byte-aligned bf16 link rows, bf16 node rows with and without
link rows), with one attention head and with two, with s from 1 to 16, time encodings whose width is not a
multiple of 4 (97, 101, 127) as well as 100 and 128, groups of 16 and of
10 queries, a partial last group, queries without a valid slot and
arguments past the fast cosine's range.  Sampled queries are compared with
the fp64 oracle, and every query with the same queries launched in groups
of one (the per-query form), which differs by summation order only.
"""
import dataclasses

import numpy as np
import pytest

import oracle
import synth
from tests.gpu_helpers import feat_to_dev, to_dev
from tests.test_gpu_parity import AGG_TOL, _agg_dev, agg_error

pytestmark = pytest.mark.gpu

# (workload whose row shapes are used, s, d_time, time weights scale, heads)
CASES = [
    (5, 10, 100, 1.0, 1),
    (5, 1, 97, 1.0, 1),
    (5, 4, 101, 1.0, 1),
    (5, 16, 128, 1.0, 1),
    (1, 13, 100, 1.0, 1),
    (1, 16, 127, 1.0, 1),
    (4, 3, 100, 1.0, 1),
    (4, 10, 98, 1.0, 1),
    (3, 8, 100, 1.0, 1),
    (5, 10, 100, 1e6, 1),     # w dt + b past 2^33: the wide-argument cosine
    # two heads (App. E) on every instantiated shape
    (5, 10, 100, 1.0, 2),
    (5, 1, 97, 1.0, 2),
    (1, 13, 101, 1.0, 2),
    (4, 10, 100, 1.0, 2),
    (3, 16, 100, 1.0, 2),
    (2, 5, 100, 1.0, 2),
]


def _ids(c):
    k, s, d, ws, heads = c
    return f"w{k}-s{s}-d{d}" + ("-wide" if ws != 1.0 else "") + (f"-h{heads}" if heads > 1 else "")


@pytest.mark.parametrize("case", CASES, ids=_ids)
def test_packed_aggregation_matches_oracle_and_unpacked(case):
    import paper_2402_01964_amd as nlb
    k, s, d_time, wscale, heads = case
    base = synth.workload(k)
    w = dataclasses.replace(synth.scaled(base, 12 * base.batch, num_nodes=min(base.num_nodes, 50000)),
                            s=s, d_time=d_time)
    src, dst, t, _ = synth.host_links(w)
    ef = synth.host_features(w, "edge") if w.edge_dim else None
    nf = synth.host_features(w, "node") if w.node_dim else None
    fw, fb = synth.time_params(w)
    fw = (fw * np.float32(wscale)).astype(np.float32)
    g = nlb.Table(w.num_nodes, s, w.alpha, w.table_seed, time_w=to_dev(fw), time_b=to_dev(fb),
                  edge_feat=feat_to_dev(ef, w.edge_dtype) if ef is not None else None,
                  node_feat=feat_to_dev(nf, w.node_dtype) if nf is not None else None)
    o = oracle.Oracle(w.num_nodes, s, w.alpha, w.table_seed)
    g.insert(to_dev(src), to_dev(dst), to_dev(t))
    o.insert(src, dst, t)
    W = synth.agg_weights(w)
    Wd = _agg_dev(W)
    rng = np.random.default_rng(900 + 7 * s + k)
    ends = np.concatenate([src, dst])
    print(f"packed aggregation: workload {k} shapes, s={s}, d_time={d_time}, time weights x{wscale}, "
          f"{heads} head(s)", flush=True)
    for nq in (70001, 20003):                      # groups of 16 and of 10 queries
        q = ends[rng.integers(0, len(ends), nq)].astype(np.int32)
        q[::13] = rng.integers(0, w.num_nodes, len(q[::13]))   # nodes with few or no links
        tq = rng.integers(0, int(t[-1]) + 2, nq).astype(np.uint32)
        tq[::11] = 0                                # no valid slot
        gz = g.aggregate(to_dev(q), to_dev(tq), Wd, heads=heads).cpu().numpy()
        # the same queries in launches of 3000 (groups of 2 queries: unpacked)
        uz = np.concatenate([g.aggregate(to_dev(q[i:i + 3000]), to_dev(tq[i:i + 3000]), Wd,
                                         heads=heads).cpu().numpy()
                             for i in range(0, nq, 3000)])
        pos = np.sort(rng.choice(nq, 1200, replace=False))
        pos[-1] = nq - 1                            # the partial last group
        oz = o.aggregate(q[pos], tq[pos], fw, fb, ef, nf, W, heads=heads)
        e_orc = agg_error(gz[pos], oz)
        e_unp = agg_error(gz, uz.astype(np.float64))
        print(f"  {nq} queries: vs oracle {e_orc:.3e}, vs unpacked {e_unp:.3e}", flush=True)
        assert e_orc <= AGG_TOL, (nq, e_orc)
        assert e_unp <= 2 * AGG_TOL, (nq, e_unp)
    assert g.status() == nlb.NLB_OK
    g.close()
