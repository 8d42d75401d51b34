"""nlb_time_encode: the App. C time encoding of a first-hop answer, computed
from its timestamp output on a stream of the caller's choice.

It must give the bits nlb_sample writes to its own tenc output (both launch
paths of nlb_sample: the streaming kernel of large launches and the encoding
inside sample_gather of small ones), match the fp64 oracle within 1e-5 in
both its vector form and its scalar form (a width that is not a multiple of
4, an output at a 4-byte offset), and stay correct when it runs on a second
stream beside the next insert, which rewrites the slots it was sampled from.
"""
import dataclasses

import numpy as np
import pytest

import synth
from tests.gpu_helpers import compare_sample, make_gpu_table, make_oracle, to_dev

pytestmark = pytest.mark.gpu

# (workload whose stream is used, d_time, output at a 4-byte offset, s or
# None for the workload's own); s = 1 with one float4 or one float per slot
# makes both divisors of the kernel 1
CASES = [(4, 100, False, None), (4, 97, False, None), (1, 100, True, None), (5, 128, False, None),
         (4, 4, False, 1), (4, 1, True, 1)]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"w{c[0]}-d{c[1]}" + ("-offset" if c[2] else "")
                         + (f"-s{c[3]}" if c[3] else ""))
def test_time_encode_matches_sample_and_oracle(case):
    import torch
    k, d_time, offset, s_slots = case
    base = synth.workload(k)
    w = dataclasses.replace(synth.scaled(base, 20 * base.batch, num_nodes=min(base.num_nodes, 50000)),
                            d_time=d_time, s=s_slots or base.s)
    src, dst, t, _ = synth.host_links(w)
    fw, fb = synth.time_params(w)
    g = make_gpu_table(w)
    g.insert(to_dev(src), to_dev(dst), to_dev(t))
    o = make_oracle(w)
    o.insert(src, dst, t)
    rng = np.random.default_rng(40 + k)
    ends = np.concatenate([src, dst])
    for nq in (30000, 500):          # both launch paths of nlb_sample
        print(f"time encode: workload {k}, d_time={d_time}, offset={offset}, {nq} queries", flush=True)
        q = ends[rng.integers(0, len(ends), nq)].astype(np.int32)
        q[::17] = rng.integers(0, w.num_nodes, len(q[::17]))
        tq = rng.integers(0, int(t[-1]) + 2, nq).astype(np.uint32)
        tq[::9] = 0                  # no valid slot
        tq_d = to_dev(tq)
        a = g.sample(to_dev(q), tq_d, want=("nbr", "ts", "tenc"))
        n = nq * w.s * d_time
        buf = torch.full((n + 1,), float("nan"), dtype=torch.float32, device="cuda")
        tenc = (buf[1:] if offset else buf[:n]).view(nq, w.s, d_time)
        g.time_encode_into(a["ts"], tq_d, tenc)
        assert torch.equal(tenc, a["tenc"]), (k, d_time, nq)
        if not offset:
            assert torch.isnan(buf[n]), "wrote past the output"
        oo = o.sample(q[:400], tq[:400], fw, fb, None, None, want=("nbr", "ts", "tenc"))
        compare_sample({"nbr": a["nbr"][:400], "ts": a["ts"][:400], "tenc": tenc[:400]},
                       {"nbr": oo["nbr"], "ts": oo["ts"], "tenc": oo["tenc"]}, f"nq={nq}")
    assert g.status() == 0
    g.close()


def test_time_encode_beside_the_next_insert():
    """The split retrieval of the benchmark: table reads on the main stream,
    the encoding on a second stream after an event, the next batch's insert
    on the main stream at the same time, and the main stream waiting for the
    encoding before the next retrieval reuses the buffers.  Every batch's
    answer equals the oracle's answer at that point of the stream."""
    import torch
    base = synth.workload(4)
    w = synth.scaled(base, 12 * base.batch)
    src, dst, t, neg = synth.host_links(w)
    fw, fb = synth.time_params(w)
    g = make_gpu_table(w)
    o = make_oracle(w)
    B = w.batch
    nq = 3 * B
    ts_buf = torch.empty((nq, w.s), dtype=torch.int32, device="cuda")
    nbr_buf = torch.empty((nq, w.s), dtype=torch.int32, device="cuda")
    tenc_buf = torch.empty((nq, w.s, w.d_time), dtype=torch.float32, device="cuda")
    main = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    results = []
    g.insert(to_dev(src[:B]), to_dev(dst[:B]), to_dev(t[:B]))
    o.insert(src[:B], dst[:B], t[:B])
    for b in range(1, len(src) // B):
        sl = slice(b * B, (b + 1) * B)
        q = np.concatenate([src[sl], dst[sl], neg[sl]]).astype(np.int32)
        tq = np.concatenate([t[sl]] * 3).astype(np.uint32)
        q_d, tq_d = to_dev(q), to_dev(tq)
        s_d, d_d, t_d = to_dev(src[sl]), to_dev(dst[sl]), to_dev(t[sl])
        g.sample_into(q_d, tq_d, {"nbr": nbr_buf, "ts": ts_buf})
        ev = torch.cuda.Event()
        ev.record(main)
        side.wait_event(ev)
        with torch.cuda.stream(side):
            g.time_encode_into(ts_buf, tq_d, tenc_buf, stream=side)
            done = torch.cuda.Event()
            done.record(side)
        g.insert(s_d, d_d, t_d)              # rewrites slots the answer came from
        main.wait_event(done)
        results.append((q, tq, nbr_buf.clone(), ts_buf.clone(), tenc_buf.clone()))
        torch.cuda.synchronize()
        oo = o.sample(q[:600], tq[:600], fw, fb, None, None, want=("nbr", "ts", "tenc"))
        o.insert(src[sl], dst[sl], t[sl])
        r = results[-1]
        compare_sample({"nbr": r[2][:600], "ts": r[3][:600], "tenc": r[4][:600]},
                       {"nbr": oo["nbr"], "ts": oo["ts"], "tenc": oo["tenc"]}, f"batch {b}")
    print(f"split retrieval beside inserts: {len(results)} batches of {nq} queries", flush=True)
    assert g.status() == 0
    g.close()


def test_time_encode_errors():
    import torch
    import paper_2402_01964_amd as nlb
    w = synth.scaled(synth.workload(1), 4 * synth.workload(1).batch)
    g = make_gpu_table(w)
    no_t = make_gpu_table(w, time=False)
    ts = torch.zeros((10, w.s), dtype=torch.int32, device="cuda")
    tq = torch.zeros(10, dtype=torch.int32, device="cuda")
    tenc = torch.zeros((10, w.s, w.d_time), dtype=torch.float32, device="cuda")
    lib = g._lib
    P = tenc.data_ptr()
    assert lib.nlb_time_encode(g._h, ts.data_ptr(), tq.data_ptr(), 0, P, None) == nlb.NLB_OK
    assert lib.nlb_time_encode(g._h, None, tq.data_ptr(), 10, P, None) == nlb.NLB_EINVAL
    assert lib.nlb_time_encode(g._h, ts.data_ptr(), tq.data_ptr(), 10, None, None) == nlb.NLB_EINVAL
    assert lib.nlb_time_encode(g._h, ts.data_ptr(), tq.data_ptr(), 10, P + 2, None) == nlb.NLB_EINVAL
    assert lib.nlb_time_encode(no_t._h, ts.data_ptr(), tq.data_ptr(), 10, P, None) == nlb.NLB_EINVAL
    assert lib.nlb_time_encode(None, ts.data_ptr(), tq.data_ptr(), 10, P, None) == nlb.NLB_EINVAL
    with pytest.raises(ValueError):
        g.time_encode_into(ts[:5], tq, tenc)
    torch.cuda.synchronize()
    assert g.status() == 0
    g.close()
    no_t.close()


def test_split_retrieval_replays_in_a_hip_graph():
    """The split retrieval captured in one HIP graph, the encoding on a
    second stream forked and joined by events inside the capture (as the
    benchmark's graph mode runs it): replayed three times with eager work on
    the outputs between replays, every replay equals the eager call."""
    import torch
    base = synth.workload(4)
    w = synth.scaled(base, 6 * base.batch)
    src, dst, t, neg = synth.host_links(w)
    g = make_gpu_table(w)
    B = w.batch
    g.insert(to_dev(src[:4 * B]), to_dev(dst[:4 * B]), to_dev(t[:4 * B]))
    sl = slice(4 * B, 5 * B)
    q = to_dev(np.concatenate([src[sl], dst[sl], neg[sl]]).astype(np.int32))
    tq = to_dev(np.concatenate([t[sl]] * 3).astype(np.uint32))
    nq = 3 * B
    out = g.alloc_outputs(nq, want=("nbr", "eid", "ts", "tenc"))
    g.sample_into(q, tq, out)                        # eager reference, one call
    torch.cuda.synchronize()
    ref = {k: v.clone() for k, v in out.items()}
    side = torch.cuda.Stream()
    ev, done = torch.cuda.Event(), torch.cuda.Event()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        ids = {k: out[k] for k in ("nbr", "eid", "ts")}
        g.sample_into(q, tq, ids)
        ev.record()
        side.wait_event(ev)
        g.time_encode_into(out["ts"], tq, out["tenc"], stream=side)
        done.record(side)
        torch.cuda.current_stream().wait_event(done)
    for rep in range(3):
        for v in out.values():
            v.fill_(7)                               # eager work on the same buffers
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for k, v in out.items():
            assert torch.equal(v, ref[k]), f"replay {rep}: {k}"
    del graph
    assert g.status() == 0
    g.close()
