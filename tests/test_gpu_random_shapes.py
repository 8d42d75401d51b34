"""Seeded sweep of table and feature shapes against the oracle.

Each case draws a table (nodes, slots, alpha, key mode), a time encoding,
link and node rows of either element type and odd widths, and a stream with
self-loops, hubs and timestamp ties; it inserts the stream in batches of
random sizes and, before each batch, compares every sample output for
random queries (the batch's endpoints, random nodes; query times at, below
and above the batch's) with the oracle -- indices and rows bit-exact, the
time encoding within 1e-5 -- and compares the final tables.
"""
import numpy as np
import pytest

import oracle
import synth
from tests.gpu_helpers import compare_sample, compare_tables, feat_to_dev, to_dev

pytestmark = pytest.mark.gpu


def _case(seed):
    rng = np.random.default_rng(9100 + seed)
    N = int(rng.choice([1, 2, 17, 300, 3000]))
    s = int(rng.choice([1, 2, 3, 5, 8, 13, 32, 100]))
    alpha = float(rng.choice([0.1, 0.5, 0.9, 1.0]))
    key_mode = int(rng.integers(0, 2))
    d_time = int(rng.choice([0, 1, 5, 33, 100]))
    E = int(rng.integers(1, 12000))
    hub = rng.random() < 0.5
    src = rng.integers(0, N, E)
    dst = rng.integers(0, N, E)
    if hub:
        src = np.where(rng.random(E) < 0.4, 0, src)
    loops = rng.random(E) < 0.05
    dst[loops] = src[loops]
    t = np.sort(rng.integers(0, int(rng.choice([50, 10**4, 10**8])), E))
    feats = {}
    for which, rows in (("edge", E + 10), ("node", N)):
        if rng.random() < 0.6:
            dtype = str(rng.choice(["f32", "bf16"]))
            # rows are a multiple of 4 bytes (an odd bf16 width is rejected)
            width = int(rng.choice([1, 3, 8, 37, 64] if dtype == "f32" else [2, 8, 10, 64, 128]))
            x = rng.standard_normal((rows, width)).astype(np.float32)
            feats[which] = (synth._to_bf16_bits(x) if dtype == "bf16" else x, dtype)
    fw = (10.0 ** -rng.uniform(0, 6, d_time)).astype(np.float32)
    fb = rng.uniform(-np.pi, np.pi, d_time).astype(np.float32)
    return dict(rng=rng, N=N, s=s, alpha=alpha, key_mode=key_mode, d_time=d_time,
                src=src.astype(np.int32), dst=dst.astype(np.int32), t=t.astype(np.uint32),
                feats=feats, fw=fw, fb=fb, seed=seed)


@pytest.mark.parametrize("seed", range(32))
def test_random_shapes_match_oracle(seed):
    import paper_2402_01964_amd as nlb
    c = _case(seed)
    rng, N, s = c["rng"], c["N"], c["s"]
    ef, ef_dt = c["feats"].get("edge", (None, None))
    nf, nf_dt = c["feats"].get("node", (None, None))
    tw = tb = None
    if c["d_time"]:
        tw, tb = to_dev(c["fw"]), to_dev(c["fb"])
    g = nlb.Table(N, s, c["alpha"], 40 + seed, time_w=tw, time_b=tb, key_mode=c["key_mode"],
                  edge_feat=feat_to_dev(ef, ef_dt) if ef is not None else None,
                  node_feat=feat_to_dev(nf, nf_dt) if nf is not None else None)
    o = oracle.Oracle(N, s, c["alpha"], 40 + seed, key_mode=c["key_mode"])
    src, dst, t = c["src"], c["dst"], c["t"]
    what = (f"seed {seed}: N={N} s={s} alpha={c['alpha']} key_mode={c['key_mode']} "
            f"d_time={c['d_time']} links={len(src)} edge={None if ef is None else (ef.shape[1], ef_dt)} "
            f"node={None if nf is None else (nf.shape[1], nf_dt)}")
    print(what, flush=True)
    lo = 0
    while lo < len(src):
        hi = min(len(src), lo + int(rng.integers(1, 3000)))
        nq = int(rng.integers(1, 400))
        q = np.concatenate([src[lo:hi], rng.integers(0, N, nq)])[: max(1, min(nq, 2000 // s + 1))]
        base = int(t[lo])
        tq = np.where(rng.random(len(q)) < 0.5, base,
                      rng.integers(max(0, base - 100), base + 1000, len(q))).astype(np.uint32)
        if rng.random() < 0.2:
            tq[:] = 0
        gout = g.sample(to_dev(q.astype(np.int32)), to_dev(tq))
        oout = o.sample(q.astype(np.int32), tq, c["fw"] if c["d_time"] else None,
                        c["fb"] if c["d_time"] else None, ef, nf)
        compare_sample(gout, oout, f"{what} batch at {lo}")
        g.insert(to_dev(src[lo:hi]), to_dev(dst[lo:hi]), to_dev(t[lo:hi]))
        o.insert(src[lo:hi], dst[lo:hi], t[lo:hi])
        lo = hi
    compare_tables(g, o)
    assert g.status() == 0
