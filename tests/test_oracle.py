"""Pins of the CPU oracle against what the paper and mathematics fix.

Each test checks the oracle against something other than itself: a
hand-worked example, published known-answer values, a brute-force
formulation that does not replay the sequential loop, a closed-form law or a
textbook special case.  All run on the CPU.
"""
import math
import os

import numpy as np
import pytest

import oracle
from oracle import Oracle

Q1, Q2 = oracle.DEFAULT_Q1, oracle.DEFAULT_Q2


# ----------------------------------------------------------------------------- helpers
def slot_residue(x, t, s, q1=Q1, q2=Q2, key_mode=0):
    """eq. (2)/(3) evaluated through residues mod s (a different formulation
    from the oracle's direct 64-bit product)."""
    x = np.asarray(x, np.uint64) % np.uint64(s)
    t = np.asarray(t, np.uint64) % np.uint64(s)
    a = (np.uint64(q1 % s) * x) % np.uint64(s)
    if key_mode == 0:
        a = (a + (np.uint64(q2 % s) * t) % np.uint64(s)) % np.uint64(s)
    return a.astype(np.int64)


def offers_of(src, dst, t):
    """Offer list in sequential order: (e, k, table n, neighbour x, t)."""
    E = len(src)
    e = np.repeat(np.arange(E, dtype=np.int64), 2)
    k = np.tile(np.array([0, 1], np.int64), E)
    n = np.stack([src, dst], 1).reshape(-1).astype(np.int64)
    x = np.stack([dst, src], 1).reshape(-1).astype(np.int64)
    tt = np.repeat(np.asarray(t, np.int64), 2)
    return e, k, n, x, tt


def random_stream(rng, N, E, tmax, self_loops=True):
    src = rng.integers(0, N, E).astype(np.int32)
    dst = rng.integers(0, N, E).astype(np.int32)
    if not self_loops:
        bad = src == dst
        while bad.any():
            dst[bad] = rng.integers(0, N, bad.sum())
            bad = src == dst
    t = np.sort(rng.integers(0, tmax, E)).astype(np.uint32)
    return src, dst, t


def table_from_winners(N, s, n, a, x, t, e):
    nbr = np.full((N, s), -1, np.int32)
    ts = np.full((N, s), 0xFFFFFFFF, np.uint32)
    eid = np.full((N, s), 0xFFFFFFFF, np.uint32)
    nbr[n, a] = x
    ts[n, a] = t
    eid[n, a] = e
    return nbr, ts, eid


def brute_force_table(N, s, src, dst, t, keep, pick_max=True, key_mode=0):
    """Per (node, slot): the max-e (or min-e) offer among offers where
    ``keep`` is True.  Group-by over the whole offer set; no sequential loop."""
    e, k, n, x, tt = offers_of(src, dst, t)
    a = slot_residue(x, tt, s, key_mode=key_mode)
    m = keep
    e, n, x, tt, a = e[m], n[m], x[m], tt[m], a[m]
    cell = n * s + a
    order = np.lexsort((e if pick_max else -e, cell))
    cell_sorted = cell[order]
    last = np.ones(len(order), bool)
    last[:-1] = cell_sorted[1:] != cell_sorted[:-1]
    w = order[last]
    return table_from_winners(N, s, n[w], a[w], x[w], tt[w], e[w])


def first_offer_mask(n, a, s):
    cell = n * s + a
    _, first_idx = np.unique(cell, return_index=True)
    m = np.zeros(len(cell), bool)
    m[first_idx] = True
    return m


def assert_tables_equal(got, want):
    for g, w, name in zip(got, want, ("nbr", "ts", "eid")):
        np.testing.assert_array_equal(g, w, err_msg=name)


# ----------------------------------------------------------------------------- known answers
def _read_golden(path):
    rows = []
    with open(path) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                rows.append(line.split())
    return rows


def test_coin_matches_splitmix64_known_answers(golden_dir):
    """coin(e, k) is the high half of SplitMix64 output 2e+k+1: pinned to the
    published outputs for start states 0 and 1234567."""
    for st, n, val in _read_golden(os.path.join(golden_dir, "splitmix64_vectors.txt")):
        st, n, val = int(st), int(n), int(val, 0)
        o = Oracle(4, 1, 0.5, seed=st)
        e, k = (n - 1) // 2, (n - 1) % 2
        assert o.coin(e, k) == val >> 32, (st, n)


def test_handworked_tables(golden_dir):
    """The hand-worked 6-link example (eq. (2), eq. (3), replacement rule)."""
    rows = _read_golden(os.path.join(golden_dir, "handworked_tables.txt"))
    params = dict(kv.split("=") for kv in rows[0][1:])
    N, s, q1, q2 = (int(params[k]) for k in ("N", "s", "q1", "q2"))
    links = np.array([[int(v) for v in r[1:]] for r in rows if r[0] == "link"])
    assert (links[:, 0] == np.arange(len(links))).all()
    src, dst, t = links[:, 1], links[:, 2], links[:, 3]
    alphas = {"latest": 1.0, "first": 1e-12}
    made = {}
    for mode, km in (("edge", 0), ("node", 1)):
        for rule, alpha in alphas.items():
            o = Oracle(N, s, alpha, seed=99, q1=q1, q2=q2, key_mode=km)
            o.insert(src, dst, t)
            made[(mode, rule)] = o
    assert made[("edge", "first")].threshold == 0
    assert made[("edge", "latest")].threshold == 2**32
    checked = 0
    for r in rows:
        if r[0] != "table":
            continue
        mode, rule, node, a, nbr = r[1], r[2], int(r[3]), int(r[4]), int(r[5])
        got_nbr, got_ts, got_eid = made[(mode, rule)].export()
        assert got_nbr[node, a] == nbr, r
        if nbr >= 0:
            assert got_ts[node, a] == int(r[6]) and got_eid[node, a] == int(r[7]), r
        else:
            assert got_ts[node, a] == 0xFFFFFFFF and got_eid[node, a] == 0xFFFFFFFF, r
        checked += 1
    assert checked == 4 * N * s
    for r in rows:
        if r[0] != "query":
            continue
        rule, node, tq, a, valid = r[1], int(r[2]), int(r[3]), int(r[4]), int(r[5])
        out = made[("edge", rule)].sample([node], [tq])
        assert (out["nbr"][0, a] >= 0) == bool(valid), r
    hop2_rows = [r for r in rows if r[0] == "hop2"]
    assert hop2_rows
    for r in hop2_rows:
        rule, node, tq, a, c, nbr = r[1], int(r[2]), int(r[3]), int(r[4]), int(r[5]), int(r[6])
        o = made[("edge", rule)]
        first = o.sample([node], [tq], want=("nbr",))["nbr"]
        out = o.sample_hop2(first, [tq], want=("nbr", "eid", "ts"))
        assert out["nbr"][0, a, c] == nbr, r
        if nbr >= 0:
            assert (out["ts"][0, a, c], out["eid"][0, a, c]) == (int(r[7]), int(r[8])), r


def test_slot_matches_eq2_bigint():
    """64-bit evaluation of eq. (2)/(3) equals arbitrary-precision integers."""
    rng = np.random.default_rng(1)
    xs = rng.integers(0, 2**31, 3000)
    ts = rng.integers(0, 2**32, 3000)
    xs[:3] = [0, 2**31 - 1, 2**31 - 1]
    ts[:3] = [0, 2**32 - 1, 0]
    for s in (1, 2, 7, 10, 20, 64, 1000):
        for km in (0, 1):
            o = Oracle(2, s, 0.5, 0, key_mode=km)
            for x, t in zip(xs[:400], ts[:400]):
                want = (Q1 * int(x) + (Q2 * int(t) if km == 0 else 0)) % s
                assert o.slot(int(x), int(t)) == want


def test_threshold_values():
    """floor(alpha * 2^32) in double (alpha = 1 -> 2^32)."""
    assert Oracle(2, 1, 1.0, 0).threshold == 2**32
    assert Oracle(2, 1, 0.5, 0).threshold == 2**31
    assert Oracle(2, 1, 0.3, 0).threshold == 1288490188
    assert Oracle(2, 1, 0.9, 0).threshold == math.floor(0.9 * 2**32)


def test_rejects_bad_parameters():
    for kw in (dict(num_nodes=0, s=1, alpha=0.5), dict(num_nodes=4, s=0, alpha=0.5),
               dict(num_nodes=4, s=2, alpha=0.0), dict(num_nodes=4, s=2, alpha=1.5)):
        with pytest.raises(ValueError):
            Oracle(seed=0, **kw)
    o = Oracle(4, 2, 0.5, 0)
    with pytest.raises(ValueError):
        o.insert([0], [4], [1])
    with pytest.raises(ValueError):
        o.sample([7], [1])


# ----------------------------------------------------------------------------- coin statistics
def test_coin_uniform_and_acceptance_rate():
    """The coin is uniform on 32 bits (chi^2 over 256 bins of its top byte)
    and passes thr = floor(alpha 2^32) with frequency alpha."""
    o = Oracle(2, 1, 0.3, seed=12345)
    n = 200000
    r = np.array([o.coin(e, k) for e in range(n // 2) for k in (0, 1)], np.uint64)
    hist = np.bincount((r >> np.uint64(24)).astype(np.int64), minlength=256)
    expect = n / 256
    chi2 = ((hist - expect) ** 2 / expect).sum()
    # 255 dof: mean 255, sd ~22.6; 6 sd bound
    assert chi2 < 255 + 6 * 22.6
    for alpha in (0.1, 0.3, 0.5, 0.9):
        thr = math.floor(alpha * 2**32)
        p = (r < thr).mean()
        assert abs(p - alpha) < 5 * math.sqrt(alpha * (1 - alpha) / n)


# ----------------------------------------------------------------------------- brute force
@pytest.mark.parametrize("s,key_mode", [(1, 0), (3, 0), (10, 0), (20, 0), (10, 1)])
def test_alpha_one_each_slot_holds_latest(s, key_mode):
    """alpha = 1: every slot holds the latest offer hashing to it."""
    rng = np.random.default_rng(s + 10 * key_mode)
    N, E = 50, 3000
    src, dst, t = random_stream(rng, N, E, 10**6)
    o = Oracle(N, s, 1.0, seed=5, key_mode=key_mode)
    o.insert(src, dst, t)
    keep = np.ones(2 * E, bool)
    assert_tables_equal(o.export(), brute_force_table(N, s, src, dst, t, keep, True, key_mode))


def test_threshold_zero_each_slot_holds_first():
    """alpha below 2^-32 (threshold 0): only empty slots take offers, so
    every slot holds the first offer hashing to it."""
    rng = np.random.default_rng(3)
    N, s, E = 40, 10, 3000
    src, dst, t = random_stream(rng, N, E, 10**6)
    o = Oracle(N, s, 1e-12, seed=5)
    assert o.threshold == 0
    o.insert(src, dst, t)
    keep = np.ones(2 * E, bool)
    assert_tables_equal(o.export(), brute_force_table(N, s, src, dst, t, keep, False))


def test_single_slot_alpha_one_is_truncation_to_one():
    """s = 1, alpha = 1: each node keeps exactly its most recent link
    (truncation with one neighbour, Sec. 4.1)."""
    rng = np.random.default_rng(4)
    N, E = 30, 2000
    src, dst, t = random_stream(rng, N, E, 10**5)
    o = Oracle(N, 1, 1.0, seed=1)
    o.insert(src, dst, t)
    nbr, ts, eid = o.export()
    for node in range(N):
        touching = np.nonzero((src == node) | (dst == node))[0]
        if len(touching) == 0:
            assert nbr[node, 0] == -1
            continue
        last = touching[-1]
        other = dst[last] if src[last] == node else src[last]
        assert (nbr[node, 0], ts[node, 0], eid[node, 0]) == (other, t[last], last)


@pytest.mark.parametrize("alpha,seed", [(0.3, 11), (0.5, 12), (0.9, 13)])
def test_set_form_brute_force(alpha, seed):
    """Any alpha: slot (n,a) holds the max-e offer of the set
    {first offer to (n,a)} U {offers to (n,a) whose coin passes} --
    a formulation that never replays the sequential loop."""
    rng = np.random.default_rng(seed)
    N, s, E = 60, 10, 4000
    src, dst, t = random_stream(rng, N, E, 10**6)
    o = Oracle(N, s, alpha, seed=seed * 7)
    o.insert(src, dst, t)
    e, k, n, x, tt = offers_of(src, dst, t)
    a = slot_residue(x, tt, s)
    coin = np.array([o.coin(int(ee), int(kk)) for ee, kk in zip(e, k)], np.uint64)
    keep = first_offer_mask(n, a, s) | (coin < np.uint64(o.threshold))
    assert_tables_equal(o.export(), brute_force_table(N, s, src, dst, t, keep, True))


def test_batching_is_invisible_to_the_table():
    """Inserting in batches of any size gives the one-at-a-time table."""
    rng = np.random.default_rng(8)
    N, s, E = 80, 10, 5000
    src, dst, t = random_stream(rng, N, E, 10**6)
    ref = Oracle(N, s, 0.5, seed=3)
    for i in range(E):
        ref.insert(src[i:i + 1], dst[i:i + 1], t[i:i + 1])
    for B in (7, 200, 4999):
        o = Oracle(N, s, 0.5, seed=3)
        for lo in range(0, E, B):
            o.insert(src[lo:lo + B], dst[lo:lo + B], t[lo:lo + B])
        assert_tables_equal(o.export(), ref.export())


def test_filtered_substream_gives_same_rows():
    """Tables are per node: inserting only the links that touch a node set,
    with their global arrival indices, gives those nodes' rows exactly."""
    rng = np.random.default_rng(9)
    N, s, E = 200, 10, 8000
    src, dst, t = random_stream(rng, N, E, 10**6)
    full = Oracle(N, s, 0.5, seed=21)
    full.insert(src, dst, t)
    nodes = np.array([0, 3, 17, 150, 199], np.int32)
    sel = np.nonzero(np.isin(src, nodes) | np.isin(dst, nodes))[0]
    part = Oracle(N, s, 0.5, seed=21)
    part.insert_ids(sel, src[sel], dst[sel], t[sel])
    for a, b in zip(part.export_nodes(nodes), full.export_nodes(nodes)):
        np.testing.assert_array_equal(a, b)


# ----------------------------------------------------------------------------- invariants
def test_kept_node_subset_gives_the_same_rows():
    """Tables are per node (Sec. 4.2): an oracle that keeps only some nodes'
    tables ends with exactly the rows the full structure has for them, and
    answers their queries identically; other nodes are refused."""
    rng = np.random.default_rng(31)
    N, s, E = 500, 6, 20000
    src, dst, t = random_stream(rng, N, E, 10**6)
    keep = np.unique(rng.integers(0, N, 60)).astype(np.int32)[::-1].copy()
    full = Oracle(N, s, 0.4, seed=5)
    part = Oracle(N, s, 0.4, seed=5, keep=np.concatenate([keep, keep[:5]]))
    assert part.rows == len(keep)
    for lo in range(0, E, 3000):
        full.insert(src[lo:lo + 3000], dst[lo:lo + 3000], t[lo:lo + 3000])
        part.insert(src[lo:lo + 3000], dst[lo:lo + 3000], t[lo:lo + 3000])
        tq = np.full(len(keep), t[min(E, lo + 3000) - 1] + 1, np.uint32)
        a = full.sample(keep, tq, want=("nbr", "eid", "ts"))
        b = part.sample(keep, tq, want=("nbr", "eid", "ts"))
        for k in a:
            np.testing.assert_array_equal(a[k], b[k])
    for x, y in zip(full.export_nodes(keep), part.export_nodes(keep)):
        np.testing.assert_array_equal(x, y)
    assert (full.export_nodes(keep)[0] >= 0).sum() > 100
    other = np.setdiff1d(np.arange(N), keep)[:1].astype(np.int32)
    with pytest.raises(ValueError):
        part.sample(other, np.ones(1, np.uint32))
    with pytest.raises(ValueError):
        part.export_nodes(other)
    with pytest.raises(ValueError):
        part.export()


def test_invariants_and_strict_query_mask():
    rng = np.random.default_rng(10)
    N, s, E = 100, 10, 6000
    src, dst, t = random_stream(rng, N, E, 10**5)
    o = Oracle(N, s, 0.5, seed=2)
    o.insert(src, dst, t)
    nbr, ts, eid = o.export()
    for node in range(N):
        for a in range(s):
            if nbr[node, a] < 0:
                continue
            e_ = int(eid[node, a])
            assert {int(src[e_]), int(dst[e_])} == {node, int(nbr[node, a])}
            assert ts[node, a] == t[e_]
            assert o.slot(int(nbr[node, a]), int(ts[node, a])) == a
    nodes = rng.integers(0, N, 500).astype(np.int32)
    tq = rng.integers(0, 10**5, 500).astype(np.uint32)
    out = o.sample(nodes, tq)
    for i in range(len(nodes)):
        row_t = ts[nodes[i]]
        valid = (nbr[nodes[i]] >= 0) & (row_t < tq[i])
        assert ((out["nbr"][i] >= 0) == valid).all()
        assert (out["ts"][i][valid] < tq[i]).all()
        assert (out["eid"][i][~valid] == 0xFFFFFFFF).all()


# ----------------------------------------------------------------------------- closed forms
@pytest.mark.parametrize("alpha", [0.3, 0.5, 0.9])
def test_survival_law_over_seeds(alpha):
    """An offer followed by m later offers to its slot is present at the end
    with probability alpha(1-alpha)^m if the slot was occupied when it
    arrived, and (1-alpha)^m if it was empty (Sec. 4.2 rule; the per-link
    replacement step used in the proof of Theorem 1)."""
    rng = np.random.default_rng(100)
    N, s, E = 6, 2, 30
    src, dst, t = random_stream(rng, N, E, 1000, self_loops=False)
    e, k, n, x, tt = offers_of(src, dst, t)
    a = slot_residue(x, tt, s)
    cell = n * s + a
    m = np.array([(cell[i + 1:] == cell[i]).sum() for i in range(len(cell))])
    occupied = np.array([(cell[:i] == cell[i]).any() for i in range(len(cell))])
    p = np.where(occupied, alpha * (1 - alpha) ** m, (1 - alpha) ** m)
    K = 20000
    hits = np.zeros(len(cell))
    for seed in range(1, K + 1):
        o = Oracle(N, s, alpha, seed=seed)
        o.insert(src, dst, t)
        _, _, eid = o.export()
        hits += eid[n, a] == e
    freq = hits / K
    sd = np.sqrt(np.maximum(p * (1 - p), 1e-12) / K)
    z = np.abs(freq - p) / sd
    assert z.max() < 4.5, (z.max(), freq[z.argmax()], p[z.argmax()])


@pytest.mark.parametrize("alpha", [0.3, 0.7])
def test_same_key_offer_is_an_ordinary_collision(alpha):
    """NLB-node (eq. (3)): a later link with the same neighbour maps to the
    same slot.  Theorem 2's proof (App. B) inserts every other temporal
    neighbour with probability alpha, so the second of two links from v to u
    replaces the first in a fraction alpha of seeds; a same-key-always-
    overwrites reading would give 1.  Binomial z-test over 20 000 seeds."""
    K = 20000
    hits = 0
    for seed in range(K):
        o = Oracle(4, 3, alpha, seed=seed, key_mode=1)
        o.insert([0, 0], [1, 1], [5, 9])
        nbr, ts, eid = o.export_nodes([0])
        held = eid[0][nbr[0] == 1]
        assert len(held) == 1
        hits += int(held[0] == 1)
    z = (hits - K * alpha) / math.sqrt(K * alpha * (1 - alpha))
    assert abs(z) < 4.5, (hits / K, alpha)


def test_theorem1_poisson_hub_survival():
    """Theorem 1 (NLB-edge achieves recent sampling): with Poisson(lambda)
    arrivals at a hub, a link that entered S_u at t_i is still there at t
    with probability exp(-alpha lambda (t - t_i) / s).  Away from the start,
    an offer enters with probability alpha, so presence = alpha * that."""
    alpha, s, lam, T, H = 0.5, 10, 1.0, 200.0, 400
    scale = 1000.0
    pres, delta = [], []
    for rep in range(4):
        rng = np.random.default_rng(500 + rep)
        times, hubs = [], []
        for h in range(H):
            n = rng.poisson(lam * T)
            times.append(rng.uniform(0, T, n))
            hubs.append(np.full(n, h))
        times = np.concatenate(times)
        hubs = np.concatenate(hubs)
        order = np.argsort(times, kind="stable")
        times, hubs = times[order], hubs[order]
        E = len(times)
        leaves = H + rng.permutation(E)          # every leaf appears once
        tt = np.floor(times * scale).astype(np.uint32)
        o = Oracle(H + E, s, alpha, seed=900 + rep)
        o.insert(hubs.astype(np.int32), leaves.astype(np.int32), tt)
        nbr, ts, eid = o.export_nodes(np.arange(H, dtype=np.int32))
        present = np.zeros(E, bool)
        got = eid[eid != 0xFFFFFFFF]
        present[got] = True
        keep = times > 60.0                       # tables long since full
        pres.append(present[keep])
        delta.append(T - times[keep])
    pres = np.concatenate(pres)
    delta = np.concatenate(delta)
    expect = alpha * np.exp(-alpha * lam * delta / s)
    edges = np.arange(0, 141, 10.0)
    for lo, hi in zip(edges[:-1], edges[1:]):
        m = (delta >= lo) & (delta < hi)
        n = m.sum()
        mu = expect[m].sum()
        var = (expect[m] * (1 - expect[m])).sum()
        assert abs(pres[m].sum() - mu) < 5 * math.sqrt(var) + 1, (lo, pres[m].sum(), mu, n)


# ----------------------------------------------------------------------------- T-encoding
def test_tenc_paper_form_cos_sin_pairs():
    """App. C: with phases b in {0, -pi/2} the encoding is the
    [cos(w t), sin(w t)] pairs of the paper.  Frequencies are powers of two
    and gaps small integers, so w*dt is exact in fp32."""
    d = 16
    w = np.repeat(2.0 ** -np.arange(d // 2), 2).astype(np.float32)
    b = np.tile(np.array([0.0, -np.pi / 2], np.float32), d // 2)
    dt = np.array([0, 1, 2, 3, 5], np.float32)
    out = oracle.tenc(dt, w, b)
    for i, g in enumerate(dt):
        for j in range(d // 2):
            x = float(w[2 * j]) * float(g)
            assert abs(out[i, 2 * j] - math.cos(x)) < 1e-7
            assert abs(out[i, 2 * j + 1] - math.sin(x)) < 1e-6


def test_tenc_zero_gap_and_exact_points():
    w = np.array([1.0, 0.5, 1e-9, 3.0], np.float32)
    b = np.array([0.0, np.float32(np.pi), 0.25, -1.0], np.float32)
    out = oracle.tenc(np.array([0.0], np.float32), w, b)[0]
    assert out[0] == 1.0
    assert abs(out[1] + 1.0) < 1e-7
    assert abs(out[2] - math.cos(0.25)) < 1e-7
    assert abs(out[3] - math.cos(-1.0)) < 1e-7


def test_sample_outputs_rows_and_zeros():
    """Sec. 4.4 retrieval: valid slots carry the link's feature row, the
    neighbour's node row and the T-encoding of tq - t'; invalid slots carry
    -1 / 0xFFFFFFFF and all-zero rows; the self row is the query node's."""
    rng = np.random.default_rng(20)
    N, s, E = 40, 4, 500
    src, dst, t = random_stream(rng, N, E, 10**4)
    o = Oracle(N, s, 0.5, seed=4)
    o.insert(src, dst, t)
    efeat = rng.standard_normal((E, 6)).astype(np.float32)
    nfeat = rng.integers(0, 2**16, (N, 5)).astype(np.uint16)
    w = rng.uniform(0, 1, 7).astype(np.float32)
    b = rng.uniform(-3, 3, 7).astype(np.float32)
    nodes = rng.integers(0, N, 100).astype(np.int32)
    tq = rng.integers(0, 10**4, 100).astype(np.uint32)
    out = o.sample(nodes, tq, w, b, efeat, nfeat)
    nbr, ts, eid = o.export()
    for i in range(100):
        np.testing.assert_array_equal(out["self"][i], nfeat[nodes[i]])
        for a in range(s):
            valid = nbr[nodes[i], a] >= 0 and ts[nodes[i], a] < tq[i]
            if valid:
                e_ = eid[nodes[i], a]
                np.testing.assert_array_equal(out["efeat"][i, a], efeat[e_])
                np.testing.assert_array_equal(out["nfeat"][i, a], nfeat[nbr[nodes[i], a]])
                gap = np.float32(int(tq[i]) - int(ts[nodes[i], a]))
                for kk in range(7):
                    arg = np.float32(float(w[kk]) * float(gap) + float(b[kk]))  # fma, one rounding
                    want = math.cos(float(arg))
                    assert abs(out["tenc"][i, a, kk] - want) < 2e-6
            else:
                assert out["nbr"][i, a] == -1 and out["eid"][i, a] == 0xFFFFFFFF
                assert out["ts"][i, a] == 0xFFFFFFFF
                assert not out["efeat"][i, a].any() and not out["nfeat"][i, a].any()
                assert not out["tenc"][i, a].any()


def test_link_rows_past_the_table_are_zero_rows():
    """A stored link whose arrival index has no row in the link-feature
    table (the table keeps only its first rows) gathers an all-zero row in
    retrieval; it equals the answer for a table padded with zero rows."""
    rng = np.random.default_rng(21)
    N, s, E = 30, 4, 400
    src, dst, t = random_stream(rng, N, E, 10**4)
    o = Oracle(N, s, 0.7, seed=9)
    o.insert(src, dst, t)
    full = rng.standard_normal((E, 6)).astype(np.float32)
    keep = 250
    part = full[:keep].copy()
    padded = np.concatenate([part, np.zeros((E - keep, 6), np.float32)])
    nodes = rng.integers(0, N, 200).astype(np.int32)
    tq = np.full(200, 10**4 + 1, np.uint32)
    got = o.sample(nodes, tq, efeat=part, want=("eid", "efeat"))
    want = o.sample(nodes, tq, efeat=padded, want=("eid", "efeat"))
    np.testing.assert_array_equal(got["efeat"], want["efeat"])
    late = (got["eid"] != 0xFFFFFFFF) & (got["eid"] >= keep)
    early = (got["eid"] != 0xFFFFFFFF) & (got["eid"] < keep)
    assert late.sum() > 50 and early.sum() > 50
    assert not got["efeat"][late].any()
    np.testing.assert_array_equal(got["efeat"][early], full[got["eid"][early]])
    hop1 = o.sample(nodes[:20], tq[:20], want=("nbr",))["nbr"]
    g2 = o.sample_hop2(hop1, tq[:20], efeat=part, want=("efeat",))
    w2 = o.sample_hop2(hop1, tq[:20], efeat=padded, want=("efeat",))
    np.testing.assert_array_equal(g2["efeat"], w2["efeat"])


def test_theorem2_nlb_node_product_form():
    """Theorem 2 (NLB-node achieves recent node-wise sampling, App. B): when
    each neighbour v_j meets the centre node as an independent Poisson
    process of rate lambda_j, the latest link with v_i, entered at t_i, is
    still stored at t with probability
        prod_{j != i} ((s-1)/s + (1/s) exp(alpha lambda_j (t_i - t))),
    the average over neighbour ids of the slot collisions of eq. (3).  Away
    from the start an offer enters with probability alpha, so presence =
    alpha * that product."""
    alpha, s, T, H, M = 0.5, 10, 150.0, 300, 30
    scale = 1000.0
    pres, expect = [], []
    for rep in range(4):
        rng = np.random.default_rng(700 + rep)
        hub_l, nbr_l, time_l = [], [], []
        lam_all, ids_all = [], []
        for h in range(H):
            lam = rng.uniform(0.05, 0.3, M)
            ids = H + rng.choice(10**6, M, replace=False)
            lam_all.append(lam)
            ids_all.append(ids)
            for j in range(M):
                n = rng.poisson(lam[j] * T)
                time_l.append(rng.uniform(0, T, n))
                hub_l.append(np.full(n, h))
                nbr_l.append(np.full(n, ids[j]))
        times = np.concatenate(time_l)
        hubs = np.concatenate(hub_l)
        nbrs = np.concatenate(nbr_l)
        order = np.argsort(times, kind="stable")
        times, hubs, nbrs = times[order], hubs[order], nbrs[order]
        tt = np.floor(times * scale).astype(np.uint32)
        o = Oracle(H + 10**6, s, alpha, seed=1700 + rep, key_mode=1)
        o.insert(hubs.astype(np.int32), nbrs.astype(np.int32), tt)
        _, _, eid = o.export_nodes(np.arange(H, dtype=np.int32))
        stored = set(int(x) for x in eid[eid != 0xFFFFFFFF])
        # latest link of every (hub, neighbour) pair
        key = hubs.astype(np.int64) * (H + 10**6) + nbrs
        last = {}
        for e_, k_ in enumerate(key):
            last[k_] = e_
        for h in range(H):
            lam, ids = lam_all[h], ids_all[h]
            for j in range(M):
                k_ = h * (H + 10**6) + ids[j]
                if k_ not in last:
                    continue
                e_ = last[k_]
                ti = times[e_]
                if ti < 60.0:           # the table has long been full
                    continue
                d = T - ti
                others = np.delete(lam, j)
                p = np.prod((s - 1) / s + np.exp(-alpha * others * d) / s)
                pres.append(e_ in stored)
                expect.append(alpha * p)
    pres = np.array(pres)
    expect = np.array(expect)
    delta_order = np.argsort(expect)
    for chunk in np.array_split(delta_order, 8):
        mu = expect[chunk].sum()
        var = (expect[chunk] * (1 - expect[chunk])).sum()
        assert abs(pres[chunk].sum() - mu) < 5 * math.sqrt(var) + 1, (pres[chunk].sum(), mu)


def test_hop2_entries_are_neighbours_of_neighbours():
    """Sec. 4.4 second hop: every valid entry (i, a, c) is a stored link of
    the first-hop neighbour v = hop1[i, a], earlier than tq[i]; empty
    first-hop entries give empty second hops; rows follow the entries."""
    rng = np.random.default_rng(31)
    N, s, E = 60, 5, 3000
    src, dst, t = random_stream(rng, N, E, 10**5)
    o = Oracle(N, s, 0.5, seed=8)
    o.insert(src, dst, t)
    nfeat = rng.integers(0, 2**16, (N, 3)).astype(np.uint16)
    nodes = rng.integers(0, N, 200).astype(np.int32)
    tq = rng.integers(0, 10**5, 200).astype(np.uint32)
    first = o.sample(nodes, tq, want=("nbr",))["nbr"]
    out = o.sample_hop2(first, tq, nfeat=nfeat, want=("nbr", "eid", "ts", "nfeat", "self"))
    for i in range(200):
        for a in range(s):
            v = first[i, a]
            if v < 0:
                assert (out["nbr"][i, a] == -1).all() and not out["self"][i, a].any()
                continue
            np.testing.assert_array_equal(out["self"][i, a], nfeat[v])
            for c in range(s):
                x = out["nbr"][i, a, c]
                if x < 0:
                    continue
                e_ = out["eid"][i, a, c]
                assert {int(src[e_]), int(dst[e_])} == {int(v), int(x)}
                assert out["ts"][i, a, c] == t[e_] < tq[i]
                np.testing.assert_array_equal(out["nfeat"][i, a, c], nfeat[x])


# ----------------------------------------------------------------------------- eq. (4)
def _unit_weights(H, k1, k3):
    z = lambda *shape: np.zeros(shape, np.float32)
    return {"w1": z(H, k1), "b1": z(H), "w2": z(H, H), "b2": z(H), "att": z(H),
            "w3": z(H, k3), "b3": z(H), "w4": z(H, H), "b4": z(H)}


def _bits(wd):
    import synth
    return {k: (synth._to_bf16_bits(v) if k[0] == "w" else v) for k, v in wd.items()}


def test_aggregate_handworked_two_slots():
    """Eq. (4) by hand, H = 1: node 0 stores neighbours 1 (status 0) and 2
    (status 1).  MLP_in passes the status through (W1 = 1 on r_v, ReLU,
    W2 = 1) and the attention vector is 1, so the logits are 0 and 1 and
    alpha = (1, e)/(1+e); the aggregate is e/(1+e).  MLP_out computes
    ReLU(2*agg - 1) + 0.5 = tanh(1/2) + 0.5.  With no valid slot the
    aggregate is 0 and Z = 0 + 0.5."""
    o = Oracle(3, 2, 1.0, seed=0, q1=5, q2=2)
    o.insert([0, 0], [1, 2], [1, 2])          # slots (5+2)%2 = 1 and (10+4)%2 = 0
    nbr, _, _ = o.export()
    assert sorted(nbr[0].tolist()) == [1, 2]
    wd = _unit_weights(1, 64, 33)             # r_v in column 0, T-enc in column 32
    wd["w1"][0, 0] = 1.0
    wd["w2"][0, 0] = 1.0
    wd["att"][0] = 1.0
    wd["w3"][0, 32] = 2.0                     # coefficient of the aggregate
    wd["b3"][0] = -1.0
    wd["w4"][0, 0] = 1.0
    wd["b4"][0] = 0.5
    nfeat = np.array([[7.0], [0.0], [1.0]], np.float32)
    w = np.zeros(1, np.float32)
    b = np.zeros(1, np.float32)
    z = o.aggregate([0, 0], [5, 0], w, b, None, nfeat, _bits(wd))
    assert abs(z[0, 0] - (math.tanh(0.5) + 0.5)) < 1e-12
    assert z[1, 0] == 0.5


def test_aggregate_is_a_set_function():
    """Eq. (4) sums over the set S_u^t: two tables holding the same entries
    in different slots (different hash constants, no collisions) give the
    same Z."""
    import synth
    rng = np.random.default_rng(3)
    N, s, E = 400, 64, 120
    src = rng.integers(0, 20, E).astype(np.int32)
    dst = rng.integers(20, N, E).astype(np.int32)
    t = np.sort(rng.choice(10**6, E, replace=False)).astype(np.uint32)
    w = synth.scaled(synth.workload(3), 10)
    W = synth.agg_weights(w)
    nf = rng.integers(0, 2**15, (N, w.node_dim)).astype(np.uint16) & 0x3FFF   # finite bf16
    fw, fb = synth.time_params(w)
    zs, sets, slots = [], [], []
    for q1, q2 in ((1000000007, 998244353), (999999937, 1000000009 % (2**31))):
        o = Oracle(N, s, 1.0, seed=1, q1=q1, q2=q2)
        o.insert(src, dst, t)
        nbr, ts, eid = o.export_nodes(np.arange(20, dtype=np.int32))
        sets.append([sorted(e for e in row if e != 0xFFFFFFFF) for row in eid])
        slots.append(eid)
        zs.append(o.aggregate(np.arange(20), np.full(20, 10**6 + 1), fw, fb, None, nf, W))
    same = [i for i in range(20) if sets[0][i] == sets[1][i] and len(sets[0][i]) > 1
            and not np.array_equal(slots[0][i], slots[1][i])]
    assert len(same) >= 3
    np.testing.assert_allclose(zs[0][same], zs[1][same], rtol=1e-12, atol=1e-12)


def test_aggregate_constant_messages_ignore_attention():
    """With W2 = 0 every message is b2, so the attention weights do not
    matter: Z is the same for every query with at least one valid slot, and
    for queries without one it is MLP_out of a zero aggregate."""
    import synth
    rng = np.random.default_rng(4)
    N, s, E = 100, 8, 2000
    src, dst, t = random_stream(rng, N, E, 10**5)
    w = synth.scaled(synth.workload(1), 10)
    W = synth.agg_weights(w)
    W["w2"] = np.zeros_like(W["w2"])
    ef = rng.standard_normal((E, w.edge_dim)).astype(np.float32)
    fw, fb = synth.time_params(w)
    o = Oracle(N, s, 0.5, seed=2)
    o.insert(src, dst, t)
    q = rng.integers(0, N, 300).astype(np.int32)
    tq = rng.integers(0, 2 * 10**5, 300).astype(np.uint32)
    z = o.aggregate(q, tq, fw, fb, ef, None, W)
    any_valid = (o.sample(q, tq, want=("nbr",))["nbr"] >= 0).any(axis=1)
    assert any_valid.any() and (~any_valid).any()
    np.testing.assert_allclose(z[any_valid], np.broadcast_to(z[any_valid][0], z[any_valid].shape),
                               rtol=0, atol=1e-12)
    np.testing.assert_allclose(z[~any_valid], np.broadcast_to(z[~any_valid][0], z[~any_valid].shape),
                               rtol=0, atol=1e-12)
    assert np.abs(z[any_valid][0] - z[~any_valid][0]).max() > 1e-6


def test_aggregate_and_gru_take_zero_rows_past_the_link_table():
    """Eq. (4) and the status GRU see a link without a row in the (partial)
    link-feature table as a zero row: the same result as a zero-padded
    table."""
    import synth
    rng = np.random.default_rng(5)
    N, s, E = 100, 8, 2000
    src, dst, t = random_stream(rng, N, E, 10**5)
    w = synth.scaled(synth.workload(1), 10)
    W = synth.agg_weights(w)
    ef = rng.standard_normal((E, w.edge_dim)).astype(np.float32)
    keep = 1200
    padded = ef.copy()
    padded[keep:] = 0.0
    fw, fb = synth.time_params(w)
    o = Oracle(N, s, 0.5, seed=2)
    o.insert(src, dst, t)
    q = rng.integers(0, N, 200).astype(np.int32)
    tq = np.full(200, 2 * 10**5, np.uint32)
    z_part = o.aggregate(q, tq, fw, fb, ef[:keep], None, W)
    np.testing.assert_array_equal(z_part, o.aggregate(q, tq, fw, fb, padded, None, W))
    assert np.abs(z_part - o.aggregate(q, tq, fw, fb, ef, None, W)).max() > 1e-6
    d = 16
    G = synth.gru_weights_for(d, w.d_time, w.edge_dim, seed=7)
    st0 = rng.standard_normal((N, d)).astype(np.float32)
    lo = keep - 100
    a, b_ = st0.copy(), st0.copy()
    oracle.gru_update(a, src[lo:lo + 200], dst[lo:lo + 200], t[lo:lo + 200], lo, fw, fb, ef[:keep], G)
    oracle.gru_update(b_, src[lo:lo + 200], dst[lo:lo + 200], t[lo:lo + 200], lo, fw, fb, padded, G)
    np.testing.assert_array_equal(a, b_)
    c = st0.copy()
    oracle.gru_update(c, src[lo:lo + 200], dst[lo:lo + 200], t[lo:lo + 200], lo, fw, fb, ef, G)
    assert np.abs(a - c).max() > 1e-6


def _bf16_to_f64(bits):
    return (np.asarray(bits).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _pad_last(a, to):
    return np.concatenate([a, np.zeros(a.shape[:-1] + (to - a.shape[-1],))], axis=-1)


@pytest.mark.parametrize("heads", [1, 2, 4])
def test_aggregate_matches_library_attention_pooling(heads):
    """Eq. (4) rebuilt from library routines in float64 on the oracle's own
    sample outputs (pinned above): torch's F.linear for the four layers
    (weights [out][in], as the layouts state) and scaled_dot_product_attention
    with the attention vector as the single query, the messages as keys and
    values, scale 1 and the validity mask; a query without a valid slot
    aggregates the zero vector.  With several heads (App. E uses two), the
    library's multi-head layout: query, keys and values split into `heads`
    consecutive slices of the hidden width, one attention per slice, the
    outputs concatenated.  A transposed square weight, a dropped bias, a
    wrong mask, a wrong order of the input segments or a head scored over
    the wrong slice fails this."""
    import torch
    import torch.nn.functional as F
    import synth
    rng = np.random.default_rng(11)
    N, s, E = 300, 8, 3000
    src, dst, t = random_stream(rng, N, E, 10**5)
    w = synth.scaled(synth.workload(3), 10)            # bf16 link and node rows
    W = synth.agg_weights(w)
    ef = synth._to_bf16_bits(rng.standard_normal((E, w.edge_dim)).astype(np.float32))
    nf = synth._to_bf16_bits(rng.standard_normal((N, w.node_dim)).astype(np.float32))
    fw, fb = synth.time_params(w)
    o = Oracle(N, s, 0.5, seed=7)
    o.insert(src, dst, t)
    q = rng.integers(0, N, 400).astype(np.int32)
    tq = rng.integers(0, 2 * 10**5, 400).astype(np.uint32)
    tq[:5] = 0                                          # no entry is older than time 0
    # queries at the time of one of their node's stored entries: the strict
    # mask of eq. (1) leaves that entry out
    _, ts_q, _ = o.export_nodes(q[5:60])
    at_entry = 0
    for i, row in enumerate(ts_q):
        live = row[row != 0xFFFFFFFF]
        if len(live) >= 2:
            tq[5 + i] = live.max()
            at_entry += 1
    assert at_entry >= 20
    z = o.aggregate(q, tq, fw, fb, ef, nf, W, heads=heads)

    out = o.sample(q, tq, fw, fb, ef, nf)
    valid = out["nbr"] >= 0
    n_valid = valid.sum(axis=1)
    assert (n_valid == 0).sum() >= 5 and (n_valid >= 2).sum() > 300
    p32 = lambda d: (d + 31) // 32 * 32
    x = np.concatenate([_pad_last(_bf16_to_f64(out["nfeat"]), p32(w.node_dim)),
                        _pad_last(_bf16_to_f64(out["efeat"]), p32(w.edge_dim)),
                        _pad_last(out["tenc"].astype(np.float64), p32(w.d_time))], axis=-1)
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float64))
    Wt = {k: T(_bf16_to_f64(v) if k[0] == "w" and k != "att" else v.astype(np.float64))
          for k, v in W.items()}
    msg = F.linear(F.relu(F.linear(T(x), Wt["w1"], Wt["b1"])), Wt["w2"], Wt["b2"])   # [nq, s, H]
    nq, H = len(q), msg.shape[-1]
    kv = msg.reshape(nq, s, heads, H // heads).transpose(1, 2).contiguous()          # [nq, heads, s, H/heads]
    query = Wt["att"].reshape(1, heads, 1, H // heads).expand(nq, -1, -1, -1).contiguous()
    mask = torch.from_numpy(valid)[:, None, None, :]
    agg = F.scaled_dot_product_attention(query, kv, kv, attn_mask=mask, scale=1.0)   # [nq, heads, 1, H/heads]
    agg = agg[:, :, 0, :].reshape(nq, H).clone()
    agg[~torch.from_numpy(valid.any(axis=1))] = 0.0
    y = torch.cat([T(_pad_last(_bf16_to_f64(out["self"]), p32(w.node_dim))), agg], dim=-1)
    ref = F.linear(F.relu(F.linear(y, Wt["w3"], Wt["b3"])), Wt["w4"], Wt["b4"]).numpy()
    np.testing.assert_allclose(z, ref, rtol=1e-9, atol=1e-9)


# ----------------------------------------------------------------------------- status RNN (Sec. 4.4)
def _gru_zero(d, d_t, e_dim):
    kx = oracle_pad32(d) + oracle_pad32(d_t) + oracle_pad32(e_dim)
    return {"w_ih": np.zeros((3 * d, kx), np.uint16), "w_hh": np.zeros((3 * d, oracle_pad32(d)), np.uint16),
            "b_ih": np.zeros(3 * d, np.float32), "b_hh": np.zeros(3 * d, np.float32)}


def oracle_pad32(x):
    return (x + 31) // 32 * 32


def test_gru_handworked_bias_only():
    """d = 1, all weights zero: r = sigmoid(b_ir + b_hr), z = sigmoid(b_iz +
    b_hz) and n = tanh(b_in + r * b_hn), so the new status is (1 - z) n + z h.
    With b_iz = ln 3 (z = 3/4), b_ir = 0 (r = 1/2), b_in = 0 and b_hn =
    2 atanh(0.6) (n = 0.6): h' = 0.15 + 0.75 h.  Node 2 is not touched."""
    W = _gru_zero(1, 0, 0)
    W["b_ih"][1] = math.log(3.0)
    W["b_hh"][2] = 2.0 * math.atanh(0.6)
    st = np.array([[0.5], [-1.0], [4.0]], np.float32)
    oracle.gru_update(st, [0], [1], [7], 0, np.zeros(0, np.float32), np.zeros(0, np.float32), None, W)
    n = math.tanh(0.5 * np.float32(2.0 * math.atanh(0.6)))
    assert abs(st[0, 0] - (0.25 * n + 0.75 * 0.5)) < 1e-7
    assert abs(st[1, 0] - (0.25 * n - 0.75)) < 1e-7
    assert st[2, 0] == 4.0


def _gru_cell_reference(W, d, d_t, e_dim, x, h):
    """torch.nn.GRUCell in float64 with the given bf16 weights (pad columns
    dropped): the textbook GRU of a library."""
    import torch
    f = lambda bits: torch.from_numpy(bf16_to_f32(bits).astype(np.float64))
    w_ih = f(W["w_ih"])
    cols = list(range(d)) + [oracle_pad32(d) + c for c in range(d_t)] + \
        [oracle_pad32(d) + oracle_pad32(d_t) + c for c in range(e_dim)]
    cell = torch.nn.GRUCell(d + d_t + e_dim, d).double()
    with torch.no_grad():
        cell.weight_ih.copy_(w_ih[:, cols])
        cell.weight_hh.copy_(f(W["w_hh"])[:, :d])
        cell.bias_ih.copy_(torch.from_numpy(W["b_ih"].astype(np.float64)))
        cell.bias_hh.copy_(torch.from_numpy(W["b_hh"].astype(np.float64)))
        return cell(torch.from_numpy(x), torch.from_numpy(h)).numpy()


@pytest.mark.parametrize("edge_dtype", ["f32", "bf16"])
def test_gru_matches_library_gru_cell(edge_dtype):
    """Links with pairwise distinct endpoints: each endpoint's new status is
    torch's GRUCell (float64) on x = [r_other ; T-enc(t) ; e] with hidden
    state r_self, both endpoints reading pre-batch statuses.  The time
    weights are dyadic with few bits, so w * t is exact in fp32 and the
    fused argument w * t + b is one fp32 addition."""
    import synth
    rng = np.random.default_rng(21)
    N, d, d_t, e_dim, E = 64, 20, 12, 9, 16
    W = synth.gru_weights_for(d, d_t, e_dim, seed=3)
    perm = rng.permutation(N)[:2 * E]
    src, dst = perm[:E].astype(np.int32), perm[E:].astype(np.int32)
    t = np.sort(rng.integers(0, 2**20, E)).astype(np.uint32)
    st = rng.standard_normal((N, d)).astype(np.float32)
    ef32 = rng.standard_normal((E + 5, e_dim)).astype(np.float32)
    ef = synth._to_bf16_bits(ef32) if edge_dtype == "bf16" else ef32
    efv = bf16_to_f32(ef) if edge_dtype == "bf16" else ef32
    fw = (rng.integers(1, 16, d_t) * 2.0**-22).astype(np.float32)
    fb = rng.uniform(-3, 3, d_t).astype(np.float32)
    before = st.copy()
    oracle.gru_update(st, src, dst, t, 5, fw, fb, ef, W)   # link i uses row 5 + i
    arg = fw[None, :] * t[:, None].astype(np.float32) + fb[None, :]
    assert arg.dtype == np.float32
    te = np.cos(arg.astype(np.float64)).astype(np.float32).astype(np.float64)
    e = efv[5:5 + E].astype(np.float64)
    b64 = before.astype(np.float64)
    want_u = _gru_cell_reference(W, d, d_t, e_dim, np.concatenate([b64[dst], te, e], 1), b64[src])
    want_v = _gru_cell_reference(W, d, d_t, e_dim, np.concatenate([b64[src], te, e], 1), b64[dst])
    np.testing.assert_allclose(st[src], want_u.astype(np.float32), rtol=0, atol=2e-7)
    np.testing.assert_allclose(st[dst], want_v.astype(np.float32), rtol=0, atol=2e-7)
    untouched = np.setdiff1d(np.arange(N), perm[:2 * E])
    np.testing.assert_array_equal(st[untouched], before[untouched])


def bf16_to_f32(bits):
    return (np.asarray(bits, np.uint32) << 16).view(np.float32)


def test_gru_batch_reads_pre_batch_statuses_and_latest_link_wins():
    """Batch semantics of the status update: in one batch, link 0 (0, 1),
    link 1 (1, 2), link 2 (3, 0).  Node 1's final status is its update from
    link 1, node 0's from link 2, and both read the statuses from before the
    batch -- so each equals the single-link update applied to the initial
    statuses.  A self-loop (4, 4) gives the same status either way."""
    import synth
    rng = np.random.default_rng(5)
    N, d = 6, 40
    W = synth.gru_weights_for(d, 0, 0, seed=9)
    init = rng.standard_normal((N, d)).astype(np.float32)
    no = np.zeros(0, np.float32)
    batch = init.copy()
    oracle.gru_update(batch, [0, 1, 3, 4], [1, 2, 0, 4], [1, 2, 3, 4], 0, no, no, None, W)
    single = {}
    for i, (u, v) in enumerate([(0, 1), (1, 2), (3, 0), (4, 4)]):
        st = init.copy()
        oracle.gru_update(st, [u], [v], [i + 1], i, no, no, None, W)
        single[i] = st
    np.testing.assert_array_equal(batch[0], single[2][0])
    np.testing.assert_array_equal(batch[1], single[1][1])
    np.testing.assert_array_equal(batch[2], single[1][2])
    np.testing.assert_array_equal(batch[3], single[2][3])
    np.testing.assert_array_equal(batch[4], single[3][4])
    np.testing.assert_array_equal(batch[5], init[5])
    # sequential application would differ: link 1 would see node 1's new status
    seq = init.copy()
    for i, (u, v) in enumerate([(0, 1), (1, 2), (3, 0), (4, 4)]):
        oracle.gru_update(seq, [u], [v], [i + 1], i, no, no, None, W)
    assert np.abs(seq[2] - batch[2]).max() > 1e-4


def test_gru_bf16_status_rounds_to_nearest_even():
    """A bf16 status table stores the update rounded to nearest even (as
    torch's fp32 -> bf16 conversion); with d = 1 and zero weights the update
    is (1 - z) n + z h with n = 0.6, z = 3/4 (see the hand-worked case)."""
    import torch
    W = _gru_zero(1, 0, 0)
    W["b_ih"][1] = math.log(3.0)
    W["b_hh"][2] = 2.0 * math.atanh(0.6)
    no = np.zeros(0, np.float32)
    h = np.array([0.5, -1.0, 0.3125, 2.0], np.float32)
    st = np.ascontiguousarray(synth_bits(h)[:, None])
    oracle.gru_update(st, [0, 2], [1, 3], [1, 2], 0, no, no, None, W)
    n = math.tanh(0.5 * np.float32(2.0 * math.atanh(0.6)))
    exact = torch.tensor([0.25 * n + 0.75 * float(bf16_to_f32(synth_bits(np.array([x], np.float32)))[0])
                          for x in h], dtype=torch.float64)
    want = exact.float().bfloat16().view(torch.int16).numpy().astype(np.uint16)
    np.testing.assert_array_equal(st[:, 0], want)


def synth_bits(x):
    import synth
    return synth._to_bf16_bits(x)


def test_gru_rejects_out_of_range_endpoint():
    import synth
    W = synth.gru_weights_for(4, 0, 0, seed=1)
    st = np.zeros((3, 4), np.float32)
    no = np.zeros(0, np.float32)
    with pytest.raises(ValueError):
        oracle.gru_update(st, [0], [3], [1], 0, no, no, None, W)
    assert not st.any()
