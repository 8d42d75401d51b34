"""CPU oracle for NLB forward recent sampling (arXiv 2402.01964).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the CPU-baseline leg
of the benchmark use it to check the GPU library.  The product path never
imports it, and it imports nothing from the product package.

The arithmetic lives in ``nlb_oracle.c`` (plain C, one link at a time, in
stream order); this module only builds that file with gcc and wraps it with
ctypes and numpy.  Which passage of the paper each function follows is stated
in the C source:

* ``slot``      -- eq. (2) (NLB-edge) / eq. (3) (NLB-node), Sec. 4.2
* ``insert*``   -- replacement rule of Sec. 4.2 (empty slot: take; occupied:
                   replace with probability alpha), both endpoints updated
* ``sample``    -- eq. (1) strict ``t' < t`` mask; Sec. 4.4 retrieval of
                   neighbour, link-feature and self rows; App. C T-encoding
* ``sample_hop2`` -- Sec. 4.4 second-hop neighbours: S_v^t of each stored v
* ``aggregate`` -- eq. (4): attention over the retrieved neighbours, fp64
* ``gru_update`` -- Sec. 4.4 node-status RNN update after each event, fp64
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "nlb_oracle.c")
_LIB = os.path.join(_HERE, "libnlb_oracle.so")

DEFAULT_Q1 = 1000000007
DEFAULT_Q2 = 998244353


def build() -> str:
    """Compile the oracle with gcc (-O2, no fp contraction, no fast-math)."""
    cmd = ["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math",
           "-Wall", "-Wextra", "-shared", "-fPIC", "-o", _LIB + ".tmp", _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(_LIB + ".tmp", _LIB)
    return _LIB


_lib = None


def _load():
    """The built oracle; NLB_ORACLE_LIB names another build of nlb_oracle.c
    to load instead (the sanitizer build of tests/test_sanitizers.py)."""
    global _lib
    if _lib is not None:
        return _lib
    path = os.environ.get("NLB_ORACLE_LIB")
    if path is None:
        path = _LIB
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    i32, i64, u32, u64, dbl = (ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32,
                               ctypes.c_uint64, ctypes.c_double)
    lib.orc_create.restype = P
    lib.orc_create.argtypes = [i64, i32, dbl, u64, u64, u64, i32]
    lib.orc_create_subset.restype = P
    lib.orc_create_subset.argtypes = [i64, i32, dbl, u64, u64, u64, i32, P, i64]
    lib.orc_rows.restype = i64
    lib.orc_rows.argtypes = [P]
    lib.orc_destroy.argtypes = [P]
    lib.orc_threshold.restype = u64
    lib.orc_threshold.argtypes = [P]
    lib.orc_count.restype = u64
    lib.orc_count.argtypes = [P]
    lib.orc_slot.restype = u32
    lib.orc_slot.argtypes = [P, u32, u32]
    lib.orc_coin.restype = u32
    lib.orc_coin.argtypes = [P, u64, u32]
    lib.orc_insert_at.restype = ctypes.c_int
    lib.orc_insert_at.argtypes = [P, u64, i32, i32, u32]
    lib.orc_insert_batch.restype = ctypes.c_int
    lib.orc_insert_batch.argtypes = [P, P, P, P, i64]
    lib.orc_insert_ids.restype = ctypes.c_int
    lib.orc_insert_ids.argtypes = [P, P, P, P, P, i64]
    lib.orc_export.argtypes = [P, P, P, P]
    lib.orc_export_nodes.restype = ctypes.c_int
    lib.orc_export_nodes.argtypes = [P, P, i64, P, P, P]
    lib.orc_sample.restype = ctypes.c_int
    lib.orc_sample.argtypes = [P, P, P, i64, i32, P, P, P, i64, i64, P, i64,
                               P, P, P, P, P, P, P]
    lib.orc_sample_hop2.restype = ctypes.c_int
    lib.orc_sample_hop2.argtypes = [P, P, P, i64, i32, P, P, P, i64, i64, P, i64,
                                    P, P, P, P, P, P, P]
    lib.orc_aggregate.restype = ctypes.c_int
    lib.orc_aggregate.argtypes = [P, P, P, i64, i32, P, P, P, i64, i32, i32, P, i32, i32, i32, i32,
                                  P, P, P, P, P, P, P, P, P, P]
    lib.orc_gru_update.restype = ctypes.c_int
    lib.orc_gru_update.argtypes = [i64, i32, P, i32, P, P, P, i64, u64, i32, P, P, P, i64, i32, i32,
                                   P, P, P, P]
    lib.orc_tenc.argtypes = [P, i64, i32, P, P, P]
    _lib = lib
    return lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


class Oracle:
    """Sequential NLB tables for ``num_nodes`` nodes with ``s`` slots each.

    ``keep``: optional node ids whose tables are kept; offers to every other
    table are dropped.  Tables are per node (Sec. 4.2), so the kept tables
    are exactly those of the full structure; queries and exports must name
    kept nodes."""

    def __init__(self, num_nodes: int, s: int, alpha: float, seed: int,
                 q1: int = DEFAULT_Q1, q2: int = DEFAULT_Q2, key_mode: int = 0, keep=None):
        lib = _load()
        self._lib = lib
        self.N, self.s, self.alpha, self.seed = int(num_nodes), int(s), float(alpha), int(seed)
        self.key_mode = int(key_mode)
        self.subset = keep is not None
        if keep is None:
            self._h = lib.orc_create(self.N, self.s, self.alpha, self.seed & (2**64 - 1),
                                     int(q1), int(q2), self.key_mode)
        else:
            keep = _c(keep, np.int32)
            self._h = lib.orc_create_subset(self.N, self.s, self.alpha, self.seed & (2**64 - 1),
                                            int(q1), int(q2), self.key_mode, _ptr(keep), len(keep))
        if not self._h:
            raise ValueError("oracle: invalid parameters or out of memory")

    def close(self):
        if self._h:
            self._lib.orc_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def threshold(self) -> int:
        return int(self._lib.orc_threshold(self._h))

    @property
    def rows(self) -> int:
        return int(self._lib.orc_rows(self._h))

    @property
    def count(self) -> int:
        return int(self._lib.orc_count(self._h))

    def slot(self, x: int, t: int) -> int:
        return int(self._lib.orc_slot(self._h, x, t))

    def coin(self, e: int, k: int) -> int:
        return int(self._lib.orc_coin(self._h, e, k))

    def insert(self, src, dst, t):
        src, dst, t = _c(src, np.int32), _c(dst, np.int32), _c(t, np.uint32)
        if self._lib.orc_insert_batch(self._h, _ptr(src), _ptr(dst), _ptr(t), len(src)) != 0:
            raise ValueError("oracle: node id out of range")

    def insert_ids(self, eids, src, dst, t):
        eids = _c(eids, np.uint64)
        src, dst, t = _c(src, np.int32), _c(dst, np.int32), _c(t, np.uint32)
        if self._lib.orc_insert_ids(self._h, _ptr(eids), _ptr(src), _ptr(dst), _ptr(t),
                                    len(src)) != 0:
            raise ValueError("oracle: node id out of range")

    def export(self):
        """Canonical table: (nbr int32, ts uint32, eid uint32), each [N, s]."""
        if self.subset:
            raise ValueError("oracle keeps a node subset: use export_nodes")
        n = self.N * self.s
        nbr = np.empty(n, np.int32)
        ts = np.empty(n, np.uint32)
        eid = np.empty(n, np.uint32)
        self._lib.orc_export(self._h, _ptr(nbr), _ptr(ts), _ptr(eid))
        return nbr.reshape(self.N, self.s), ts.reshape(self.N, self.s), eid.reshape(self.N, self.s)

    def export_nodes(self, nodes):
        nodes = _c(nodes, np.int32)
        c = len(nodes)
        nbr = np.empty((c, self.s), np.int32)
        ts = np.empty((c, self.s), np.uint32)
        eid = np.empty((c, self.s), np.uint32)
        if self._lib.orc_export_nodes(self._h, _ptr(nodes), c, _ptr(nbr), _ptr(ts), _ptr(eid)) != 0:
            raise ValueError("oracle: node out of range or its table is not kept")
        return nbr, ts, eid

    def sample(self, node, tq, w=None, b=None, efeat=None, nfeat=None,
               want=("nbr", "eid", "ts", "tenc", "efeat", "nfeat", "self")):
        """Answer queries; returns a dict of numpy outputs (see nlb_oracle.c).

        ``efeat``/``nfeat`` are 2-D arrays of any dtype (rows are copied as
        bytes); outputs keep that dtype.  A stored link whose arrival index
        is not below ``len(efeat)`` gathers a zero row.
        """
        node, tq = _c(node, np.int32), _c(tq, np.uint32)
        nq, s = len(node), self.s
        d_t = 0 if w is None else len(w)
        w = None if w is None else _c(w, np.float32)
        b = None if b is None else _c(b, np.float32)
        out = {}
        if "nbr" in want:
            out["nbr"] = np.empty((nq, s), np.int32)
        if "eid" in want:
            out["eid"] = np.empty((nq, s), np.uint32)
        if "ts" in want:
            out["ts"] = np.empty((nq, s), np.uint32)
        if "tenc" in want and d_t > 0:
            out["tenc"] = np.empty((nq, s, d_t), np.float32)
        erb = nrb = erows = 0
        if efeat is not None:
            efeat = np.ascontiguousarray(efeat)
            erb, erows = efeat.shape[1] * efeat.itemsize, efeat.shape[0]
            if "efeat" in want:
                out["efeat"] = np.empty((nq, s, efeat.shape[1]), efeat.dtype)
        if nfeat is not None:
            nfeat = np.ascontiguousarray(nfeat)
            nrb = nfeat.shape[1] * nfeat.itemsize
            if "nfeat" in want:
                out["nfeat"] = np.empty((nq, s, nfeat.shape[1]), nfeat.dtype)
            if "self" in want:
                out["self"] = np.empty((nq, nfeat.shape[1]), nfeat.dtype)
        rc = self._lib.orc_sample(
            self._h, _ptr(node), _ptr(tq), nq, d_t, _ptr(w), _ptr(b),
            _ptr(efeat), erows, erb, _ptr(nfeat), nrb,
            _ptr(out.get("nbr")), _ptr(out.get("eid")), _ptr(out.get("ts")),
            _ptr(out.get("tenc")), _ptr(out.get("efeat")), _ptr(out.get("nfeat")),
            _ptr(out.get("self")))
        if rc != 0:
            raise ValueError("oracle: query node out of range")
        return out


    def sample_hop2(self, hop1_nbr, tq, w=None, b=None, efeat=None, nfeat=None,
                    want=("nbr", "eid", "ts", "tenc", "efeat", "nfeat", "self")):
        """Second-hop retrieval (Sec. 4.4): for every first-hop entry
        (i, a) with neighbour v = hop1_nbr[i, a] >= 0, the answer to query
        (v, tq[i]); empty entries (-1) give empty answers.  Outputs are shaped
        [nq, s, s, ...] (self: [nq, s, ...])."""
        hop1 = _c(hop1_nbr, np.int32).reshape(-1)
        tq = _c(tq, np.uint32)
        nq, s = len(tq), self.s
        assert len(hop1) == nq * s
        d_t = 0 if w is None else len(w)
        w = None if w is None else _c(w, np.float32)
        b = None if b is None else _c(b, np.float32)
        out = {}
        if "nbr" in want:
            out["nbr"] = np.empty((nq, s, s), np.int32)
        if "eid" in want:
            out["eid"] = np.empty((nq, s, s), np.uint32)
        if "ts" in want:
            out["ts"] = np.empty((nq, s, s), np.uint32)
        if "tenc" in want and d_t > 0:
            out["tenc"] = np.empty((nq, s, s, d_t), np.float32)
        erb = nrb = erows = 0
        if efeat is not None:
            efeat = np.ascontiguousarray(efeat)
            erb, erows = efeat.shape[1] * efeat.itemsize, efeat.shape[0]
            if "efeat" in want:
                out["efeat"] = np.empty((nq, s, s, efeat.shape[1]), efeat.dtype)
        if nfeat is not None:
            nfeat = np.ascontiguousarray(nfeat)
            nrb = nfeat.shape[1] * nfeat.itemsize
            if "nfeat" in want:
                out["nfeat"] = np.empty((nq, s, s, nfeat.shape[1]), nfeat.dtype)
            if "self" in want:
                out["self"] = np.empty((nq, s, nfeat.shape[1]), nfeat.dtype)
        rc = self._lib.orc_sample_hop2(
            self._h, _ptr(hop1), _ptr(tq), nq, d_t, _ptr(w), _ptr(b),
            _ptr(efeat), erows, erb, _ptr(nfeat), nrb,
            _ptr(out.get("nbr")), _ptr(out.get("eid")), _ptr(out.get("ts")),
            _ptr(out.get("tenc")), _ptr(out.get("efeat")), _ptr(out.get("nfeat")),
            _ptr(out.get("self")))
        if rc != 0:
            raise ValueError("oracle: first-hop neighbour out of range")
        return out


    def aggregate(self, node, tq, w, b, efeat, nfeat, weights, heads=1):
        """Eq. (4) attention aggregation (forward, fp64) for queries
        (node[i], tq[i]); ``weights`` holds w1, b1, w2, b2, att, w3, b3, w4, b4
        (bf16 matrices as uint16 bits in the padded layouts of
        nlb_oracle.c).  ``efeat``/``nfeat``: 2-D float32 or bf16-bits (uint16)
        arrays or None.  ``heads`` attention heads, each over its own slice
        of MLP_in's outputs (App. E uses two).  Returns z [nq, H] (float64)."""
        node, tq = _c(node, np.int32), _c(tq, np.uint32)
        w, b = _c(w, np.float32), _c(b, np.float32)
        H = int(weights["b1"].shape[0])

        def feat(a):
            if a is None:
                return None, 0, 1
            a = np.ascontiguousarray(a)
            return a, a.shape[1], (0 if a.dtype == np.float32 else 1)
        erows = 0 if efeat is None else int(np.shape(efeat)[0])
        ef, e_dim, e_dt = feat(efeat)
        nf, n_dim, n_dt = feat(nfeat)
        W = {k: np.ascontiguousarray(weights[k], np.uint16 if k[0] == "w" and k != "att" else np.float32)
             for k in ("w1", "b1", "w2", "b2", "att", "w3", "b3", "w4", "b4")}
        z = np.empty((len(node), H), np.float64)
        rc = self._lib.orc_aggregate(
            self._h, _ptr(node), _ptr(tq), len(node), len(w), _ptr(w), _ptr(b),
            _ptr(ef), erows, e_dim, e_dt, _ptr(nf), n_dim, n_dt, H, int(heads),
            _ptr(W["w1"]), _ptr(W["b1"]), _ptr(W["w2"]), _ptr(W["b2"]), _ptr(W["att"]),
            _ptr(W["w3"]), _ptr(W["b3"]), _ptr(W["w4"]), _ptr(W["b4"]), _ptr(z))
        if rc == -2:
            raise ValueError("oracle: heads must divide the hidden width")
        if rc != 0:
            raise ValueError("oracle: query node out of range")
        return z


def gru_update(status, src, dst, t, e0, w, b, efeat, weights):
    """Node-status update of Sec. 4.4 (GRU, batch semantics: updates read
    the statuses from before the batch, the latest link of a node wins), in
    place on ``status`` ([N, d] float32, or uint16 bf16 bits).  ``weights``:
    w_ih, w_hh (uint16 bf16 bits, padded layouts of nlb_oracle.c), b_ih, b_hh
    (float32).  ``efeat``: [E, e_dim] float32 / bf16 bits, or None."""
    lib = _load()
    assert status.flags.c_contiguous
    src, dst, t = _c(src, np.int32), _c(dst, np.int32), _c(t, np.uint32)
    w, b = _c(w, np.float32), _c(b, np.float32)
    s_dt = 0 if status.dtype == np.float32 else 1
    if efeat is None:
        ef, e_rows, e_dim, e_dt = None, 0, 0, 1
    else:
        ef = np.ascontiguousarray(efeat)
        e_rows, e_dim, e_dt = ef.shape[0], ef.shape[1], (0 if ef.dtype == np.float32 else 1)
    W = {k: np.ascontiguousarray(weights[k], np.uint16 if k.startswith("w_") else np.float32)
         for k in ("w_ih", "w_hh", "b_ih", "b_hh")}
    rc = lib.orc_gru_update(status.shape[0], status.shape[1], _ptr(status), s_dt, _ptr(src), _ptr(dst),
                            _ptr(t), len(src), int(e0), len(w), _ptr(w), _ptr(b), _ptr(ef), e_rows, e_dim, e_dt,
                            _ptr(W["w_ih"]), _ptr(W["w_hh"]), _ptr(W["b_ih"]), _ptr(W["b_hh"]))
    if rc != 0:
        raise ValueError("oracle: node id out of range")
    return status


def tenc(dt, w, b):
    """T-encoding of gaps ``dt`` (fp32) -> [len(dt), len(w)] fp32."""
    lib = _load()
    dt, w, b = _c(dt, np.float32), _c(w, np.float32), _c(b, np.float32)
    out = np.empty((len(dt), len(w)), np.float32)
    lib.orc_tenc(_ptr(dt), len(dt), len(w), _ptr(w), _ptr(b), _ptr(out))
    return out


def run_stream(oracle: Oracle, src, dst, t, neg, batch, w=None, b=None, efeat=None,
               nfeat=None, batches=None, want=("nbr", "eid", "ts", "tenc", "efeat", "nfeat", "self")):
    """Drive the oracle over a stream in batches (Sec. 4.2 timing: the queries
    of a batch -- both endpoints and one negative, all at the link's time --
    are answered from the tables as they stand before the batch is inserted).

    Yields ``(batch_index, outputs)`` for the batches in ``batches`` (all when
    None); every batch is inserted either way.
    """
    E = len(src)
    nb = (E + batch - 1) // batch
    wanted = None if batches is None else set(int(x) for x in batches)
    for bi in range(nb):
        lo, hi = bi * batch, min(E, (bi + 1) * batch)
        if wanted is None or bi in wanted:
            node = np.concatenate([src[lo:hi], dst[lo:hi], neg[lo:hi]])
            tq = np.concatenate([t[lo:hi], t[lo:hi], t[lo:hi]])
            yield bi, oracle.sample(node, tq, w, b, efeat, nfeat, want=want)
        oracle.insert(src[lo:hi], dst[lo:hi], t[lo:hi])
