"""Seeded synthetic workloads for NLB forward recent sampling.

Input generation only (no part of the sampling method): the five workload
shapes, their link streams, feature tables and time-encoding parameters.
Streams and features are counter-based functions of (seed, index) computed
by ``csrc/synth.hip`` with integer arithmetic and host-built lookup tables, so
the host copy handed to the CPU oracle and the device copy handed to the GPU
library are bit-identical without either being derived from the other.

Workloads (stand-ins, by shape, for the paper's datasets, which are not
available here):
  1 tiny-bipartite      1 000 nodes (200 src / 800 dst), 20 000 links, Zipf(1.2)
                        per side, t sorted in [0, 1e6], s=10, alpha=0.5, batch 200,
                        fp32 edge features 100-dim
  2 small-bipartite     11 000 nodes (10 000 src / 1 000 dst), 700 000 links,
                        Zipf(1.1) per side, 30% repeats of a prior partner, t sorted
                        over [0, 2.7e6], s=20, alpha=0.5, batch 600, fp32 edge 172-dim
  3 medium-homogeneous  100 000 nodes, 10M links, Chung-Lu endpoints with degree
                        exponent 2.1, bursty Markov-modulated Poisson time, s=64,
                        alpha=0.3, batch 4 000, bf16 edge 128-dim and node 128-dim
  4 dense-repeated      17 000 nodes, 200M links, 80% from a fixed set of 2M pairs,
                        t in integer minutes over 2 years, s=10, alpha=0.5, batch
                        10 000, bf16 edge 186-dim
  5 large-sparse        120M nodes, 1.3B links, Zipf(1.05), t in [0, 1e8], s=10,
                        alpha=0.5, batch 100 000, bf16 node 128-dim, no edge features
All use a 100-dim time encoding; queries per link are its two endpoints and one
uniform negative (destination side for bipartite streams, any node otherwise),
all at the link's timestamp.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
import subprocess
from functools import lru_cache

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "csrc", "synth.hip")
LIB_PATH = os.path.join(_HERE, "libnlbsynth.so")


@dataclasses.dataclass(frozen=True)
class Workload:
    key: int
    name: str
    num_nodes: int
    links: int
    s: int
    alpha: float
    batch: int
    kind: int                 # 0 bipartite, 1 homogeneous power law, 2 pair set
    n_src: int                # bipartite: source side size; else num_nodes
    n_dst: int
    exponent: float           # Zipf exponent of endpoint popularity
    T: int                    # timestamps in [0, T)
    d_time: int = 100
    edge_dim: int = 0
    edge_dtype: str = "f32"
    node_dim: int = 0
    node_dtype: str = "bf16"
    repeat: float = 0.0       # workload 2
    bursty: bool = False      # workload 3
    n_pairs: int = 0          # workload 4
    p_pair: float = 0.0
    table_seed: int = 42

    @property
    def stream_seed(self):
        return 1000 + self.key

    @property
    def edge_seed(self):
        return 2000 + self.key

    @property
    def node_seed(self):
        return 3000 + self.key

    @property
    def time_seed(self):
        return 4000 + self.key

    @property
    def batches(self):
        return (self.links + self.batch - 1) // self.batch

    @property
    def stateless(self):
        """True when every link is a pure function of its index (the device
        can generate the stream itself)."""
        return self.repeat == 0.0 and not self.bursty

    def elem_bytes(self, which):
        dt = self.edge_dtype if which == "edge" else self.node_dtype
        return 4 if dt == "f32" else 2

    def row_bytes(self, which):
        d = self.edge_dim if which == "edge" else self.node_dim
        return d * self.elem_bytes(which)

    def batch_range(self, b):
        lo = b * self.batch
        return lo, min(self.links, lo + self.batch)


WORKLOADS = {
    1: Workload(1, "tiny-bipartite", 1000, 20000, 10, 0.5, 200, 0, 200, 800, 1.2, 1_000_001,
                edge_dim=100, edge_dtype="f32"),
    2: Workload(2, "small-bipartite", 11000, 700_000, 20, 0.5, 600, 0, 10000, 1000, 1.1, 2_700_001,
                edge_dim=172, edge_dtype="f32", repeat=0.3),
    3: Workload(3, "medium-homogeneous", 100_000, 10_000_000, 64, 0.3, 4000, 1, 100_000, 0,
                1.0 / 1.1, 0, edge_dim=128, edge_dtype="bf16", node_dim=128, node_dtype="bf16",
                bursty=True),
    4: Workload(4, "dense-repeated", 17000, 200_000_000, 10, 0.5, 10000, 2, 17000, 0, 0.0,
                1_051_200, edge_dim=186, edge_dtype="bf16", n_pairs=2_000_000, p_pair=0.8),
    5: Workload(5, "large-sparse", 120_000_000, 1_300_000_000, 10, 0.5, 100_000, 1, 120_000_000, 0,
                1.05, 100_000_001, node_dim=128, node_dtype="bf16"),
}


def workload(key) -> Workload:
    return WORKLOADS[int(key)]


def scaled(w: Workload, links: int, num_nodes: int | None = None) -> Workload:
    """Same shape with fewer links (and optionally nodes), for quick checks."""
    kw = dict(links=int(links))
    if num_nodes is not None and w.kind != 0:
        kw.update(num_nodes=int(num_nodes), n_src=int(num_nodes))
    if w.n_pairs:
        kw["n_pairs"] = max(1, int(w.n_pairs * links / w.links))
    if w.T and w.kind != 0:
        kw["T"] = max(2, int(w.T * links / w.links))
    return dataclasses.replace(w, **kw)


# ----------------------------------------------------------------------------- build / load
def build() -> str:
    hipcc = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")
    cmd = [hipcc, "-O3", "-std=c++17", "--offload-arch=gfx950", "-fPIC", "-shared",
           "-ffp-contract=off", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-pthread", "-o", LIB_PATH + ".tmp", _SRC]
    subprocess.run(cmd, check=True)
    os.replace(LIB_PATH + ".tmp", LIB_PATH)
    return LIB_PATH


class _SynStream(ctypes.Structure):
    _fields_ = [("seed", ctypes.c_uint64), ("E", ctypes.c_int64), ("kind", ctypes.c_int32),
                ("neg_all", ctypes.c_int32), ("n_src", ctypes.c_int64), ("n_dst", ctypes.c_int64),
                ("T", ctypes.c_uint64), ("a_prob", ctypes.c_void_p), ("a_alias", ctypes.c_void_p),
                ("b_prob", ctypes.c_void_p), ("b_alias", ctypes.c_void_p),
                ("n_pairs", ctypes.c_int64), ("p_pair", ctypes.c_uint32), ("pad", ctypes.c_int32)]


_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: run synth.build()")
    # bind to torch's HIP runtime (same soname as the system one): one runtime per process
    import torch  # noqa: F401
    lib = ctypes.CDLL(LIB_PATH)
    P, I64, I32, U32, U64, D = (ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_uint32,
                                ctypes.c_uint64, ctypes.c_double)
    S = ctypes.POINTER(_SynStream)
    lib.syn_alias_powerlaw.argtypes = [I64, D, P, P]
    lib.syn_links_host.argtypes = [S, I64, I64, P, P, P, P, ctypes.c_int]
    lib.syn_links_device.argtypes = [S, I64, I64, I64, P, P, P]
    lib.syn_apply_repeats_host.argtypes = [U64, I64, I64, U32, P, P]
    lib.syn_bursty_times_host.argtypes = [U64, I64, D, D, D, D, P]
    lib.syn_features_host.argtypes = [U64, P, I64, U32, U32, P, P, ctypes.c_int]
    lib.syn_features_device.argtypes = [U64, I64, U32, U32, P, P, P]
    for f in ("syn_alias_powerlaw", "syn_links_host", "syn_links_device", "syn_apply_repeats_host",
              "syn_bursty_times_host", "syn_features_host", "syn_features_device"):
        getattr(lib, f).restype = ctypes.c_int
    _lib = lib
    return lib


def _p(a):
    return ctypes.c_void_p(a.ctypes.data)


def host_threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


# ----------------------------------------------------------------------------- tables
@lru_cache(maxsize=8)
def alias_table(n: int, exponent: float):
    """Alias table of popularity weights (k+1)^-exponent over ranks k < n."""
    prob = np.empty(n, np.uint32)
    alias = np.empty(n, np.int32)
    if _load().syn_alias_powerlaw(int(n), float(exponent), _p(prob), _p(alias)) != 0:
        raise ValueError("alias table")
    return prob, alias


@lru_cache(maxsize=1)
def normal_quantiles():
    """fp32 and bf16 tables of the standard-normal quantiles at (i+0.5)/65536."""
    from scipy.special import ndtri
    q = ndtri((np.arange(65536, dtype=np.float64) + 0.5) / 65536.0).astype(np.float32)
    bits = q.view(np.uint32).astype(np.uint64)
    bf = ((bits + 0x7FFF + ((bits >> 16) & 1)) >> 16).astype(np.uint16)  # round to nearest even
    return q, bf


def _stream_struct(w: Workload, tables):
    st = _SynStream()
    st.seed, st.E, st.kind = w.stream_seed, w.links, w.kind
    st.neg_all = 0 if w.kind == 0 else 1
    st.n_src, st.n_dst = w.n_src, w.n_dst
    st.T = w.T if w.T else 1
    (ap, aa), (bp, ba) = tables
    st.a_prob, st.a_alias = ap, aa
    st.b_prob, st.b_alias = bp, ba
    st.n_pairs = w.n_pairs
    st.p_pair = int(w.p_pair * 2**32) if w.p_pair else 0
    return st


def _host_tables(w: Workload):
    a = b = (np.zeros(1, np.uint32), np.zeros(1, np.int32))
    if w.kind in (0, 1):
        a = alias_table(w.n_src, w.exponent)
    if w.kind == 0:
        b = alias_table(w.n_dst, w.exponent)
    return a, b


# ----------------------------------------------------------------------------- streams
def host_links(w: Workload, i0: int = 0, i1: int | None = None, threads: int | None = None,
               out=None):
    """Links [i0, i1) as numpy (src, dst, t, neg).  Stateful workloads (2, 3)
    are only generated whole.  ``out``: four contiguous arrays of i1 - i0
    elements (int32, int32, uint32 or int32 bits, int32) to write into, e.g.
    views of pinned host memory."""
    i1 = w.links if i1 is None else int(i1)
    if not w.stateless and (i0 != 0 or i1 != w.links):
        raise ValueError("workloads with repeats or bursty time are generated whole")
    lib = _load()
    a, b = _host_tables(w)
    st = _stream_struct(w, ((_p(a[0]), _p(a[1])), (_p(b[0]), _p(b[1]))))
    n = i1 - i0
    if out is None:
        src, dst, neg = (np.empty(n, np.int32) for _ in range(3))
        t = np.empty(n, np.uint32)
    else:
        src, dst, t, neg = out
        for x in out:
            if len(x) != n or x.itemsize != 4 or not x.flags.c_contiguous:
                raise ValueError("out: four contiguous 4-byte arrays of the range's length")
    lib.syn_links_host(ctypes.byref(st), i0, i1, _p(src), _p(dst), _p(t), _p(neg),
                       threads or host_threads())
    if w.repeat:
        lib.syn_apply_repeats_host(w.stream_seed, n, w.n_src, int(w.repeat * 2**32), _p(src), _p(dst))
    if w.bursty:
        # normal gaps mean 10, bursts mean 0.1; switch 0.01 into and 0.05 out of bursts
        lib.syn_bursty_times_host(w.stream_seed, n, 10.0, 0.1, 0.01, 0.05, _p(t))
    return src, dst, t, neg


def blocked(w: Workload, src, dst, t, neg):
    """Batch-blocked query layout: batch b holds [src | dst | neg] of its links
    (nodes) and [t | t | t] (timestamps)."""
    E, B = len(src), w.batch
    nodes = np.empty(3 * E, np.int32)
    ts = np.empty(3 * E, np.uint32)
    for lo in range(0, E, B):
        hi = min(E, lo + B)
        n = hi - lo
        base = 3 * lo
        for k, arr in enumerate((src, dst, neg)):
            nodes[base + k * n: base + (k + 1) * n] = arr[lo:hi]
            ts[base + k * n: base + (k + 1) * n] = t[lo:hi]
    return nodes, ts


def device_links(w: Workload, device="cuda"):
    """The whole stream on the device in the batch-blocked layout: int32
    tensors ``nodes`` and ``ts`` of 3*E entries (ts holds uint32 values)."""
    import torch
    dev = torch.device(device)
    if not w.stateless:
        nodes, ts = blocked(w, *host_links(w))
        return (torch.from_numpy(nodes).to(dev), torch.from_numpy(ts.view(np.int32)).to(dev))
    lib = _load()
    a, b = _host_tables(w)
    keep = [torch.from_numpy(x.view(np.int32)).to(dev) for x in (a[0], a[1], b[0], b[1])]
    st = _stream_struct(w, ((keep[0].data_ptr(), keep[1].data_ptr()),
                            (keep[2].data_ptr(), keep[3].data_ptr())))
    nodes = torch.empty(3 * w.links, dtype=torch.int32, device=dev)
    ts = torch.empty(3 * w.links, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    chunk = 1 << 28
    for i0 in range(0, w.links, chunk):
        rc = lib.syn_links_device(ctypes.byref(st), i0, min(w.links, i0 + chunk), w.batch,
                                  ctypes.c_void_p(nodes.data_ptr()), ctypes.c_void_p(ts.data_ptr()),
                                  ctypes.c_void_p(stream))
        if rc != 0:
            raise RuntimeError("device stream generation failed")
    torch.cuda.synchronize(dev)
    del keep
    return nodes, ts


def batch_views(w: Workload, nodes, ts, b):
    """(src, dst, t, queries, tq) views of batch b in the blocked layout."""
    lo, hi = w.batch_range(b)
    n = hi - lo
    base = 3 * lo
    q = nodes[base: base + 3 * n]
    tq = ts[base: base + 3 * n]
    return q[:n], q[n:2 * n], tq[:n], q, tq


# ----------------------------------------------------------------------------- features
def feature_spec(w: Workload, which: str):
    dim = w.edge_dim if which == "edge" else w.node_dim
    rows = w.links if which == "edge" else w.num_nodes
    seed = w.edge_seed if which == "edge" else w.node_seed
    return dim, rows, seed, w.elem_bytes(which)


def host_feature_rows(w: Workload, which: str, rows):
    """Rows of the edge or node feature table: float32, or uint16 bf16 bits."""
    dim, _, seed, eb = feature_spec(w, which)
    rows = np.ascontiguousarray(rows, np.int64)
    q32, qbf = normal_quantiles()
    table = q32 if eb == 4 else qbf
    out = np.empty((len(rows), dim), np.float32 if eb == 4 else np.uint16)
    _load().syn_features_host(seed, _p(rows), len(rows), dim, eb, _p(table), _p(out), host_threads())
    return out


def host_features(w: Workload, which: str):
    _, rows, _, _ = feature_spec(w, which)
    return host_feature_rows(w, which, np.arange(rows))


def device_features(w: Workload, which: str, device="cuda"):
    """The whole feature table filled on the device (fp32 or bf16 tensor)."""
    import torch
    dim, rows, seed, eb = feature_spec(w, which)
    if dim == 0:
        return None
    dev = torch.device(device)
    q32, qbf = normal_quantiles()
    table = torch.from_numpy(q32 if eb == 4 else qbf.view(np.int16)).to(dev)
    out = torch.empty((rows, dim), dtype=torch.float32 if eb == 4 else torch.bfloat16, device=dev)
    rc = _load().syn_features_device(seed, rows, dim, eb, ctypes.c_void_p(table.data_ptr()),
                                     ctypes.c_void_p(out.data_ptr()),
                                     ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream))
    if rc != 0:
        raise RuntimeError("device feature fill failed")
    torch.cuda.synchronize(dev)
    return out


def time_params(w: Workload):
    """Time-encoding frequencies w_k = 10^(-9k/(d-1)) (log-spaced, in the
    style of the T-encoding line of work) and phases b_k ~ U[-pi, pi)."""
    d = w.d_time
    k = np.arange(d, dtype=np.float64)
    freq = (10.0 ** (-9.0 * k / max(d - 1, 1))).astype(np.float32)
    rng = np.random.default_rng(w.time_seed)
    phase = rng.uniform(-np.pi, np.pi, d).astype(np.float32)
    return freq, phase


# ----------------------------------------------------------------------------- eq. (4) weights
AGG_HIDDEN = 64


def _pad32(d):
    return (d + 31) // 32 * 32


def _to_bf16_bits(x):
    bits = np.ascontiguousarray(x, np.float32).view(np.uint32).astype(np.uint64)
    return ((bits + 0x7FFF + ((bits >> 16) & 1)) >> 16).astype(np.uint16)   # nearest even


def agg_weights(w: Workload, hidden: int = AGG_HIDDEN, seed: int | None = None):
    """Random weights of the attention aggregation of eq. (4): bf16 matrices
    (uint16 bits) in the padded layouts the library and the oracle take --
    w1 [H][pad32(node_dim) + pad32(edge_dim) + pad32(d_time)] for (r_v | e |
    T-enc), w2 [H][H], w3 [H][pad32(node_dim) + H] for (r_u | aggregate),
    w4 [H][H] -- with zero pad columns; fp32 biases and attention vector.
    Entries ~ N(0, 1/fan_in), biases ~ U(-0.1, 0.1)."""
    rng = np.random.default_rng(5000 + w.key if seed is None else seed)
    H, dn, de, dt = hidden, w.node_dim, w.edge_dim, w.d_time

    def dense(rows, segs):
        fan = sum(segs)
        out = np.zeros((rows, sum(_pad32(s) for s in segs)), np.float32)
        col = 0
        for sgl in segs:
            out[:, col:col + sgl] = rng.normal(0.0, 1.0 / np.sqrt(max(fan, 1)), (rows, sgl))
            col += _pad32(sgl)
        return _to_bf16_bits(out)

    def vec(n, lo=-0.1, hi=0.1):
        return rng.uniform(lo, hi, n).astype(np.float32)
    return {"w1": dense(H, [dn, de, dt]), "b1": vec(H), "w2": dense(H, [H]), "b2": vec(H),
            "att": rng.normal(0.0, 1.0 / np.sqrt(H), H).astype(np.float32),
            "w3": dense(H, [dn, H]), "b3": vec(H), "w4": dense(H, [H]), "b4": vec(H)}


STATUS_DIM_DEFAULT = 100


def status_spec(w: Workload):
    """Width and element type of the node statuses r_u that the RNN update
    maintains: a workload with node-feature rows updates those rows in place
    (so later queries gather the updated statuses); one without keeps an fp32
    status table of width 100 (the paper tunes status widths from 50 to 100)."""
    if w.node_dim:
        return w.node_dim, w.node_dtype
    return STATUS_DIM_DEFAULT, "f32"


def gru_weights(w: Workload, seed: int | None = None):
    """Random weights of the node-status GRU for workload ``w`` (see
    ``gru_weights_for``), seeded by the workload."""
    d, _ = status_spec(w)
    return gru_weights_for(d, w.d_time, w.edge_dim, 6000 + w.key if seed is None else seed)


def gru_weights_for(d: int, d_time: int, edge_dim: int, seed: int):
    """Random weights of a node-status GRU of width d: bf16 (uint16 bits)
    w_ih [3d][pad32(d) + pad32(d_time) + pad32(edge_dim)] for (r_other |
    T-enc(t) | e) and w_hh [3d][pad32(d)], gate rows r | z | n, zero pad
    columns; fp32 biases b_ih, b_hh [3d].  Entries ~ U(-1/sqrt(d),
    1/sqrt(d)), the usual GRU initialisation."""
    rng = np.random.default_rng(seed)
    k = 1.0 / np.sqrt(d)

    def dense(segs):
        out = np.zeros((3 * d, sum(_pad32(s) for s in segs)), np.float32)
        col = 0
        for sgl in segs:
            out[:, col:col + sgl] = rng.uniform(-k, k, (3 * d, sgl))
            col += _pad32(sgl)
        return _to_bf16_bits(out)
    return {"w_ih": dense([d, d_time, edge_dim]), "w_hh": dense([d]),
            "b_ih": rng.uniform(-k, k, 3 * d).astype(np.float32),
            "b_hh": rng.uniform(-k, k, 3 * d).astype(np.float32)}
