"""NLB forward recent sampling on MI355X (gfx950).

Python binding of ``libnlb.so`` (the C ABI in ``include/nlb.h``).  It only
marshals arguments: every step of insertion and sampling runs in the HIP
kernels of the library.  torch is used for device memory and streams.

Method: Luo & Li, "Scalable and Efficient Temporal Graph Representation
Learning via Forward Recent Sampling", arXiv 2402.01964 (Sec. 4.2 table
maintenance, Sec. 4.4 retrieval, attention aggregation and status update,
App. C time encoding).
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libnlb.so")

NLB_OK, NLB_EINVAL, NLB_ENOMEM, NLB_EDEVICE, NLB_EORDER, NLB_ERANGE, NLB_ESCRATCH = range(7)
NOALLOC_SCRATCH = 64 << 20
KEY_EDGE, KEY_NODE = 0, 1
MAX_SLOTS = 1024

# Symbols declared in include/nlb.h.
ABI_SYMBOLS = ("nlb_create", "nlb_insert_batch", "nlb_sample", "nlb_sample_hop2", "nlb_time_encode", "nlb_aggregate",
               "nlb_rnn_update", "nlb_rnn_update_noalloc", "nlb_destroy", "nlb_get_info", "nlb_export", "nlb_status",
               "nlb_strerror")
AGG_HIDDEN = 64
RNN_MAX_DIM = 1024
DTYPE_F32, DTYPE_BF16 = 0, 1
RNN_FORM_NONE, RNN_FORM_TILED, RNN_FORM_WEIGHT_STATIONARY = 0, 1, 2
EID_LAST_BATCH = 2**64 - 1   # first_eid of rnn_update: the links inserted last (device count)


class NLBError(RuntimeError):
    def __init__(self, code: int, what: str):
        self.code = code
        super().__init__(f"{what}: {strerror(code)} (code {code})")


class _Config(ctypes.Structure):
    _fields_ = [("num_nodes", ctypes.c_int64), ("s", ctypes.c_int32),
                ("key_mode", ctypes.c_int32), ("alpha", ctypes.c_double),
                ("seed", ctypes.c_uint64), ("q1", ctypes.c_uint64), ("q2", ctypes.c_uint64),
                ("d_time", ctypes.c_int32), ("time_w", ctypes.c_void_p),
                ("time_b", ctypes.c_void_p), ("edge_feat", ctypes.c_void_p),
                ("edge_rows", ctypes.c_int64), ("edge_row_bytes", ctypes.c_int32),
                ("node_feat", ctypes.c_void_p), ("node_row_bytes", ctypes.c_int32),
                ("device", ctypes.c_int32)]


class _SampleOut(ctypes.Structure):
    _fields_ = [(k, ctypes.c_void_p) for k in ("nbr", "eid", "ts", "tenc", "efeat", "nfeat", "self")]


class _AggWeights(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int32), ("node_dtype", ctypes.c_int32),
                ("edge_dtype", ctypes.c_int32), ("heads", ctypes.c_int32)] + \
               [(k, ctypes.c_void_p) for k in ("w1", "b1", "w2", "b2", "att", "w3", "b3", "w4", "b4")]


class _GruWeights(ctypes.Structure):
    _fields_ = [("status_dim", ctypes.c_int32), ("status_dtype", ctypes.c_int32),
                ("edge_dtype", ctypes.c_int32)] + \
               [(k, ctypes.c_void_p) for k in ("w_ih", "w_hh", "b_ih", "b_hh")]


class _Info(ctypes.Structure):
    _fields_ = [("num_nodes", ctypes.c_int64), ("s", ctypes.c_int32), ("key_mode", ctypes.c_int32),
                ("threshold", ctypes.c_uint64), ("q1", ctypes.c_uint64), ("q2", ctypes.c_uint64),
                ("interactions", ctypes.c_uint64), ("table_bytes", ctypes.c_int64),
                ("block_bytes", ctypes.c_int32), ("device", ctypes.c_int32), ("rnn_form", ctypes.c_int32)]


_lib = None


def load_library(path: str | None = None):
    """Load libnlb.so (or the build named by NLB_LIBRARY, e.g. a sanitizer
    build of the same sources).  Fails loudly when it has not been built:
    there is no other implementation to fall back to."""
    global _lib
    if _lib is not None:
        return _lib
    if path is None:
        path = os.environ.get("NLB_LIBRARY", LIB_PATH)
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with "
                          f"`python -m paper_2402_01964_amd.build` (hipcc, gfx950)")
    # torch ships its own HIP runtime with the same soname as the system one
    # the library links against.  Loading torch first makes the library bind
    # to that copy, so one runtime owns the devices, streams and allocations
    # that torch hands to the library.
    import torch  # noqa: F401
    lib = ctypes.CDLL(path)
    P, I, U32, U64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_uint32, ctypes.c_uint64
    lib.nlb_create.argtypes = [ctypes.POINTER(_Config), ctypes.POINTER(P)]
    lib.nlb_create.restype = I
    lib.nlb_insert_batch.argtypes = [P, P, P, P, U32, P]
    lib.nlb_insert_batch.restype = I
    lib.nlb_sample.argtypes = [P, P, P, U32, ctypes.POINTER(_SampleOut), P]
    lib.nlb_sample.restype = I
    lib.nlb_sample_hop2.argtypes = [P, P, P, U32, ctypes.POINTER(_SampleOut), P]
    lib.nlb_sample_hop2.restype = I
    lib.nlb_time_encode.argtypes = [P, P, P, U32, P, P]
    lib.nlb_time_encode.restype = I
    lib.nlb_aggregate.argtypes = [P, P, P, U32, ctypes.POINTER(_AggWeights), P, P]
    lib.nlb_aggregate.restype = I
    lib.nlb_rnn_update.argtypes = [P, P, P, P, U32, U64, ctypes.POINTER(_GruWeights), P, P]
    lib.nlb_rnn_update.restype = I
    lib.nlb_rnn_update_noalloc.argtypes = [P, P, P, P, U32, U64, ctypes.POINTER(_GruWeights), P, P]
    lib.nlb_rnn_update_noalloc.restype = I
    lib.nlb_destroy.argtypes = [P]
    lib.nlb_destroy.restype = I
    lib.nlb_get_info.argtypes = [P, ctypes.POINTER(_Info)]
    lib.nlb_get_info.restype = I
    lib.nlb_export.argtypes = [P, P, P, P, P]
    lib.nlb_export.restype = I
    lib.nlb_status.argtypes = [P, P]
    lib.nlb_status.restype = I
    lib.nlb_strerror.argtypes = [I]
    lib.nlb_strerror.restype = ctypes.c_char_p
    _lib = lib
    return lib


def strerror(code: int) -> str:
    return load_library().nlb_strerror(int(code)).decode()


def _check(rc: int, what: str):
    if rc != NLB_OK:
        raise NLBError(rc, what)


def _dev_ptr(t, dtype_bytes=None, name="tensor"):
    import torch
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype_bytes is not None and t.element_size() != dtype_bytes:
        raise TypeError(f"{name} must have {dtype_bytes}-byte elements")
    return t.data_ptr()


def _stream_ptr(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


class Table:
    """Per-node NLB tables on one GPU (Sec. 4.2).

    ``time_w``/``time_b``: fp32 [d_time] CUDA tensors; ``edge_feat``: 2-D
    CUDA tensor indexed by arrival index; ``node_feat``: 2-D CUDA tensor with
    one row per node.  The library borrows them; this object keeps them alive.
    Timestamps are passed as int32 or uint32 tensors holding uint32 values.
    """

    def __init__(self, num_nodes: int, s: int, alpha: float, seed: int, *, key_mode: int = KEY_EDGE,
                 q1: int = 0, q2: int = 0, time_w=None, time_b=None, edge_feat=None,
                 node_feat=None, device: int = -1):
        import torch
        lib = load_library()
        self._lib = lib
        self._h = ctypes.c_void_p()
        self._keep = (time_w, time_b, edge_feat, node_feat)
        self.edge_feat, self.node_feat = edge_feat, node_feat
        self.d_time = 0 if time_w is None else int(time_w.numel())
        if time_w is not None and (time_w.dtype != torch.float32 or time_b is None
                                   or time_b.dtype != torch.float32
                                   or time_b.numel() != self.d_time):
            raise TypeError("time_w and time_b must be fp32 tensors of equal length")
        cfg = _Config()
        cfg.num_nodes, cfg.s, cfg.key_mode = int(num_nodes), int(s), int(key_mode)
        cfg.alpha, cfg.seed = float(alpha), int(seed) & (2**64 - 1)
        cfg.q1, cfg.q2 = int(q1), int(q2)
        cfg.d_time = self.d_time
        cfg.time_w = _dev_ptr(time_w, 4, "time_w")
        cfg.time_b = _dev_ptr(time_b, 4, "time_b")
        if edge_feat is not None:
            cfg.edge_feat = _dev_ptr(edge_feat, None, "edge_feat")
            cfg.edge_rows = int(edge_feat.shape[0])
            cfg.edge_row_bytes = int(edge_feat[0].numel() * edge_feat.element_size())
        if node_feat is not None:
            cfg.node_feat = _dev_ptr(node_feat, None, "node_feat")
            if node_feat.shape[0] < num_nodes:
                raise ValueError("node_feat needs one row per node")
            cfg.node_row_bytes = int(node_feat[0].numel() * node_feat.element_size())
        cfg.device = int(device)
        _check(lib.nlb_create(ctypes.byref(cfg), ctypes.byref(self._h)), "nlb_create")
        self.num_nodes, self.s = int(num_nodes), int(s)

    # -- lifetime
    def close(self):
        if self._h:
            rc = self._lib.nlb_destroy(self._h)
            self._h = ctypes.c_void_p()
            _check(rc, "nlb_destroy")

    def __del__(self):
        try:
            if self._h:
                self._lib.nlb_destroy(self._h)
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    # -- calls
    def insert(self, src, dst, t, stream=None):
        n = int(src.numel())
        if dst.numel() != n or t.numel() != n:
            raise ValueError("src, dst and t must have the same length")
        _check(self._lib.nlb_insert_batch(self._h, _dev_ptr(src, 4, "src"), _dev_ptr(dst, 4, "dst"),
                                          _dev_ptr(t, 4, "t"), n, _stream_ptr(stream)),
               "nlb_insert_batch")

    def sample_into(self, node, tq, out: dict, stream=None):
        """Answer queries into caller-provided output tensors (keys of
        ``nlb_sample_out``; missing keys are skipped)."""
        nq = int(node.numel())
        if tq.numel() != nq:
            raise ValueError("node and tq must have the same length")
        so = _SampleOut()
        for k in ("nbr", "eid", "ts", "tenc", "efeat", "nfeat", "self"):
            setattr(so, k, _dev_ptr(out.get(k), None, k))
        _check(self._lib.nlb_sample(self._h, _dev_ptr(node, 4, "node"), _dev_ptr(tq, 4, "tq"), nq,
                                    ctypes.byref(so), _stream_ptr(stream)), "nlb_sample")
        return out

    def sample_hop2_into(self, hop1_nbr, tq, out: dict, stream=None):
        """Second-hop answers (Sec. 4.4) for the [nq, s] first-hop neighbours
        ``hop1_nbr`` of queries with times ``tq``, into caller tensors shaped
        for nq*s queries."""
        nq = int(tq.numel())
        if hop1_nbr.numel() != nq * self.s:
            raise ValueError("hop1_nbr must hold s entries per query")
        so = _SampleOut()
        for k in ("nbr", "eid", "ts", "tenc", "efeat", "nfeat", "self"):
            setattr(so, k, _dev_ptr(out.get(k), None, k))
        _check(self._lib.nlb_sample_hop2(self._h, _dev_ptr(hop1_nbr, 4, "hop1_nbr"),
                                         _dev_ptr(tq, 4, "tq"), nq, ctypes.byref(so),
                                         _stream_ptr(stream)), "nlb_sample_hop2")
        return out

    def time_encode_into(self, ts, tq, tenc, stream=None):
        """App. C time encoding of a first-hop answer from its timestamp
        output ``ts`` [nq, s] and query times ``tq`` [nq] into ``tenc``
        [nq, s, d_time]: the values ``sample_into`` writes to its own tenc
        output.  The caller orders it after the sample that wrote ``ts``."""
        nq = int(tq.numel())
        if ts.numel() != nq * self.s:
            raise ValueError("ts must hold s entries per query")
        if tenc.numel() != nq * self.s * self.d_time:
            raise ValueError("tenc must hold s * d_time values per query")
        _check(self._lib.nlb_time_encode(self._h, _dev_ptr(ts, 4, "ts"), _dev_ptr(tq, 4, "tq"), nq,
                                         _dev_ptr(tenc, 4, "tenc"), _stream_ptr(stream)),
               "nlb_time_encode")
        return tenc

    def sample_hop2(self, hop1_nbr, tq, want=("nbr", "eid", "ts", "tenc", "efeat", "nfeat", "self"),
                    stream=None):
        """Second-hop answers as new tensors shaped [nq, s, s, ...] (self:
        [nq, s, ...])."""
        nq = int(tq.numel())
        out = self.alloc_outputs(nq * self.s, want)
        self.sample_hop2_into(hop1_nbr, tq, out, stream)
        return {k: v.view(nq, self.s, *v.shape[1:]) for k, v in out.items()}

    def aggregate(self, node, tq, weights: dict, out=None, stream=None, heads: int = 1):
        """Eq. (4) attention aggregation for queries (node[i], tq[i]).
        ``weights``: device tensors w1..w4 (bf16, or 16-bit ints holding bf16
        bits, padded layouts of include/nlb.h) and b1..b4, att (fp32);
        ``heads`` attention heads, each over its own slice of the hidden
        width.  Returns (or fills) z, fp32 [nq, AGG_HIDDEN]."""
        import torch
        nq = int(node.numel())
        if tq.numel() != nq:
            raise ValueError("node and tq must have the same length")
        aw = _AggWeights()
        aw.hidden = AGG_HIDDEN
        aw.heads = int(heads)

        def dt(feat):
            return DTYPE_F32 if feat is None or feat.dtype == torch.float32 else DTYPE_BF16
        aw.node_dtype, aw.edge_dtype = dt(self.node_feat), dt(self.edge_feat)
        for k in ("w1", "w2", "w3", "w4"):
            setattr(aw, k, _dev_ptr(weights[k], 2, k))
        for k in ("b1", "b2", "b3", "b4", "att"):
            setattr(aw, k, _dev_ptr(weights[k], 4, k))
        if out is None:
            out = torch.empty((nq, AGG_HIDDEN), dtype=torch.float32, device=node.device)
        _check(self._lib.nlb_aggregate(self._h, _dev_ptr(node, 4, "node"), _dev_ptr(tq, 4, "tq"), nq,
                                       ctypes.byref(aw), _dev_ptr(out, 4, "z"), _stream_ptr(stream)),
               "nlb_aggregate")
        return out

    def rnn_update(self, src, dst, t, first_eid: int, weights: dict, status, stream=None,
                   noalloc: bool = False):
        """Node-status GRU update of Sec. 4.4 after the links (src[i], dst[i],
        t[i]) whose link rows are first_eid + i, in place on ``status`` (a
        CUDA tensor [N, d], fp32 or bf16 -- e.g. this table's node_feat).
        ``weights``: w_ih, w_hh (bf16, or 16-bit ints holding bf16 bits, padded
        layouts of include/nlb.h) and b_ih, b_hh (fp32).  ``noalloc`` calls
        nlb_rnn_update_noalloc (working memory in the library's static
        array; NLBError with NLB_ESCRATCH when it does not fit)."""
        import torch
        n = int(src.numel())
        if dst.numel() != n or t.numel() != n:
            raise ValueError("src, dst and t must have the same length")
        if status.dim() != 2:
            raise ValueError("status must be [N, d]")
        gw = _GruWeights()
        gw.status_dim = int(status.shape[1])
        gw.status_dtype = DTYPE_F32 if status.dtype == torch.float32 else DTYPE_BF16
        if status.dtype not in (torch.float32, torch.bfloat16, torch.int16):
            raise TypeError("status must be float32 or bfloat16 (int16 bits)")
        gw.edge_dtype = DTYPE_F32 if self.edge_feat is None or self.edge_feat.dtype == torch.float32 \
            else DTYPE_BF16
        for k in ("w_ih", "w_hh"):
            setattr(gw, k, _dev_ptr(weights[k], 2, k))
        for k in ("b_ih", "b_hh"):
            setattr(gw, k, _dev_ptr(weights[k], 4, k))
        fn, name = ((self._lib.nlb_rnn_update_noalloc, "nlb_rnn_update_noalloc") if noalloc
                    else (self._lib.nlb_rnn_update, "nlb_rnn_update"))
        _check(fn(self._h, _dev_ptr(src, 4, "src"), _dev_ptr(dst, 4, "dst"), _dev_ptr(t, 4, "t"), n,
                  int(first_eid), ctypes.byref(gw), _dev_ptr(status, None, "status"), _stream_ptr(stream)),
               name)
        return status

    def alloc_outputs(self, nq: int, want=("nbr", "eid", "ts", "tenc", "efeat", "nfeat", "self")):
        import torch
        dev = torch.device("cuda", self.info()["device"])
        s = self.s
        out = {}
        if "nbr" in want:
            out["nbr"] = torch.empty((nq, s), dtype=torch.int32, device=dev)
        if "eid" in want:
            out["eid"] = torch.empty((nq, s), dtype=torch.int32, device=dev)
        if "ts" in want:
            out["ts"] = torch.empty((nq, s), dtype=torch.int32, device=dev)
        if "tenc" in want and self.d_time:
            out["tenc"] = torch.empty((nq, s, self.d_time), dtype=torch.float32, device=dev)
        if "efeat" in want and self.edge_feat is not None:
            out["efeat"] = torch.empty((nq, s, *self.edge_feat.shape[1:]),
                                       dtype=self.edge_feat.dtype, device=dev)
        if self.node_feat is not None:
            if "nfeat" in want:
                out["nfeat"] = torch.empty((nq, s, *self.node_feat.shape[1:]),
                                           dtype=self.node_feat.dtype, device=dev)
            if "self" in want:
                out["self"] = torch.empty((nq, *self.node_feat.shape[1:]),
                                          dtype=self.node_feat.dtype, device=dev)
        return out

    def sample(self, node, tq, want=("nbr", "eid", "ts", "tenc", "efeat", "nfeat", "self"),
               stream=None):
        """Answer queries (node[i], tq[i]); returns a dict of new tensors.
        eid and ts are int32 tensors holding uint32 bit patterns."""
        out = self.alloc_outputs(int(node.numel()), want)
        return self.sample_into(node, tq, out, stream)

    def export(self, stream=None):
        """Canonical table (nbr, ts, eid) as int32 tensors [N, s] (ts/eid hold uint32 bits)."""
        import torch
        dev = torch.device("cuda", self.info()["device"])
        shape = (self.num_nodes, self.s)
        nbr = torch.empty(shape, dtype=torch.int32, device=dev)
        ts = torch.empty(shape, dtype=torch.int32, device=dev)
        eid = torch.empty(shape, dtype=torch.int32, device=dev)
        _check(self._lib.nlb_export(self._h, nbr.data_ptr(), ts.data_ptr(), eid.data_ptr(),
                                    _stream_ptr(stream)), "nlb_export")
        return nbr, ts, eid

    def status(self, stream=None) -> int:
        """Synchronise and return (and clear) device-detected errors."""
        return int(self._lib.nlb_status(self._h, _stream_ptr(stream)))

    def info(self) -> dict:
        inf = _Info()
        _check(self._lib.nlb_get_info(self._h, ctypes.byref(inf)), "nlb_get_info")
        return {k: getattr(inf, k) for k, _ in _Info._fields_}
