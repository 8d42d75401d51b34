"""Shared helpers of the GPU parity tests: run the GPU library and the CPU
oracle on the same seeded workload and compare."""
import numpy as np

import oracle
import synth

TENC_TOL = 1e-5   # max abs error of the fp32 time encoding


def torch_dev():
    import torch
    return torch.device("cuda", 0)


def to_dev(a, dtype=None):
    import torch
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint32:
        a = a.view(np.int32)
    t = torch.from_numpy(a)
    if dtype is not None:
        t = t.view(dtype)
    return t.to(torch_dev())


def feat_to_dev(arr, dtype_name):
    import torch
    if dtype_name == "bf16":
        return to_dev(arr.view(np.int16), torch.bfloat16)
    return to_dev(arr)


def u32(t):
    return t.cpu().numpy().view(np.uint32)


def host_np(t):
    import torch
    if t.dtype == torch.bfloat16:
        return t.cpu().view(torch.int16).numpy().view(np.uint16)
    return t.cpu().numpy()


def make_gpu_table(w, efeat_dev=None, nfeat_dev=None, time=True, **kw):
    import paper_2402_01964_amd as nlb
    tw = tb = None
    if time and w.d_time:
        fw, fb = synth.time_params(w)
        tw, tb = to_dev(fw), to_dev(fb)
    return nlb.Table(w.num_nodes, w.s, w.alpha, w.table_seed, time_w=tw, time_b=tb,
                     edge_feat=efeat_dev, node_feat=nfeat_dev, **kw)


def make_oracle(w, **kw):
    return oracle.Oracle(w.num_nodes, w.s, w.alpha, w.table_seed, **kw)


def compare_tables(gpu_table, orc, nodes=None):
    nbr, ts, eid = gpu_table.export()
    g = (nbr.cpu().numpy(), u32(ts), u32(eid))
    o = orc.export() if nodes is None else orc.export_nodes(nodes)
    if nodes is not None:
        g = tuple(x[nodes] for x in g)
    for a, b, name in zip(g, o, ("nbr", "ts", "eid")):
        if not np.array_equal(a, b):
            bad = np.argwhere(a != b)
            raise AssertionError(f"table {name} differs at {len(bad)} cells, first {bad[:5].tolist()}: "
                                 f"gpu {a[tuple(bad[0])]} oracle {b[tuple(bad[0])]}")


def compare_sample(gout, oout, what=""):
    """Bit-exact indices and feature rows; time encoding within TENC_TOL."""
    for k, ov in oout.items():
        gv = gout[k]
        gv = host_np(gv)
        if k in ("eid", "ts"):
            gv = gv.view(np.uint32)
        if k == "tenc":
            err = np.abs(gv.astype(np.float64) - ov.astype(np.float64))
            assert err.max() <= TENC_TOL, f"{what} tenc max err {err.max()}"
            # invalid slots must be exact zeros
            inval = oout["nbr"] < 0 if "nbr" in oout else None
            if inval is not None:
                assert not gv[inval].any(), f"{what} tenc nonzero on invalid slots"
        else:
            if not np.array_equal(gv, ov):
                bad = np.argwhere(gv != ov)
                raise AssertionError(f"{what} {k} differs at {len(bad)} positions, first "
                                     f"{bad[:3].tolist()}")
