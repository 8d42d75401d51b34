"""nlb_rnn_update_noalloc (working memory in the library's static array)
against nlb_rnn_update (working memory of the table) through the C ABI.

Both run the same kernels on the same inputs, so the new statuses must be
identical; they are also held to the oracle's GRU (Sec. 4.4 status update)
within the tolerance of nlb_rnn_update.  Two calls in a row, the second
with a smaller batch, in both GRU forms; then a table too large for the
static array is refused before anything is enqueued.
"""
import dataclasses

import numpy as np
import pytest

import oracle
import synth
from tests.gpu_helpers import feat_to_dev, host_np, make_gpu_table, to_dev

pytestmark = pytest.mark.gpu

RNN_TOL = 1e-4
BF16_REL = 2.0 ** -7


def _log(*a):
    print("[no-alloc]", *a, flush=True)


def _bf16(bits):
    return (np.asarray(bits, np.uint32) << 16).view(np.float32).astype(np.float64)


def _close_to_oracle(got, want, what):
    if got.dtype == np.uint16:
        g, o = _bf16(got), _bf16(want)
        assert (np.abs(g - o) <= RNN_TOL + BF16_REL * np.abs(o)).all(), what
    else:
        assert np.abs(got.astype(np.float64) - want.astype(np.float64)).max() <= RNN_TOL, what


@pytest.mark.parametrize("k", [5, 1])   # bf16 128-wide statuses (weight-stationary GRU); fp32 100 (tiled)
def test_noalloc_matches_the_allocating_update(k):
    import paper_2402_01964_amd as nlb
    import torch
    base = synth.workload(k)
    w = dataclasses.replace(synth.scaled(base, 3 * base.batch, num_nodes=min(base.num_nodes, 100000)),
                            batch=base.batch)
    src, dst, t, _ = synth.host_links(w)
    d, dtype = synth.status_spec(w)
    ef = synth.host_features(w, "edge") if w.edge_dim else None
    g = make_gpu_table(w, feat_to_dev(ef, w.edge_dtype) if ef is not None else None, None)
    rng = np.random.default_rng(k)
    x = rng.standard_normal((w.num_nodes, d)).astype(np.float32)
    st0 = synth._to_bf16_bits(x) if dtype == "bf16" else x
    a = feat_to_dev(st0, dtype)
    b = a.clone()
    W = synth.gru_weights(w)
    Wd = {kk: (to_dev(v.view(np.int16)) if v.dtype == np.uint16 else to_dev(v)) for kk, v in W.items()}
    fw, fb = synth.time_params(w)
    host = st0.copy()
    forms = []
    for lo, hi in ((0, w.batch), (w.batch, w.batch + w.batch // 3)):   # second call smaller
        s_, d_, t_ = to_dev(src[lo:hi]), to_dev(dst[lo:hi]), to_dev(t[lo:hi])
        g.rnn_update(s_, d_, t_, lo, Wd, a)
        g.rnn_update(s_, d_, t_, lo, Wd, b, noalloc=True)
        forms.append(g.info()["rnn_form"])
        torch.cuda.synchronize()
        ga, gb = host_np(a), host_np(b)
        assert np.array_equal(ga, gb), f"workload {k} links {lo}..{hi}: the two entry points differ"
        host = oracle.gru_update(host, src[lo:hi], dst[lo:hi], t[lo:hi], lo, fw, fb, ef, W)
        _close_to_oracle(gb, host, f"workload {k} links {lo}..{hi}")
        host = gb.copy()   # next call starts from the GPU's statuses on both sides
        _log(f"workload {k}: {hi - lo} links, form {forms[-1]}, identical to nlb_rnn_update")
    assert g.status() == 0
    want_form = nlb.RNN_FORM_WEIGHT_STATIONARY if k == 5 else nlb.RNN_FORM_TILED
    assert forms == [want_form, want_form]


def test_noalloc_refuses_a_table_beyond_its_array():
    import paper_2402_01964_amd as nlb
    import torch
    N, d = 9_000_000, 32                       # 72 MB of winner words alone
    g = nlb.Table(N, 4, 0.5, 1)
    st = torch.zeros((N, d), dtype=torch.float32, device="cuda")
    W = synth.gru_weights_for(d, 0, 0, seed=1)
    Wd = {kk: (to_dev(v.view(np.int16)) if v.dtype == np.uint16 else to_dev(v)) for kk, v in W.items()}
    src = to_dev(np.arange(10, dtype=np.int32))
    with pytest.raises(nlb.NLBError) as e:
        g.rnn_update(src, src, to_dev(np.zeros(10, np.uint32)), 0, Wd, st, noalloc=True)
    assert e.value.code == nlb.NLB_ESCRATCH
    torch.cuda.synchronize()
    assert not st.any()                         # nothing was enqueued
    assert g.status() == 0
