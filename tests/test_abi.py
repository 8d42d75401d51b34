"""The C ABI boundary, checked without a GPU: every symbol declared in
include/nlb.h is exported, host-side validation runs before any device work,
and the product path has no route to the oracle or a CPU fallback."""
import ctypes
import os
import re

import pytest

import paper_2402_01964_amd as nlb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    text = open(os.path.join(ROOT, "include", "nlb.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(nlb_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_binding_symbols():
    assert _declared() == sorted(nlb.ABI_SYMBOLS)


def test_library_exports_every_declared_symbol():
    lib = nlb.load_library()
    for name in _declared():
        assert hasattr(lib, name), name


def _cfg(**kw):
    c = nlb._Config()
    c.num_nodes, c.s, c.alpha, c.device = 100, 10, 0.5, -1
    for k, v in kw.items():
        setattr(c, k, v)
    return c


@pytest.mark.parametrize("bad", [
    dict(num_nodes=0), dict(num_nodes=2**31), dict(s=0), dict(s=1025), dict(alpha=0.0),
    dict(alpha=1.0000001), dict(alpha=-1.0), dict(key_mode=2), dict(q1=2**31), dict(q2=2**40),
    dict(d_time=5), dict(d_time=-1), dict(edge_feat=64), dict(edge_row_bytes=8),
    dict(node_feat=64, node_row_bytes=6), dict(edge_feat=64, edge_row_bytes=8, edge_rows=0),
    dict(node_feat=66, node_row_bytes=8),
])
def test_create_rejects_bad_config_before_touching_a_device(bad):
    lib = nlb.load_library()
    h = ctypes.c_void_p(12345)
    assert lib.nlb_create(ctypes.byref(_cfg(**bad)), ctypes.byref(h)) == nlb.NLB_EINVAL
    assert h.value == 12345   # *out untouched on failure


def test_null_arguments():
    lib = nlb.load_library()
    h = ctypes.c_void_p()
    assert lib.nlb_create(None, ctypes.byref(h)) == nlb.NLB_EINVAL
    assert lib.nlb_create(ctypes.byref(_cfg()), None) == nlb.NLB_EINVAL
    assert lib.nlb_destroy(None) == nlb.NLB_OK
    assert lib.nlb_insert_batch(None, None, None, None, 0, None) == nlb.NLB_EINVAL
    assert lib.nlb_sample(None, None, None, 0, None, None) == nlb.NLB_EINVAL
    assert lib.nlb_export(None, None, None, None, None) == nlb.NLB_EINVAL
    assert lib.nlb_status(None, None) == nlb.NLB_EINVAL
    assert lib.nlb_get_info(None, None) == nlb.NLB_EINVAL


def test_strerror():
    assert nlb.strerror(nlb.NLB_OK) == "success"
    for c in range(1, 7):
        assert nlb.strerror(c) and nlb.strerror(c) != "unknown error"
    assert nlb.strerror(77) == "unknown error"


def test_no_gpu_gives_edevice():
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    lib = nlb.load_library()
    h = ctypes.c_void_p()
    assert lib.nlb_create(ctypes.byref(_cfg()), ctypes.byref(h)) == nlb.NLB_EDEVICE
    assert not h.value


def test_missing_library_fails_loudly(tmp_path):
    saved = nlb._lib
    nlb._lib = None
    try:
        with pytest.raises(ImportError):
            nlb.load_library(str(tmp_path / "nope.so"))
    finally:
        nlb._lib = saved


def test_product_path_never_reaches_the_oracle():
    pkg = os.path.join(ROOT, "paper_2402_01964_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                text = open(os.path.join(dirpath, f)).read()
                assert not re.search(r"\boracle\b", text), f
                assert "nlb_oracle" not in text and "orc_" not in text, f


def test_one_hip_runtime_per_process():
    """The library and the input generator bind to torch's HIP runtime
    whatever the import order, so torch's streams and allocations belong to
    the same runtime as the library's kernels."""
    import subprocess
    import sys
    code = (
        "import sys; sys.path.insert(0, %r)\n"
        "import synth; synth._load()\n"
        "import paper_2402_01964_amd as nlb; nlb.load_library()\n"
        "print(len(set(l.split()[-1] for l in open('/proc/self/maps') if 'libamdhip64' in l)))\n"
    ) % ROOT
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300)
    assert out.returncode == 0, out.stderr
    assert out.stdout.strip() == "1"
