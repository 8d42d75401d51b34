"""AddressSanitizer and UndefinedBehaviorSanitizer over the host code, on
the CPU: the oracle (oracle/nlb_oracle.c) and the host side of libnlb.so
(argument validation, the no-GPU NLB_EDEVICE route, the host logic of every
entry point; the device code is built as usual).

Both are built with ROCm's clang so that one sanitizer runtime serves the
process, which preloads it; the rest of the CPU suite then runs against the
two sanitizer builds (NLB_ORACLE_LIB, NLB_LIBRARY).  A planted heap overflow
and a planted signed overflow, built with the same flags, show that the
runtime reports such mistakes.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
CLANG = os.path.join(ROCM, "llvm", "bin", "clang")
HIPCC = os.path.join(ROCM, "bin", "hipcc")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer", "-g"]


def _runtime():
    out = subprocess.run([CLANG, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True,
                         text=True).stdout.strip()
    if not os.path.isabs(out):
        import glob
        hits = glob.glob(os.path.join(ROCM, "llvm", "lib", "clang", "*", "lib", "linux",
                                      "libclang_rt.asan-x86_64.so"))
        out = hits[0] if hits else ""
    return out


@pytest.fixture(scope="module")
def san_env(tmp_path_factory):
    if not (os.path.exists(CLANG) and os.path.exists(HIPCC)):
        pytest.skip("ROCm clang / hipcc not found")
    rt = _runtime()
    if not os.path.exists(rt):
        pytest.skip("no sanitizer runtime")
    d = tmp_path_factory.mktemp("san")
    orc = str(d / "libnlb_oracle_san.so")
    subprocess.run([CLANG, "-O1", "-std=c11", "-ffp-contract=off", *SAN, "-shared", "-fPIC", "-o", orc,
                    os.path.join(ROOT, "oracle", "nlb_oracle.c"), "-lm"], check=True)
    lib = str(d / "libnlb_san.so")
    from paper_2402_01964_amd import build as nlb_build
    host_san = []
    for f in SAN:
        host_san += ["-Xarch_host", f]
    flags = [f for f in nlb_build.HIPCC_FLAGS if f != "-O3"]
    subprocess.run([HIPCC, "-O1", *flags, *host_san, "-I", os.path.join(ROOT, "include"), "-o", lib,
                    *nlb_build.SRCS], check=True, capture_output=True)
    env = dict(os.environ, LD_PRELOAD=rt, ASAN_OPTIONS="detect_leaks=0:verify_asan_link_order=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", NLB_ORACLE_LIB=orc, NLB_LIBRARY=lib)
    return d, env


@pytest.mark.parametrize("kind,source,report", [
    ("heap", "#include <stdlib.h>\nint main(int c, char **v) { int *a = malloc(4 * sizeof(int));"
             " int s = a[3 + c]; free(a); return s; }\n", "heap-buffer-overflow"),
    ("signed", "#include <limits.h>\nint main(int c, char **v) { int x = INT_MAX - 1; x += c + 1;"
               " return x == 0; }\n", "signed integer overflow"),
])
def test_runtime_reports_planted_mistakes(san_env, kind, source, report):
    d, env = san_env
    src, exe = d / f"planted_{kind}.c", d / f"planted_{kind}"
    src.write_text(source)
    subprocess.run([CLANG, "-O0", *SAN, "-o", str(exe), str(src)], check=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True,
                       env={k: v for k, v in env.items() if k != "LD_PRELOAD"})
    assert r.returncode != 0 and report in r.stderr, r.stderr[-2000:]


def test_cpu_suite_under_sanitizers(san_env):
    _, env = san_env
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests"), "-q", "-m", "not gpu",
                        "-p", "no:cacheprovider", "--deselect", "tests/test_sanitizers.py",
                        "--ignore", os.path.join(ROOT, "tests", "test_sanitizers.py")],
                       capture_output=True, text=True, env=env, cwd=ROOT, timeout=1200)
    tail = (r.stdout + r.stderr)[-3000:]
    assert r.returncode == 0, tail
    assert "passed" in r.stdout and "ERROR: AddressSanitizer" not in r.stderr, tail
