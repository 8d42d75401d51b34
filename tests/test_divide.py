"""Exactness of the library's index division (csrc/nlb_divide.h) on the CPU.

The helper is plain integer arithmetic shared by host and device code; the
kernels split flat output indices into (row, column) and slot rows into
(query, slot) with it.  The check compiles the header with g++ and runs
tests/divide_check.cpp: every row boundary for every divisor up to 65536
and tiles of up to 1024 rows, every numerator below 2^26 for a set of
divisors, quotient boundaries over the whole 32-bit range (divisor 1
included), every pair of the 12-bit slot-row form, and random pairs.
"""
import os
import subprocess

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_division_helper_is_exact(tmp_path):
    exe = tmp_path / "divide_check"
    subprocess.run(["g++", "-O2", "-std=c++17", "-Wall", "-Wextra", "-Werror",
                    "-I", os.path.join(ROOT, "paper_2402_01964_amd", "csrc"),
                    "-o", str(exe), os.path.join(ROOT, "tests", "divide_check.cpp")], check=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300)
    assert out.returncode == 0, out.stdout + out.stderr
    assert out.stdout.startswith("ok "), out.stdout
    # the boundary set is sharp enough to catch the former 40-bit helper
    wrong = int(out.stdout.split("wrong at ")[1].split()[0])
    assert wrong > 0, out.stdout
