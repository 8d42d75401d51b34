"""Host logic of bench.py (CPU only): the algorithmic byte and FLOP counts
behind its roofline figures, the gate that keeps stale counter summaries out
of its output, and the one-GPU contract."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import synth  # noqa: E402


# Bytes per query at full table occupancy (every slot valid), from the
# workloads' shapes: reads 8 + 12 s + row_n + s (row_e + row_n), writes
# s (12 + 4 d_time + row_e + row_n) + row_n.
FULL_OCCUPANCY_BYTES = {
    "tiny-bipartite": 12248,
    "small-bipartite": 36008,
    "medium-homogeneous": 93192,
    "dense-repeated": 11688,
    "large-sparse": 9880,
}


@pytest.mark.parametrize("k", range(1, 6))
def test_sample_bytes_at_full_occupancy(k):
    w = synth.workload(k)
    assert bench.sample_bytes(w, w.s, 1) == FULL_OCCUPANCY_BYTES[w.name]
    # every invalid slot removes exactly its two row reads
    assert (bench.sample_bytes(w, w.s, 1) - bench.sample_bytes(w, 0, 1)
            == w.s * (w.row_bytes("edge") + w.row_bytes("node")))


def test_insert_and_hop2_bytes():
    assert bench.insert_bytes(1) == 52          # 12 B input + 2 offers x (8 + 8 + 4) B
    w = synth.workload(5)                       # s = 10
    # one first-hop query: 10 entries (8 B each), all valid (12 B x 10 slots
    # read each), 100 second-hop slots written (12 B each)
    assert bench.hop2_bytes(w, 10, 1) == 80 + 1200 + 1200


def test_rnn_and_aggregate_counts():
    w = synth.workload(5)                       # node rows 128, no link rows, d_time 100
    assert bench.rnn_flops(w, 128, 1) == 2 * 3 * 128 * (128 + 100) + 2 * 3 * 128 * 128
    assert bench.rnn_bytes(w, 128, 2, 1, 1) == 12 + 3 * 256
    H = 64
    per_slot = 2 * (228 * H + H)
    per_query = 2 * (H * H + (128 + H) * H + H * H)
    assert bench.aggregate_flops(w, 7, 1) == 7 * per_slot + per_query


def test_counter_summary_is_used_only_for_the_current_sources(monkeypatch):
    w = synth.workload(5)
    t = bench.measured_traffic(w)
    assert t is not None and 1e9 < t < 1e10
    monkeypatch.setattr(bench, "kernel_source_hash", lambda call="nlb_sample": "0" * 64)
    assert bench.measured_traffic(w) is None
    assert bench.measured_traffic(synth.workload(1)) is None   # no summary for that workload


def test_aggregate_counter_summary_and_kernel_choice(monkeypatch):
    w = synth.workload(5)
    t = bench.measured_traffic(w, "nlb_aggregate")
    assert t is not None and 1e8 < t < 1e10
    monkeypatch.setattr(bench, "kernel_source_hash", lambda call="nlb_sample": "0" * 64)
    assert bench.measured_traffic(w, "nlb_aggregate") is None
    # 300 000 queries on 256 CUs: groups of 16 (packed); 600 queries: groups of 1
    assert bench.aggregate_kernel(w, 300000, 256) == "aggregate_packed"
    assert bench.aggregate_kernel(synth.workload(1), 600, 256) == "aggregate_rows"
    assert bench.aggregate_kernel(synth.workload(3), 12000, 256) == "aggregate_rows"   # s = 64
    assert bench.aggregate_kernel(w, 300000, 256, heads=2) == "aggregate_packed"
    assert bench.aggregate_kernel(w, 3000, 256, heads=2) == "aggregate_rows"
    assert bench.aggregate_kernel(w, 300000, 256, heads=4) == "aggregate_fused"


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr


def test_binding_roofline_is_the_slower_peak():
    # 86 us of bytes at 8 TB/s against 28 us of FLOPs at 2.5 PFLOP/s: HBM binds
    r = bench.binding_roofline(7.0e10, 6.9e8, 3.9e-4)
    assert r["bound"] == "hbm" and r["unit"] == "GB/s" and r["other"]["bound"] == "mfma"
    assert abs(r["frac"] - 6.9e8 / 3.9e-4 / 8e12) < 1e-12
    # 8.7 us of FLOPs against 7.8 us of bytes: the matrix cores bind
    r = bench.binding_roofline(2.17e10, 6.2e7, 4.8e-5)
    assert r["bound"] == "mfma" and r["unit"] == "TFLOP/s"
    assert abs(r["floor_seconds"] - 2.17e10 / 2.5e15) < 1e-15
