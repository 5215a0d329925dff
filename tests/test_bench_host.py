"""Host logic of bench.py, no device: the byte model of the roofline, the checks that decide
whether the committed counter summary may be reported, and the one-GPU rule."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_byte_model_at_full_sizes():
    # c4: n = 2^21, nnz = 62,914,560, F = 128; c5 layer 2: n = 2^22, nnz = 67,108,864, F = 64
    n4, nnz4, n5, nnz5 = 1 << 21, 62914560, 1 << 22, 67108864
    assert bench.spmm_bytes(n4, nnz4, 128) == 2667577348
    assert bench.spmm_bytes(n5, nnz5, 64) == 2717908996
    # a bfloat16 output halves the output term only
    assert bench.spmm_bytes(n5, nnz5, 128) - bench.spmm_bytes(n5, nnz5, 128, 2) == 2 * n5 * 128
    # the fused junction reads X (F_in) and writes T (F_out) once
    assert bench.fused_bytes(n5, nnz5, 128, 64) == 3791650820
    assert bench.fused_bytes(n5, nnz5, 128, 128) == bench.spmm_bytes(n5, nnz5, 128)


def _summary(tmp_path, workload="c5", kernel="spmm_xw_kernel<32>", digest=None):
    p = tmp_path / "summary.md"
    p.write_text("# counters\n\nworkload: %s\nkernel: %s\ntraffic_bytes_per_launch: 123456\n"
                 "kernel_source_sha256: %s\n" % (workload, kernel, digest or bench.kernel_source_hash()))
    return str(p)


def test_counter_summary_is_reported_only_when_it_matches(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "COUNTER_SUMMARY", _summary(tmp_path))
    assert bench.counter_traffic("c5", "spmm_xw_kernel<32>")[0] == 123456
    assert bench.counter_traffic("c4", "spmm_xw_kernel<32>")[0] is None
    assert bench.counter_traffic("c5", "spmm_dual_kernel<32, 4, true>")[0] is None
    monkeypatch.setattr(bench, "COUNTER_SUMMARY", _summary(tmp_path, digest="0" * 64))
    value, why = bench.counter_traffic("c5", "spmm_xw_kernel<32>")
    assert value is None and "changed" in why
    monkeypatch.setattr(bench, "COUNTER_SUMMARY", str(tmp_path / "missing.md"))
    assert bench.counter_traffic("c5", "spmm_xw_kernel<32>")[0] is None


def test_committed_counter_summary_names_the_default_kernel():
    text = open(bench.COUNTER_SUMMARY).read()
    assert "workload: c5" in text and "kernel: spmm_xw_kernel<32>" in text


@pytest.mark.parametrize("gpus", ["2", "8"])
def test_more_than_one_gpu_is_refused(gpus):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", gpus],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    line = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in line["error"] and line["n_gpus"] == int(gpus)
