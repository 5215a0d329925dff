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


RUN = {"graph_sha256": "8f58468c61854d5c", "F_in": 128, "F_out": 64, "walks_per_node": 16,
       "walk_len": 5}


def _summary(tmp_path, workload="c5", kernel="spmm_xw_kernel<32>", digest=None, run=RUN):
    p = tmp_path / "summary.md"
    p.write_text("# counters\n\nworkload: %s\nkernel: %s\ntraffic_bytes_per_launch: 123456\n"
                 "kernel_source_sha256: %s\n" % (workload, kernel, digest or bench.kernel_source_hash())
                 + "".join(f"{k}: {v}\n" for k, v in run.items()))
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


def test_counter_summary_must_match_the_run(tmp_path, monkeypatch):
    """Counters taken on another graph, feature widths or walk parameters are not reported,
    and the plan's sources (partition, walks) are part of the source hash."""
    monkeypatch.setattr(bench, "COUNTER_SUMMARY", _summary(tmp_path))
    assert bench.counter_traffic("c5", "spmm_xw_kernel<32>", RUN)[0] == 123456
    for key, other in (("graph_sha256", "0123456789abcdef"), ("F_in", 256), ("F_out", 128),
                       ("walks_per_node", 50), ("walk_len", 30)):
        value, why = bench.counter_traffic("c5", "spmm_xw_kernel<32>", dict(RUN, **{key: other}))
        assert value is None and key in why
    # a summary without the run's lines is not reported either
    monkeypatch.setattr(bench, "COUNTER_SUMMARY", _summary(tmp_path, run={}))
    assert bench.counter_traffic("c5", "spmm_xw_kernel<32>", RUN)[0] is None
    names = [os.path.basename(p) for p in bench.KERNEL_SOURCES]
    assert "partition.hip" in names and "spmm.hip" in names and "arw.hip" in names


def test_cpu_baseline_states_each_part_fraction():
    """On c1 (no walks: one SpMM), the baseline names its sample as a fraction of the whole,
    and the same samples on all host cores give a context figure with the thread count."""
    import numpy as np
    from graphgen import configs
    w = configs.WORKLOADS["c1"]
    g = configs.load_graph("c1")
    X = configs.load_features("c1")
    out = bench.cpu_baseline(w, g, X, [], part_budget_s=0.05)
    assert out["cores"] == 1 and out["kind"] == "oracle" and out["value"] > 0
    assert out["parts"] and all(0 < p["fraction"] <= 1 for p in out["parts"])
    assert "%" in out["sample"] and out["all_cores"]["cores"] >= 1
    est = sum(p["seconds"] / p["fraction"] for p in out["parts"])
    assert abs(est - out["est_step_s"]) <= 1e-3 * est + 1e-3


def test_committed_counter_summary_names_the_default_kernel():
    """The committed summary is for the kernel the default run times: c5's layer-1
    aggregation fused with layer 2's update, with cache classes (the plan marks cold
    columns and the 2 GiB operand is within the classes' range)."""
    text = open(bench.COUNTER_SUMMARY).read()
    cp = bench.gather_classes({"cold_marked": 1}, 1 << 22, 128)
    assert "workload: c5" in text and f"kernel: spmm_xw_kernel<32, {'true' if cp else 'false'}>" in text


@pytest.mark.parametrize("gpus", ["2", "8"])
def test_more_than_one_gpu_is_refused(gpus):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", gpus],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    line = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in line["error"] and line["n_gpus"] == int(gpus)


def test_gather_class_rule_names_the_kernel_that_runs():
    """The bench names the instantiation the library launches: cache classes only on plans
    that marked their cold columns, for rows of more than 16 floats, with the operand above
    the 256 MiB memory-side cache and within the 4 GiB a buffer load addresses."""
    marked, unmarked = {"cold_marked": 1}, {"cold_marked": 0}
    n5 = 1 << 22
    assert bench.gather_classes(marked, n5, 128)          # c5 layer 1: 2 GiB
    assert bench.gather_classes(marked, n5, 64)           # c5 layer 2: 1 GiB
    assert not bench.gather_classes(marked, n5, 256)      # 4 GiB: beyond 32-bit offsets
    assert not bench.gather_classes(unmarked, n5, 128)
    assert not bench.gather_classes(marked, n5, 16)       # rows of a quarter line
    assert not bench.gather_classes(marked, 1 << 17, 64)  # 32 MiB: fits the memory-side cache
    assert not bench.gather_classes(marked, 1 << 18, 256) # exactly 256 MiB
