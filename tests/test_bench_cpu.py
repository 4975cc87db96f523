"""Host-side pieces of the benchmark and the counter post-processing (no GPU)."""
import csv
import json
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2303_10384_amd import profiling  # noqa: E402
from paper_2303_10384_amd.workloads import WORKLOADS, make_lengths_labels  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_algorithmic_bytes_of_the_bpe_workload():
    w = WORKLOADS["bpe"]
    tl, ul, _ = make_lengths_labels(w)
    ab = bench.algorithmic_bytes(w, tl, ul, 4, 4)
    r_valid = int(sum(int(t) * (int(u) + 1) for t, u in zip(tl, ul)))
    assert ab["valid_rows"] == r_valid and ab["padded_rows"] == 32 * 250 * 81
    assert ab["k1_populate"] == r_valid * 1025 * 4
    assert ab["k3_grad"] == r_valid * 1025 * 4 + 648000 * 1025 * 4 + 648000 * 16
    assert ab["step"] == 2 * r_valid * 1025 * 4 + 648000 * 1025 * 4
    # bf16 logits with a float32 gradient
    ab2 = bench.algorithmic_bytes(w, tl, ul, 2, 4)
    assert ab2["k3_grad"] == r_valid * 1025 * 2 + 648000 * 1025 * 4 + 648000 * 16
    # only the rows whose gradient is not identically zero are read a second time
    r_grad = r_valid * 3 // 5
    ab3 = bench.algorithmic_bytes(w, tl, ul, 4, 4, r_grad)
    assert ab3["gradient_rows"] == r_grad and ab3["k1_populate"] == ab["k1_populate"]
    assert ab3["k3_grad"] == r_grad * 1025 * 4 + 648000 * 1025 * 4 + 648000 * 16
    assert ab3["step"] == (r_valid + r_grad) * 1025 * 4 + 648000 * 1025 * 4


def test_gradient_rows_counts_valid_rows_with_a_nonzero_element():
    import torch
    g = torch.zeros(2, 4, 3, 5)
    g[0, 1, 2, 4] = 1e-30   # a valid row (t < 3, u <= 2)
    g[0, 3, 0, 0] = 1.0     # a padding frame: not counted
    g[1, 0, 1, 2] = -2.0    # valid (t < 2, u <= 1)
    g[1, 0, 2, 0] = 5.0     # u > 1: padding, not counted
    tl = np.array([3, 2]); ul = np.array([2, 1])
    assert bench.gradient_rows(torch, g, tl, ul) == 2


def test_step_times_median_and_mean():
    class Events:  # events are plain times in ms here
        @staticmethod
        def elapsed_ms(a, b):
            return b - a
    # four steps of 1.0, 1.2, 5.0 (an outlier) and 1.1 ms, back to back
    starts, spans = [0.0, 1.0, 2.2, 7.2], [1.0, 1.2, 5.0, 1.1]
    events = [[t, t + 0.3, t + d] for t, d in zip(starts, spans)]
    median, mean = bench.step_times(Events, events, 2)
    assert abs(median - 1.15) < 1e-12
    assert abs(mean - 8.3 / 4) < 1e-12


def test_cpu_baseline_reports_pool_and_single_core_rates():
    w = WORKLOADS["tiny"]
    tl, ul, labels = make_lengths_labels(w)
    for mode in ("loss", "viterbi", "arc"):
        cb = bench.cpu_baseline(w, tl, ul, labels, budget_s=0.2, mode=mode)
        assert cb["kind"] == "oracle" and cb["unit"] == "joint-logit elements/s"
        assert cb["value"] > 0 and cb["single_core_value"] > 0 and 1 <= cb["cores"] <= 16
        assert cb["cores_available"] == len(os.sched_getaffinity(0))
        assert "freshly drawn" in cb["sample"]
        # the pool's rate cannot exceed its workers' summed single-core rates
        assert cb["value"] <= cb["single_core_value"] * cb["cores"] * 1.5


def _counter_csv(path, rows):
    os.makedirs(path, exist_ok=True)
    with open(os.path.join(path, "x_counter_collection.csv"), "w", newline="") as f:
        wr = csv.writer(f)
        wr.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        for i, (k, c, v) in enumerate(rows):
            wr.writerow([i, k, c, v])


def test_traffic_record_scales_counters_by_the_copy(tmp_path):
    copy = 1 << 30
    # the copy probe reads half its size in FETCH_SIZE units and all of it in WRITE_SIZE
    _counter_csv(tmp_path / "cf", [("__amd_rocclr_copyBuffer", "FETCH_SIZE", copy / 2048)] * 3 +
                 [("__amd_rocclr_copyBuffer", "FETCH_SIZE", 1.5)])
    _counter_csv(tmp_path / "cw", [("__amd_rocclr_copyBuffer", "WRITE_SIZE", copy / 1024)] * 3)
    kn = {"k1": "void rnnt::k1_populate<float, 8, 2, true, true>(rnnt::PopulateParams)",
          "k2": "void rnnt::k2_lattice<2, 24, 0, 1, false>(rnnt::LatticeParams)",
          "k2b": "void rnnt::k2b_posteriors<false>(rnnt::PostParams)",
          "k3": "void rnnt::k3_grad<float, float, false>(rnnt::GradParams)"}
    _counter_csv(tmp_path / "f", [(kn["k1"], "FETCH_SIZE", 1000.0), (kn["k2"], "FETCH_SIZE", 10.0),
                                  (kn["k2b"], "FETCH_SIZE", 20.0), (kn["k3"], "FETCH_SIZE", 3000.0),
                                  (kn["k3"], "FETCH_SIZE", 3002.0), (kn["k3"], "FETCH_SIZE", 2998.0)])
    _counter_csv(tmp_path / "w", [(kn["k1"], "WRITE_SIZE", 5.0), (kn["k2"], "WRITE_SIZE", 10.0),
                                  (kn["k2b"], "WRITE_SIZE", 10.0), (kn["k3"], "WRITE_SIZE", 8000.0)])
    algo = tmp_path / "bench.json"
    algo.write_text(json.dumps({"algorithmic_bytes": {"k3_grad": 14_000_000}}) + "\n")
    rec = profiling.main(["--workload", "unit", "--fetch", str(tmp_path / "f"), "--write", str(tmp_path / "w"),
                          "--copy-fetch", str(tmp_path / "cf"), "--copy-write", str(tmp_path / "cw"),
                          "--copy-bytes", str(copy), "--algorithmic", str(algo), "--out", str(tmp_path / "out")])
    assert np.isclose(rec["calibration"]["fetch_bytes_per_kib"], 2048.0)
    assert np.isclose(rec["calibration"]["write_bytes_per_kib"], 1024.0)
    k3 = rec["kernels"]["k3_grad"]
    assert k3["fetch_bytes"] == 3000 * 2048 and k3["write_bytes"] == 8000 * 1024
    assert rec["hbm_bytes_per_launch"] == 3000 * 2048 + 8000 * 1024
    assert k3["algorithmic_bytes"] == 14_000_000
    assert rec["source_digest"] == profiling.source_digest(profiling.KERNEL_SOURCES)
    saved = json.loads((tmp_path / "out" / "k3_grad_unit_traffic.json").read_text())
    assert saved["hbm_bytes_per_launch"] == rec["hbm_bytes_per_launch"]


def test_stale_traffic_record_is_ignored(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "PROFILE_DIR", str(tmp_path))
    rec = {"hbm_bytes_per_launch": 123, "source_digest": "0" * 16}
    (tmp_path / "k3_grad_bpe_traffic.json").write_text(json.dumps(rec))
    assert bench.profiled_traffic("bpe") is None
    rec["source_digest"] = profiling.source_digest(profiling.KERNEL_SOURCES)
    (tmp_path / "k3_grad_bpe_traffic.json").write_text(json.dumps(rec))
    assert bench.profiled_traffic("bpe") == 123


def test_gradient_rows_of_a_16_bit_gradient_are_counted_in_float32():
    # a row whose tiny elements an fp16 store rounds to 0 still needed its logits read
    import torch
    tl, ul = np.array([2, 1], np.int32), np.array([1, 0], np.int32)
    exact = torch.zeros((2, 2, 2, 3), dtype=torch.float32)
    exact[0, 0, 0, 1] = 1e-9   # below fp16's smallest subnormal
    exact[0, 1, 1, 2] = 0.25
    exact[1, 0, 0, 0] = -3e-9
    exact[1, 1, 1, 0] = 1.0    # padding row: not counted
    g16 = exact.to(torch.float16)
    assert bench.gradient_rows(torch, g16, tl, ul) == 1
    calls = []

    def call_f32(g32):
        calls.append(g32.dtype)
        g32.copy_(exact)

    assert bench.gradient_rows_f32(torch, g16, tl, ul, call_f32) == 3
    assert calls == [torch.float32]
    assert bench.gradient_rows_f32(torch, exact, tl, ul, call_f32) == 3 and len(calls) == 1
