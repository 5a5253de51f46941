"""Host logic of bench.py (no GPU): the one-GPU guard, the FLOP count behind
MFU, the stale-source check of stored counter traffic, and the arithmetic
that turns two rocprofv3 counter passes into HBM bytes per launch."""
import csv
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import oracle  # noqa: E402
from paper_2609_28568_amd import synth  # noqa: E402


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_flops_per_token_counts_the_oracle_matmul_weights():
    """6 FLOPs per matmul weight per token, the head over the real vocabulary
    only, plus causal attention: for query t, q.k and p.v each take 2 C (t+1)
    FLOPs forward, twice that backward; averaged over the T positions."""
    w = synth.WORKLOADS["gpt2_124m"]
    cfg = oracle.Config.from_dict({**w, **synth.OPTIM})
    shapes = oracle.param_shapes(cfg)
    n_mm = sum(int(np.prod(shapes[k])) for k in ("qkvw", "attprojw", "fcw", "fcprojw"))
    n_mm += w["vocab"] * shapes["wte"][1]   # tied head, real rows only
    T, C, L = w["T"], w["d_model"], w["n_layer"]
    per_query = [3 * 2 * (2 * C * (t + 1)) for t in range(T)]
    attn = L * sum(per_query) / T
    assert bench.flops_per_token(w) == pytest.approx(6 * n_mm + attn, rel=1e-12)
    assert bench.flops_per_token(w) == 797_870_592


def test_stored_traffic_goes_stale_when_its_sources_change(monkeypatch):
    tag, wl = "gemm_dw_grouped", "gpt2_124m"
    path = bench.traffic_path(tag, wl)
    if not os.path.exists(path):
        pytest.skip("no stored traffic record")
    real = bench.kernel_source_hash(tag, wl)
    import json
    stored = json.load(open(path))
    if stored["source_sha256"] == real:
        assert bench.traffic_from_profiles(tag, wl) == stored["bytes_per_launch"]
    monkeypatch.setattr(bench, "kernel_source_hash", lambda t, w: "0" * 64)
    assert bench.traffic_from_profiles(tag, wl) is None


def _counter_csv(path, counter, rows):
    with open(path, "w", newline="") as f:
        wr = csv.DictWriter(f, fieldnames=["Kernel_Name", "Grid_Size", "Counter_Name", "Counter_Value"])
        wr.writeheader()
        for name, grid, kib in rows:
            wr.writerow({"Kernel_Name": name, "Grid_Size": grid, "Counter_Name": counter, "Counter_Value": kib})


def test_counter_passes_scaled_by_the_calibration_copy(tmp_path):
    """FETCH_SIZE and WRITE_SIZE (KiB per dispatch) of the class's kernels,
    averaged over dispatches, each scaled so that the 1 GiB copy reads as
    1 GiB, times the kernels per launch (the attention backward is two)."""
    k1 = "void (anonymous namespace)::attn_bwd_dq_kernel<128>(AttnArgs)"
    k2 = "void (anonymous namespace)::attn_bwd_dkdv8_kernel<128>(AttnArgs)"
    copy = "__amd_rocclr_copyBuffer"
    fetch, write = tmp_path / "f.csv", tmp_path / "w.csv"
    # the copy's FETCH_SIZE reads half the bytes, its WRITE_SIZE all of them
    _counter_csv(fetch, "FETCH_SIZE", [(k1, 1024, 100.0), (k2, 1024, 300.0), (copy, 1 << 20, 512.0 * 1024),
                                       (copy, 64, 1.0), ("other_kernel", 1024, 9e9)])
    _counter_csv(write, "WRITE_SIZE", [(k1, 1024, 10.0), (k2, 1024, 30.0), (copy, 1 << 20, 1024.0 * 1024)])
    d = bench.pmc_summary("attn_bwd", "qwen3_06b_lora", str(fetch), str(write), "cmd")
    assert d["fetch_scale"] == pytest.approx(2.0)
    assert d["write_scale"] == pytest.approx(1.0)
    assert d["dispatches"] == 2
    mean_fetch, mean_write = 200.0 * 1024, 20.0 * 1024
    assert d["bytes_per_launch"] == pytest.approx(2 * (2.0 * mean_fetch + mean_write))
    assert d["command"] == "cmd"
    assert d["source_sha256"] == bench.kernel_source_hash("attn_bwd", "qwen3_06b_lora")


def test_counter_pass_without_the_calibration_copy_is_an_error(tmp_path):
    fetch, write = tmp_path / "f.csv", tmp_path / "w.csv"
    k = "void (anonymous namespace)::attn_bwd_dq_kernel<128>(AttnArgs)"
    _counter_csv(fetch, "FETCH_SIZE", [(k, 1024, 100.0)])
    _counter_csv(write, "WRITE_SIZE", [(k, 1024, 10.0)])
    with pytest.raises(SystemExit):
        bench.pmc_summary("attn_bwd", "qwen3_06b_lora", str(fetch), str(write), "")
