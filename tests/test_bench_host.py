"""Host-side logic of bench.py (no GPU): the one-GPU guard, the roofline's algorithmic work, and
the rocprofv3 counter ingest that writes profiles/lmhead_traffic.json."""
import csv
import json
import os
import subprocess
import sys

import pytest

import bench
from workloads import CONFIGS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_with_a_message():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120)
    assert res.returncode == 2
    assert "one GPU" in res.stderr
    assert res.stdout == ""


def test_lmhead_work_is_the_fused_launch_minimum():
    # W and h read once, 12 bytes of results per row; 2 T d V flops
    cfg = CONFIGS["llada8b_b1"]
    nbytes, flops = bench.lmhead_work(cfg, 32)
    assert nbytes == 126464 * 4096 * 2 + 32 * 4096 * 2 + 12 * 32
    assert flops == 2.0 * 32 * 4096 * 126464
    cfg = CONFIGS["tiny_f32_b1"]
    nbytes, _ = bench.lmhead_work(cfg, 7)
    assert nbytes == cfg.vocab * cfg.hidden * 4 + 7 * cfg.hidden * 4 + 12 * 7


def test_attention_bytes_count_the_prefix_once_and_the_block_in_and_out():
    cfg = CONFIGS["dream7b_b64"]
    T, S = 100, 5000
    e = 2
    want = 2 * S * cfg.hkv * cfg.head_dim * e + T * (2 * cfg.hq + 2 * cfg.hkv) * cfg.head_dim * e
    assert bench.attention_bytes(cfg, T, S) == want


@pytest.mark.parametrize("name,T,bound", [("llada8b_b1", 32, "hbm"), ("dream7b_b64", 9626, "mfma"),
                                          ("tiny_f32_b1", 32, "alu")])
def test_roofline_bound_and_fraction(name, T, bound, monkeypatch):
    monkeypatch.setattr(bench, "measured_traffic", lambda workload: None)
    cfg = CONFIGS[name]
    ms = 0.5
    r = bench.roofline_of(cfg, T, 512, ms, with_attn=False)
    assert r["bound"] == bound
    nbytes, flops = bench.lmhead_work(cfg, T)
    achieved = nbytes / (ms * 1e-3) / 1e9 if bound == "hbm" else flops / (ms * 1e-3) / 1e12
    assert r["achieved"] == pytest.approx(achieved)
    assert r["frac"] == pytest.approx(achieved / r["peak"])
    with_attn = bench.roofline_of(cfg, T, 512, ms, with_attn=True)
    assert with_attn["algorithmic_bytes"] == nbytes + bench.attention_bytes(cfg, T, 512)
    assert with_attn["includes_attention"]


def _write_run(directory, run, counter, rows):
    d = os.path.join(directory, f"{run}_{counter}", "host", "1")
    os.makedirs(d)
    with open(os.path.join(d, "r_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name",
                                          "Counter_Value"])
        w.writeheader()
        for i, (kernel, value) in enumerate(rows):
            w.writerow({"Dispatch_Id": i, "Kernel_Name": kernel, "Counter_Name": counter,
                        "Counter_Value": value})


def test_counter_ingest_scales_by_the_copy_and_tags_the_source(tmp_path, monkeypatch):
    out = tmp_path / "traffic.json"
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(out))
    gib_kib = (1 << 30) / 1024
    # the copy reads 0.8x and writes 1.25x its true KiB: factors 1.25 and 0.8; a small copy
    # dispatch (not a 1 GiB one) is ignored
    _write_run(tmp_path, "copy", "FETCH_SIZE", [("__amd_rocclr_copyBuffer", 0.8 * gib_kib),
                                                ("__amd_rocclr_copyBuffer", 0.8 * gib_kib),
                                                ("__amd_rocclr_copyBuffer", 10.0)])
    _write_run(tmp_path, "copy", "WRITE_SIZE", [("__amd_rocclr_copyBuffer", 1.25 * gib_kib)])
    kernel = bench.lmhead_kernel_name("bf16", 32)
    _write_run(tmp_path, "llada8b_b1", "FETCH_SIZE", [(f"void eb::{kernel}<16>(...)", 1000.0),
                                                      (f"void eb::{kernel}<16>(...)", 3000.0),
                                                      ("void eb::step_finish_kernel<128>", 9e9)])
    _write_run(tmp_path, "llada8b_b1", "WRITE_SIZE", [(f"void eb::{kernel}<16>(...)", 40.0)])
    assert bench.ingest_counters(str(tmp_path)) == 0
    rec = json.loads(out.read_text())["llada8b_b1"]
    assert rec["kernel"] == kernel
    assert rec["fetch_kib"] == pytest.approx(2000.0)
    assert rec["write_kib"] == pytest.approx(40.0)
    assert rec["dispatches"] == [2, 1]
    assert rec["bytes_per_launch"] == pytest.approx(2000.0 * 1024 * 1.25 + 40.0 * 1024 * 0.8)
    assert rec["source_hash"] == bench.lmhead_source_hash()
    # the bench line reads it back only while the kernel source is the one it was taken on
    assert bench.measured_traffic("llada8b_b1") == pytest.approx(rec["bytes_per_launch"])
    monkeypatch.setattr(bench, "lmhead_source_hash", lambda: "0" * 16)
    assert bench.measured_traffic("llada8b_b1") is None
