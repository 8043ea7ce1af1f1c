"""bench.py's host-side contract, on the CPU: more than one GPU is refused
before any GPU work, the roofline object picks the bound from the product's
arithmetic intensity, measured HBM traffic is used only for the exact
configuration and kernel sources it was taken on, and the CPU baseline is
the oracle on whole steps of the workload."""
import json
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
import paper_2309_08978_amd as nj  # noqa: E402
import workloads  # noqa: E402


def test_more_than_one_gpu_is_refused(capsys):
    assert bench.main(["--gpus", "2"]) == 2
    assert "one GPU only" in capsys.readouterr().err


def test_roofline_bound_follows_arithmetic_intensity():
    prefill = workloads.workload("llama2_7b_prefill512_f32")[0]      # AI ~ 220 FLOP/B > fp32 ridge 19.7
    r = bench.roofline_of(prefill, 400.0)
    assert r["bound"] == "mfma" and r["unit"] == "TFLOP/s" and r["peak"] == 157.3
    assert r["achieved"] == pytest.approx(prefill.flops / 400e-6 / 1e12)
    assert r["frac"] == pytest.approx(r["achieved"] / 157.3)
    decode = workloads.workload("llama2_7b_decode_f16")[0]           # AI ~ 1 FLOP/B: HBM
    r = bench.roofline_of(decode, 20.0)
    assert r["bound"] == "hbm" and r["unit"] == "GB/s" and r["peak"] == 8000.0
    assert r["achieved"] == pytest.approx(decode.bytes / 20e-6 / 1e9)
    q4 = workloads.workload("llama2_7b_decode_q4")[0]                # no matrix cores: HBM
    assert bench.roofline_of(q4, 10.0)["bound"] == "hbm"


def test_measured_traffic_needs_the_exact_config_and_sources(tmp_path):
    nj.load()
    info = "name=gemm_f32w_64x32x16_k4_s4 split=2"
    key = "bart_base_layer_seq128_f32|bart.ffn_down|gemm_f32w_64x32x16_k4_s4|2"
    db = tmp_path / "traffic.json"
    db.write_text(json.dumps({key: {"digest": nj.kernel_digest(), "hbm_bytes_per_launch": 12345}}))
    assert bench.measured_traffic(str(db), "bart_base_layer_seq128_f32", "bart.ffn_down", info) == 12345
    assert bench.measured_traffic(str(db), "bart_base_layer_seq128_f32", "bart.ffn_down",
                                  "name=gemm_f32w_64x32x16_k4_s4 split=4") is None
    db.write_text(json.dumps({key: {"digest": "0" * 16, "hbm_bytes_per_launch": 12345}}))
    assert bench.measured_traffic(str(db), "bart_base_layer_seq128_f32", "bart.ffn_down", info) is None
    assert bench.measured_traffic(str(tmp_path / "missing.json"), "w", "op", info) is None


def test_cpu_baseline_runs_whole_oracle_steps():
    r = bench.cpu_baseline("matmul_64x768x768_f32", 0.01)
    assert r["kind"] == "oracle" and r["unit"] == "GFLOP/s" and r["cores"] >= 1 and r["value"] > 0
    assert "full step(s) of 1/1 products" in r["sample"]
