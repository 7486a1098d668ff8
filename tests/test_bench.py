"""bench.py's accounting and contract pieces that need no GPU."""
import subprocess
import sys

import numpy as np
import pytest

import bench
import synth


def _brute_pairs(B, H, Nq, Nk, causal):
    i = np.arange(Nq)[:, None]
    j = np.arange(Nk)[None, :]
    vis = (j <= i + (Nk - Nq)) if causal else np.ones((Nq, Nk), bool)
    return int(vis.sum()) * B * H


@pytest.mark.parametrize("Nq,Nk,causal", [(5, 5, True), (3, 9, True), (7, 4, False), (128, 128, True)])
def test_visible_pairs_brute_force(Nq, Nk, causal):
    w = synth.Workload("t", 2, 3, Nq, Nk, 64, 64, "bf16", causal)
    assert bench.visible_pairs(w) == _brute_pairs(2, 3, Nq, Nk, causal)
    assert bench.algorithmic_flops(w) == 2.0 * 128 * _brute_pairs(2, 3, Nq, Nk, causal)


def test_workload_figures():
    c4 = synth.WORKLOADS["causal_long_b1h32_n16384_d128_bf16_qk_sigma3"]
    assert bench.visible_pairs(c4) == 32 * 16384 * 16385 // 2 == 4_295_229_440
    assert bench.compulsory_bytes(c4, 2) == 4 * 32 * 16384 * 128 * 2
    c5 = synth.WORKLOADS["decode_b64h32_nk8192_d128_bf16"]
    assert bench.compulsory_bytes(c5, 2) == 64 * 32 * ((128 + 8192 * 256) * 2 + 128 * 2)


def test_traffic_is_gated_on_kernel_source(monkeypatch):
    real = bench.kernel_source_hash("prefill_bf16")
    monkeypatch.setattr(bench, "kernel_source_hash", lambda k: "0" * 16)
    assert bench.measured_traffic("prefill_bf16", "causal_long_b1h32_n16384_d128_bf16_qk_sigma3") is None
    monkeypatch.setattr(bench, "kernel_source_hash", lambda k: real)
    assert bench.measured_traffic("prefill_bf16", "some_other_workload") is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, bench.__file__, "--gpus", "2"], capture_output=True, text=True)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_backward_flops_are_two_and_a_half_forwards():
    for name in ("causal_long_b1h32_n16384_d128_bf16_qk_sigma3", "mha_b4h8_n1024_d64_bf16"):
        w = synth.WORKLOADS[name]
        assert bench.backward_flops(w) == 2.5 * bench.algorithmic_flops(w)


def test_config_records():
    ws = synth.WORKLOADS
    r = bench.config_record(ws["causal_b2h16_n4096_d128_bf16"], 0.1, 2)
    assert r["bound"] == "mfma" and r["out"] == "bf16"
    assert r["tflops"] == round(bench.algorithmic_flops(ws["causal_b2h16_n4096_d128_bf16"]) / 1e-4 / 1e12, 2)
    assert r["frac"] == round(r["tflops"] / bench.PEAK_BF16_TFLOPS, 4)
    r = bench.config_record(ws["decode_b64h32_nk8192_d128_bf16"], 1.0, 2)
    assert r["bound"] == "hbm" and abs(r["frac"] - r["GBps"] / bench.PEAK_HBM_GBS) < 1e-4
    r = bench.config_record(ws["single_head_f32_n128_d64"], 0.02, 4)
    assert r["bound"] == "latency" and r["frac"] is None
