"""Host logic of bench.py: algorithmic units, least bytes and roofline
bounds of each call, the committed-profile lookup, and the single-GPU
refusal (none of it touches a GPU)."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
from paper_2412_04787_amd import workloads as W  # noqa: E402


def test_units_of_the_hidden_4096_block():
    wl = W.WORKLOADS["llama_h4096"]
    u = bench.algorithmic_units(wl)
    M = 8192
    weights = 4 * 4096 * 4096 + 3 * 4096 * 11008
    assert wl.n_weights == weights
    assert u["fwd"] == 2 * M * weights
    assert u["bwd"] == u["bwd_sr"] == 4 * M * weights
    assert u["bwd_dx"] == u["bwd_dw"] == 2 * M * weights
    assert u["fwd"] + u["bwd"] == wl.train_flops
    assert u["sr"] == pytest.approx(4.5 * weights)          # 0.25 + 4 + 0.25 B per weight
    assert u["adamw_sr"] == pytest.approx(20.5 * weights)   # g, m, v read; m, v written; codes
    assert u["upd_force"] == pytest.approx(16.5 * weights)  # three selection passes, then the update
    # act-quant: 4 distinct inputs (q/k/v share one, gate/up one), bf16 in, 1 B out, 4 B scale a row
    widths = [4096, 4096, 4096, 11008]
    assert u["act_quant"] == sum(M * k * 3 + 4 * M for k in widths)


def test_every_block_is_mfma_bound():
    """Each GEMM call's least bytes at 8 TB/s take less time than its flops at
    the dtype's peak (the hidden-768 forward comes closest, near the ridge)."""
    for name in ("llama_h768", "llama_h2048", "llama_h4096", "llama_h2048_int4", "llama_h2048_int3"):
        wl = W.WORKLOADS[name]
        u, mb = bench.algorithmic_units(wl), bench.gemm_min_bytes(wl)
        peak = {"fwd": 5000.0, "bwd": 2500.0, "bwd_sr": 2500.0, "bwd_dx": 2500.0, "bwd_dw": 2500.0}
        for k, p in peak.items():
            t_flops = u[k] / (p * 1e12)
            t_bytes = mb[k] / (bench.PEAK_HBM_GBS * 1e9)
            assert t_bytes < t_flops, (name, k, t_bytes, t_flops)


def test_least_bytes_of_the_fused_call():
    """The fused backward reads dY and the quantised inputs once, reads and
    writes the codes, writes dX: no dW."""
    wl = W.WORKLOADS["llama_h768"]
    mb = bench.gemm_min_bytes(wl)
    M = wl.M
    dy = sum(M * l.d_out * 2 for l in wl.linears)
    dx = sum(M * l.d_in * 2 for l in wl.linears)
    xq = sum(M * wl.input_width(n) + 4 * M for n in wl.inputs)
    assert mb["bwd_sr"] == pytest.approx(dy + xq + 2 * 0.25 * wl.n_weights + dx)
    assert mb["bwd"] - mb["bwd_sr"] == pytest.approx(4 * wl.n_weights - 0.25 * wl.n_weights)


def test_traffic_read_only_from_a_profile_of_the_current_sources(tmp_path, monkeypatch):
    prof = tmp_path / "profiles"
    prof.mkdir()
    (tmp_path / "paper_2412_04787_amd").mkdir()
    for f in ("csrc", "build_lib.py"):
        os.symlink(os.path.join(ROOT, "paper_2412_04787_amd", f), tmp_path / "paper_2412_04787_amd" / f)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    h = bench.kernel_source_hash()
    body = "# comment = 1\nkernel_source_hash = {}\nfetch_write_bytes_per_launch = 1234\n" \
           "gemm_kernel_fetch_write_bytes = 1000\n"
    (prof / "bwd_sr_wl_counters.txt").write_text(body.format(h))
    assert bench.read_traffic("bwd_sr", "wl") == 1234.0
    assert bench.read_traffic("bwd_sr", "wl", kernel_only=True) == 1000.0
    (prof / "bwd_sr_wl_counters.txt").write_text(body.format("0" * 16))
    assert bench.read_traffic("bwd_sr", "wl") is None          # taken on other sources
    assert bench.read_traffic("fwd", "wl") is None             # no summary


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in r.stdout
