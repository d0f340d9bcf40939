"""Host-side logic of bench.py (no GPU): the one-GPU refusal, the algorithmic attention
bytes the roofline divides by, the GEMM flop counts, and the provenance check that
reports the counted attention traffic only for the kernel sources it was counted on."""
import hashlib
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2505_17218_amd import synth  # noqa: E402


def test_multi_gpu_request_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_attention_bytes_closed_form_headline():
    """Per layer and decode step t (context P + t): the group's P shared prompt positions
    once per group, every row's own t positions, q and o per row.  Summed over t = 1..T-1
    this is (T-1)(N/G P + N qo/kvb) kvb + N kvb T(T-1)/2; at the 1.5B shape with 1024
    sequences, prompt 256 and 1024 tokens the mean per launch is 576,716,800 bytes."""
    wl = synth.WORKLOADS["1.5b-b1024"]
    s = wl.shape
    N, P, G, T = wl.n_seqs, wl.prompt_len, wl.group, wl.gen_len
    kvb = 2 * s.n_kv_heads * s.head_dim * 2
    qo = 2 * s.n_heads * s.head_dim * 2
    assert (kvb, qo) == (1024, 6144)
    uniq, logi = bench.attention_bytes(wl, T)
    want_u = ((T - 1) * ((N // G) * P * kvb + N * qo) + N * kvb * T * (T - 1) // 2) * s.n_layers
    want_l = ((T - 1) * (N * P * kvb + N * qo) + N * kvb * T * (T - 1) // 2) * s.n_layers
    assert uniq == want_u and logi == want_l
    assert uniq / (T - 1) / s.n_layers == 576_716_800
    # the shared prompt pages are the only difference between the two counts
    assert logi - uniq == (T - 1) * (N - N // G) * P * kvb * s.n_layers


def test_gemm_flops_headline():
    wl = synth.WORKLOADS["1.5b-b1024"]
    f = bench.gemm_flops(wl, 1024)
    L = wl.shape.n_layers
    assert f["gemm_lm_head"] == 2.0 * 1024 * 151936 * 1536  # 478 GFLOP per step
    assert f["gemm_qkv"] == 2.0 * 1024 * 2048 * 1536 * L
    assert f["gemm_o"] == 2.0 * 1024 * 1536 * 1536 * L
    assert f["gemm_gate_up"] == 2.0 * 1024 * 17920 * 1536 * L
    assert f["gemm_down"] == 2.0 * 1024 * 1536 * 8960 * L


def test_traffic_reported_only_for_the_counted_sources(tmp_path, monkeypatch):
    for rel in bench.ATTN_TRAFFIC["sources"]:
        dst = tmp_path / rel
        dst.parent.mkdir(parents=True, exist_ok=True)
        shutil.copyfile(os.path.join(ROOT, rel), dst)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    digests = {rel: hashlib.sha256((tmp_path / rel).read_bytes()).hexdigest() for rel in bench.ATTN_TRAFFIC["sources"]}
    if digests != bench.ATTN_TRAFFIC["sources"]:
        pytest.skip("the attention sources changed since the traffic was counted (bench reports null)")
    assert bench.measured_attention_traffic("1.5b-b1024") == bench.ATTN_TRAFFIC["bytes_per_launch"]
    assert bench.measured_attention_traffic("3b-b1024") is None  # counted on the 1.5B workload only
    rel = next(iter(bench.ATTN_TRAFFIC["sources"]))
    (tmp_path / rel).write_bytes((tmp_path / rel).read_bytes() + b"\n// edited\n")
    assert bench.measured_attention_traffic("1.5b-b1024") is None
