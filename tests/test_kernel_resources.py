"""Register budgets of the hot kernels, read from the compiler's resource-usage remarks
(a gfx950 cross-compile, no GPU needed).  They guard measured occupancy cliffs:

* sample_k: with 82 scalar registers (scalar registers are allocated in blocks of 16,
  so 96 per wave) the sampler ran 30% slower at 1024 x 151,936 than with 70-76 (80 per
  wave), with the same instructions otherwise;
* decode_attn_bf16_k<128>: two waves per SIMD need at most 256 vector registers, and
  the per-row chain must not spill;
* decode_attn_bf16_k<64>: four waves per SIMD (9-10% faster than three at short
  contexts) need at most 128.
"""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2505_17218_amd", "csrc")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"


def _resources(src: str, contract: str) -> dict:
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature", "-Xclang",
           "-packed-fp32-ops", "-I", os.path.join(ROOT, "include"), "-I", CSRC, f"-ffp-contract={contract}",
           "--cuda-device-only", "-c", "-o", os.devnull, os.path.join(CSRC, src),
           "-Rpass-analysis=kernel-resource-usage"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    out, cur = {}, None
    for line in r.stderr.splitlines():
        m = re.search(r"remark: Function Name: (\S+)", line)
        if m:
            cur = m.group(1)
            out[cur] = {}
            continue
        m = re.search(r"remark:\s+(TotalSGPRs|VGPRs|AGPRs|ScratchSize \[bytes/lane\]|SGPRs Spill|VGPRs Spill): (\d+)", line)
        if m and cur:
            out[cur][m.group(1)] = int(m.group(2))
    return out


needs_hipcc = pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")


@needs_hipcc
def test_sampler_scalar_registers():
    res = _resources("sampler.hip", "off")
    ks = {k: v for k, v in res.items() if "sample_k" in k}
    assert len(ks) == 8, list(res)
    for name, r in ks.items():
        assert r["TotalSGPRs"] <= 80, (name, r)
        assert r.get("ScratchSize [bytes/lane]", 0) == 0, (name, r)


@needs_hipcc
def test_decode_attention_registers():
    res = _resources("attention.hip", "fast")
    for name, r in res.items():
        if "decode_attn_bf16_k" not in name:
            continue
        vg = r["VGPRs"] + r.get("AGPRs", 0)
        limit = 256 if "ILi128E" in name else 128
        assert vg <= limit, (name, r)
        assert r.get("ScratchSize [bytes/lane]", 0) == 0, (name, r)
