"""Register budget of the gfx950 kernels, checked on the CPU (hipcc
cross-compiles): every kernel keeps its values in registers (no spill to
per-lane scratch, whose stores and reloads travel through the memory
hierarchy and add HBM traffic), and the attention kernel keeps two
wavefronts per SIMD, which its paired orders rely on."""
import os
import re
import shutil
import subprocess

import pytest

from paper_2606_22968_amd import build

HIP_SOURCES = ["chunk_attn.hip", "kv_append.hip", "lse_merge.hip"]


def resource_report(src, out_dir):
    """Per kernel: the figures hipcc's kernel-resource-usage remarks print."""
    if shutil.which(build.HIPCC) is None and not os.path.exists(build.HIPCC):
        pytest.skip("hipcc not available")
    obj = os.path.join(out_dir, os.path.splitext(src)[0] + ".o")
    cmd = [build.HIPCC, *build.FLAGS, "-Rpass-analysis=kernel-resource-usage", "-x", "hip", "-c",
           os.path.join(build.CSRC, src), "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-2000:]
    kernels, cur = {}, None
    for line in res.stderr.splitlines():
        m = re.search(r"remark:\s+Function Name: (\S+)", line)
        if m:
            cur = kernels.setdefault(m.group(1), {})
            continue
        m = re.search(r"remark:\s+(.+?):\s+(\d+)\b", line)
        if m and cur is not None:
            cur[m.group(1).strip()] = int(m.group(2))
    assert kernels, f"no resource remarks for {src}"
    return kernels


@pytest.mark.parametrize("src", HIP_SOURCES)
def test_no_register_spills(src, tmp_path):
    for name, r in resource_report(src, str(tmp_path)).items():
        assert r.get("VGPRs Spill", 0) == 0, f"{name}: {r}"
        assert r.get("ScratchSize [bytes/lane]", 0) == 0, f"{name}: {r}"


def test_attention_two_waves_per_simd(tmp_path):
    report = resource_report("chunk_attn.hip", str(tmp_path))
    attn = {n: r for n, r in report.items() if "chunk_attn_kernel" in n}
    assert len(attn) == 4, sorted(report)  # head_dim 64/128, one or two stores
    for name, r in attn.items():
        assert r["Occupancy [waves/SIMD]"] >= 2, f"{name}: {r}"
        assert r["VGPRs"] + r.get("AGPRs", 0) <= 256, f"{name}: {r}"
