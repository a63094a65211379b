"""The FP8 MFMAs compile to the unscaled encoding (CPU; hipcc cross-compiles
gfx950 assembly of this repository's own sources).

The kernels call the scaled builtin with both E8M0 scale operands 0, which
the compiler turns into the unscaled v_mfma_f32_{16x16x128,32x32x64}_f8f6f4
(no block scales; the fp32 scales are applied to the results).  If the
scaled form were emitted with those operands, every product would be scaled
by 2^-254; this test fails at build time instead of on the GPU."""
import concurrent.futures as cf
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_10493_amd", "csrc")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
SOURCES = ["ffn_prefill.hip", "ffn_decode.hip", "ffn_decode_combine.hip"]


def _asm(src, tmp):
    out = os.path.join(tmp, src + ".s")
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "--cuda-device-only", "-S",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC, os.path.join(CSRC, src), "-o", out]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-2000:]
    with open(out) as f:
        return f.read()


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
def test_fp8_mfmas_are_unscaled(tmp_path):
    with cf.ThreadPoolExecutor(len(SOURCES)) as ex:
        asm = dict(zip(SOURCES, ex.map(lambda s: _asm(s, str(tmp_path)), SOURCES)))
    for src, text in asm.items():
        scaled = re.findall(r"v_mfma_scale_\w+", text)
        plain = re.findall(r"v_mfma_f32_(?:16x16x128|32x32x64)_f8f6f4", text)
        assert not scaled, f"{src}: scaled MFMA encoding emitted ({len(scaled)})"
        assert plain, f"{src}: no FP8 MFMA found"
