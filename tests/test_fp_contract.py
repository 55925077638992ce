"""Kernels whose binary32 results decide integers are built without multiply-add fusion:
their gfx950 assembly, compiled the way the build script compiles them, holds no fused
multiply-add (the library's exact decisions would otherwise round differently from a
plain IEEE evaluation of the same steps)."""
import os
import re
import subprocess

import pytest

from paper_2404_09267_amd import build as B

FMA = re.compile(r"\bv_(fma|fmac|fmaak|fmamk|pk_fma)_f32\b|\bv_fma_mix")


@pytest.mark.parametrize("src", ["merge.hip", "unstitch.hip"])
def test_no_fused_multiply_add(tmp_path, src):
    assert src in B.EXACT_FP32
    out = tmp_path / (src + ".s")
    cmd = [B.hipcc(), *B.HIP_FLAGS, "-ffp-contract=off", "--cuda-device-only", "-S",
           os.path.join(B.CSRC, src), "-o", str(out)]
    subprocess.run(cmd, check=True, capture_output=True)
    hits = [l for l in out.read_text().splitlines() if FMA.search(l)]
    assert not hits, hits[:5]
