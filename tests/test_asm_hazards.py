"""The inline asm of the decode kernels against the MFMA wait-state rules, on the
gfx950 device assembly of the library's own build flags (CPU only: hipcc)."""
import os
import shutil
import subprocess

import pytest

from asm_scan import scan

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="hipcc not installed")
def test_inline_asm_respects_mfma_wait_states(tmp_path):
    from paper_2605_17757_amd import build as B
    src = "decode_mfma.hip"
    out = tmp_path / "decode_mfma.s"
    cmd = [B.HIPCC, *B.COMMON, *B.SOURCES[src], "--cuda-device-only", "-S",
           os.path.join(B.CSRC, src), "-o", str(out)]
    subprocess.run(cmd, check=True, stderr=subprocess.DEVNULL)
    r = scan(out.read_text())
    assert r["blocks"] > 100  # the helpers are inlined into every instance
    assert r["war"] == [], r["war"][:5]
    assert r["raw"] == [], r["raw"][:5]
    assert r["dpp"] == [], r["dpp"][:5]
