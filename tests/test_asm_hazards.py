"""The inline asm of the decode kernels against the MFMA wait-state rules, on the
gfx950 device assembly of the library's own build flags (CPU only: hipcc)."""
import os
import re
import shutil
import subprocess

import pytest

from asm_scan import scan

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2605_17757_amd", "csrc")
SCANNED = {"decode_mfma.hip"}
# the units built from it (the second with the two-chunk instances only)
UNITS = ["decode_mfma.hip", "decode_mfma_wide2.hip"]


def test_inline_asm_only_in_scanned_sources():
    """The scan below covers every source with inline asm: any other kernel source
    that gains an asm statement must be added to it."""
    with_asm = set()
    for name in sorted(os.listdir(CSRC)):
        if name.endswith((".hip", ".h")):
            text = open(os.path.join(CSRC, name)).read()
            if re.search(r"\basm\s*(volatile\s*)?\(", text):
                with_asm.add(name)
    assert with_asm == SCANNED, with_asm


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="hipcc not installed")
@pytest.mark.parametrize("unit", UNITS)
def test_inline_asm_respects_mfma_wait_states(tmp_path, unit):
    from paper_2605_17757_amd import build as B
    out = tmp_path / unit.replace(".hip", ".s")
    cmd = [B.HIPCC, *B.COMMON, *B.SOURCES[unit], "--cuda-device-only", "-S",
           os.path.join(B.CSRC, unit), "-o", str(out)]
    subprocess.run(cmd, check=True, stderr=subprocess.DEVNULL)
    r = scan(out.read_text())
    assert r["blocks"] > 20  # the helpers are inlined into every instance
    assert r["war"] == [], r["war"][:5]
    assert r["raw"] == [], r["raw"][:5]
    assert r["dpp"] == [], r["dpp"][:5]
