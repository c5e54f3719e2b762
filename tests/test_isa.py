"""Code-generation guard (no GPU needed): no kernel of the library may address memory
with FLAT instructions.  A generic pointer that can point into LDS compiles to FLAT
loads, and FLAT decides the LDS aperture from the register address before the
instruction's immediate offset is added; when the compiler folds part of an LDS index
into that offset, the register address can fall below the aperture and the access goes
to an illegal global address.  Every LDS access must therefore be a ds_* instruction and
every global access a global_* one."""
import glob
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2003_05148_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


@pytest.mark.skipif(not os.path.exists(HIPCC) and shutil.which("hipcc") is None, reason="hipcc not installed")
@pytest.mark.parametrize("src", sorted(os.path.basename(p) for p in glob.glob(os.path.join(CSRC, "*.hip"))))
def test_no_flat_memory_instructions(src, tmp_path):
    out = tmp_path / (src + ".s")
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-ffp-contract=off",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "--cuda-device-only", "-S",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC, os.path.join(CSRC, src), "-o", str(out)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    flat = [l.strip() for l in out.read_text().splitlines() if re.match(r"\s+flat_(load|store|atomic)", l)]
    assert not flat, f"{src}: FLAT memory instructions: {flat[:5]}"
