"""CPU check of the swept-tile index arithmetic (tests/layout_check.hip).

The sweeps' LDS addresses come from the helpers in csrc/sweep.hpp, which are
host-callable.  layout_check.hip simulates every DMA instruction of a tile
with them and checks each fragment and transposing read the kernels issue
against the rows and features its MFMA operand needs, plus bounds, coverage
and bank conflicts, for every row width the interface accepts.  Built with
hipcc and run on the host; nothing launches on a GPU.
"""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _hipcc():
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    return None


def test_swept_tile_layout(tmp_path):
    cc = _hipcc()
    if cc is None:
        pytest.skip("hipcc not available")
    exe = str(tmp_path / "layout_check")
    cmd = [cc, "--offload-arch=gfx950", "-O1", "-std=c++17",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(ROOT, "paper_2410_17243_amd", "csrc"),
           os.path.join(ROOT, "tests", "layout_check.hip"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr[-4000:]
    assert "layout ok (8 row widths)" in r.stdout
