"""Host check of the bf16 attention's query-tile enumeration (whole tiles, key-split tiles,
XCD remap): compiles tests/tile_order_check.cpp against the kernels' internal header and runs
it on the CPU."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_32415_amd", "csrc")


def _hipcc():
    return shutil.which("hipcc") or ("/opt/rocm/bin/hipcc" if os.path.exists("/opt/rocm/bin/hipcc") else None)


def test_tile_orders_are_bijections_that_spread_split_tiles(tmp_path):
    cc = _hipcc()
    if cc is None:
        pytest.skip("hipcc not found")
    exe = str(tmp_path / "tile_order_check")
    src = os.path.join(ROOT, "tests", "tile_order_check.cpp")
    r = subprocess.run([cc, "-x", "hip", "--offload-arch=gfx950", "-O2", "-std=c++17", "-I", CSRC, src, "-o", exe],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "violations 0" in r.stdout
