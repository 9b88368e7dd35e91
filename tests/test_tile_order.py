"""The Gram kernels enumerate upper-triangle tiles in super-tile order (csrc/tile_order.hpp);
compiled for the host, the mapping must hit every tile (ti <= tj < nt) exactly once."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(os.path.dirname(HERE), "paper_2311_14908_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
def test_tile_order_is_bijective(tmp_path):
    exe = tmp_path / "tile_order_check"
    subprocess.run([HIPCC, "-O2", "-x", "hip", "--offload-arch=gfx950", "-I", CSRC,
                    os.path.join(HERE, "tile_order_check.cpp"), "-o", str(exe)], check=True, capture_output=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout
    assert out.startswith("ok")
