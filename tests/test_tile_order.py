"""Host checks of index and bit arithmetic that the gfx950 kernels use, compiled with hipcc
for the host: the upper-triangle tile order of the Gram kernels (csrc/tile_order.hpp) hits every
tile exactly once, the solver's exchange record (csrc/xchg_record.hpp) round-trips, and the
working-set candidate words (csrc/ws_record.hpp) keep the fp64 order and round-trip."""
import os
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(os.path.dirname(HERE), "paper_2311_14908_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _run(src, tmp_path):
    exe = tmp_path / os.path.splitext(src)[0]
    subprocess.run([HIPCC, "-O2", "-x", "hip", "--offload-arch=gfx950", "-I", CSRC, os.path.join(HERE, src), "-o",
                    str(exe)], check=True, capture_output=True)
    return subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
def test_tile_order_is_bijective(tmp_path):
    assert _run("tile_order_check.cpp", tmp_path).startswith("ok")


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
def test_exchange_record_round_trip(tmp_path):
    assert _run("xchg_record_check.cpp", tmp_path).startswith("ok")


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
def test_working_set_candidate_words(tmp_path):
    assert _run("ws_record_check.cpp", tmp_path).startswith("ok")
