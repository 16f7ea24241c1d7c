"""The row copy engine's chunk-to-row map, checked on the host for every
row width the library accepts (no GPU needed): each 16- or 4-byte chunk
of a 64-row tile must decode to its own row and column, including widths
with one chunk per row or one tail word, whose divisor of 1 has no 32-bit
multiplier."""
import os
import subprocess

from tests import helpers

CSRC = os.path.join(helpers.ROOT, "paper_2606_02916_amd", "csrc")


def test_chunk_to_row_map_for_every_row_width():
    exe = helpers.build_helper("copy_geom_map.cpp", extra=["-std=c++17", "-I" + CSRC],
                               compiler="g++", subdir="host")
    out = subprocess.run([exe], capture_output=True, text=True)
    assert out.returncode == 0, out.stdout
    assert int(out.stdout.split()[-1]) == 32768 // 4
