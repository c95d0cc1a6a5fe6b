"""The row kernels' unit layout on the host (no GPU): tests/row_unit_check.cpp runs the library's
own row_unit (kparams.hpp) over planes described by the library's planner and checks that the
units of an item cover its (row group, chunk) pairs exactly once, never address past a row, and,
where narrow interleaved bands are packed into wavefronts of their own, that no full wavefront
mixes band chunks with the rest."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_row_units_cover_every_chunk_once(tmp_path):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    exe = str(tmp_path / "row_unit_check")
    subprocess.run([gxx, "-O2", "-std=c++20", "-Wall", "-Wextra", "-Werror",
                    "-I" + os.path.join(ROOT, "include"), "-I" + os.path.join(ROOT, "paper_2606_01065_amd", "csrc"),
                    os.path.join(ROOT, "tests", "row_unit_check.cpp"),
                    os.path.join(ROOT, "paper_2606_01065_amd", "csrc", "plan.cpp"), "-o", exe], check=True)
    out = subprocess.run([exe], capture_output=True, text=True)
    assert out.returncode == 0, out.stdout + out.stderr
    packs = [int(line.split()[-1]) for line in out.stdout.split("\n") if line.startswith("plane")]
    # DeepSeek-V3 MLA rows (bf16 and fp32) and other narrow interleaved bands are packed;
    # half-split, band-less and odd rows are not
    assert packs[:5] == [8, 4, 8, 8, 32] and packs[5:] == [0, 0, 0, 0]
