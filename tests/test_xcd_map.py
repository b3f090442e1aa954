"""The XCD-aware tile map of the level and lazy products, built for the host
with g++ from the same header the kernels include, is a bijection onto the
tile grid for every unit-tile count up to 64 (a regression test for a map
that divided by zero with fewer than 8 unit tiles and sent workgroups out of
bounds)."""
import os
import subprocess
import tempfile

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_xcd_tile_map_is_a_bijection():
    src = os.path.join(ROOT, "tests", "xcd_map_check.cpp")
    inc = os.path.join(ROOT, "paper_1712_04048_amd", "csrc")
    with tempfile.TemporaryDirectory() as d:
        exe = os.path.join(d, "xcd_map_check")
        subprocess.check_call(["g++", "-std=c++17", "-O1", "-I", inc, src, "-o", exe])
        out = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert out.returncode == 0, out.stdout + out.stderr
    assert out.stdout.strip() == "ok"
