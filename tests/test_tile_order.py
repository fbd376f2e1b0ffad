"""K1's tile order on the host: xcd_tile and tile_coords (the device functions themselves,
compiled for the host by hipcc from the library's header) take every tile of a launch exactly
once, for every grid size up to 4096 blocks and for slab-major and blocked orders with ragged
blocks. CPU only: the check runs as a host program."""
import os
import shutil
import subprocess

import pytest

from paper_2609_02897_amd import _build

HERE = os.path.dirname(os.path.abspath(__file__))


def test_tile_order_is_one_to_one(tmp_path):
    hipcc = _build.hipcc()
    if shutil.which(hipcc) is None and not os.path.exists(hipcc):
        pytest.skip("hipcc not found")
    exe = str(tmp_path / "tile_order_check")
    cmd = [hipcc, "--offload-arch=gfx950", "-O1", "-std=c++17",
           "-I", os.path.join(_build.ROOT, "paper_2609_02897_amd", "csrc"),
           "-I", os.path.join(_build.ROOT, "include"),
           os.path.join(HERE, "tile_order_check.cpp"), "-o", exe]
    res = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert res.returncode == 0, res.stderr[-2000:]
    run = subprocess.run([exe], capture_output=True, text=True, timeout=300)
    assert run.returncode == 0 and run.stdout.startswith("ok"), run.stdout + run.stderr
