"""Host checks of device functions, compiled for the host by hipcc from the library's own
headers (CPU only: each check runs as a host program):

- K1's tile order: xcd_tile and tile_coords take every tile of a launch exactly once, for every
  grid size up to 4096 blocks and for slab-major and blocked orders with ragged blocks;
- the draft head's (logit, id) keys: their unsigned order is the pair order over special and
  random float values and ids, and they decode to the pair;
- the LDS swizzle: under the measured ds_read_b128 pass model every fragment read of every K1
  and K5 tile family puts the 16 lanes of each pass on 16 distinct bank groups (no conflict
  cycles)."""
import os
import shutil
import subprocess

import pytest

from paper_2609_02897_amd import _build

HERE = os.path.dirname(os.path.abspath(__file__))


def _run_host_check(tmp_path, name):
    hipcc = _build.hipcc()
    if shutil.which(hipcc) is None and not os.path.exists(hipcc):
        pytest.skip("hipcc not found")
    exe = str(tmp_path / name)
    cmd = [hipcc, "--offload-arch=gfx950", "-O1", "-std=c++17",
           "-I", os.path.join(_build.ROOT, "paper_2609_02897_amd", "csrc"),
           "-I", os.path.join(_build.ROOT, "include"),
           os.path.join(HERE, name + ".cpp"), "-o", exe]
    res = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert res.returncode == 0, res.stderr[-2000:]
    run = subprocess.run([exe], capture_output=True, text=True, timeout=300)
    assert run.returncode == 0 and run.stdout.startswith("ok"), run.stdout + run.stderr


def test_tile_order_is_one_to_one(tmp_path):
    _run_host_check(tmp_path, "tile_order_check")


def test_draft_keys_order_pairs(tmp_path):
    _run_host_check(tmp_path, "draft_key_check")


def test_lds_swizzle_is_conflict_free(tmp_path):
    _run_host_check(tmp_path, "lds_swizzle_check")
