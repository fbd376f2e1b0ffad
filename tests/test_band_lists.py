"""The stored band lists (tests/golden/band_lists.json, written by make_band_lists.py from the
oracle alone) are current: the walk bands recomputed from the oracle tables and the seeded
trees give the same rows, nodes and requests. The full-size GPU parity tests assert that the
requests they band are exactly these."""

import json
import os
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
GOLDEN = os.path.join(HERE, "golden")
sys.path.insert(0, GOLDEN)

import make_band_lists as mbl  # noqa: E402
from workloads import CONFIGS, make_trees  # noqa: E402


@pytest.fixture(scope="module")
def stored():
    with open(os.path.join(GOLDEN, "band_lists.json")) as f:
        return json.load(f)


@pytest.mark.parametrize("cfg", [1, 3, 4])
def test_band_lists_current(stored, cfg):
    tab = mbl.load_table(cfg)
    off, parent, _ = make_trees(cfg, 0)
    for tau in CONFIGS[cfg]["taus"]:
        got, _ = mbl.walk_bands(tab, 0, off, parent, tau)
        want = stored[f"cfg{cfg}_tau{tau}"]
        for k in ("rows", "nodes", "requests"):
            assert got[k] == want[k], (cfg, tau, k)
        assert len(got["requests"]) <= 0.1 * got["n_requests"]


def test_band_lists_current_cfg2(stored):
    tab = mbl.load_table(2)
    total = 0
    for step in range(int(tab["steps"])):
        off, parent, _ = make_trees(2, step)
        got, _ = mbl.walk_bands(tab, step, off, parent, CONFIGS[2]["taus"][0])
        want = stored[f"cfg2_step{step}"]
        for k in ("rows", "nodes", "requests"):
            assert got[k] == want[k], (step, k)
        total += len(got["requests"])
    assert total <= 0.1 * CONFIGS[2]["B"] * int(tab["steps"])
