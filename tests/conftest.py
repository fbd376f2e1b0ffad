import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
HERE = os.path.dirname(os.path.abspath(__file__))
if HERE not in sys.path:
    sys.path.insert(0, HERE)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built libasv.so")


def pytest_sessionfinish(session, exitstatus):
    """Write every banded decision the parity tests met (rows, nodes, requests, tree shapes,
    histories that followed the GPU), by test and id, to parity_bands.json in the run's output
    folder at the repository root."""
    harness = sys.modules.get("harness")
    if harness is None or not harness.BAND_LOG:
        return
    out = os.path.join(ROOT, "gpurun_out")
    os.makedirs(out, exist_ok=True)
    with open(os.path.join(out, "parity_bands.json"), "w") as f:
        json.dump(harness.BAND_LOG, f, indent=1)
