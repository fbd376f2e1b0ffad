"""Seeded random shapes against the float64 oracle on the GPU.

Each case draws H (a multiple of 64 up to 512), V (ragged vocabulary slabs included), a batch of
random trees, per-request thresholds, an LM-head tile (the library's pick or a forced one), the
weight layout (row-major or packed) and whether draft logits are given, then compares every
output with the oracle's (floats within the tolerance, decisions bit-exact outside the bands).
"""

import os

import numpy as np
import pytest

import oracle
from harness import compare, device_inputs, reference, resolve_with_oracle, to_host
from workloads import custom_workload

pytestmark = pytest.mark.gpu

# ASV_RANDOM_CASES widens the sweep (e.g. to 300); the default keeps the suite short.
N_CASES = int(os.environ.get("ASV_RANDOM_CASES", "24"))


@pytest.fixture(scope="module")
def dev():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


@pytest.fixture(scope="module")
def asv():
    import paper_2609_02897_amd as m
    m.load()
    return m


def _rand_tree(rng, n):
    """A random tree of n nodes in parents-first order (depth and fan-out drawn per tree)."""
    depth_max, branch_max = int(rng.integers(1, 9)), int(rng.integers(1, 6))
    parent, depth, kids = [-1], [0], [0]
    while len(parent) < n:
        open_nodes = [i for i in range(len(parent)) if depth[i] < depth_max and
                      kids[i] < branch_max]
        if not open_nodes:
            break
        p = int(open_nodes[rng.integers(len(open_nodes))])
        parent.append(p)
        depth.append(depth[p] + 1)
        kids.append(0)
        kids[p] += 1
    return parent


def _case(i):
    rng = np.random.default_rng([2609, i])
    H = 64 * int(rng.integers(1, 9))
    V = int(rng.choice([int(rng.integers(16, 300)), int(rng.integers(300, 5000))]))
    B = int(rng.integers(1, 12))
    trees = [_rand_tree(rng, int(rng.integers(1, 70))) for _ in range(B)]
    tau = rng.choice([0.0, 0.05, 0.2, 0.5, 1.0], size=B).astype(np.float32)
    w = custom_workload(f"random{i}", H, V, trees, tau, seed=300 + i,
                        w_std=float(rng.uniform(0.05, 0.2)),
                        draft_logits=bool(rng.integers(0, 2)))
    tile = int(rng.choice([0, 0, 64, 128, 192, 256]))
    packed = bool(rng.integers(0, 2))
    return w, tile, packed


@pytest.mark.parametrize("i", range(N_CASES))
def test_random_shapes(asv, dev, i):
    import torch
    w, tile, packed = _case(i)
    print(f"[random {i}] H={w.H} V={w.V} B={w.B} N={w.N} tile={tile} packed={packed} "
          f"draft_logits={w.draft_logits is not None}", flush=True)
    W = w.weights()
    w64 = oracle.widen_weights(W)
    resolve_with_oracle(w, w64)
    d = device_inputs(w, W, dev)
    w_lm = asv.pack_lm_head(d["w_lm"]) if packed else d["w_lm"]
    out = asv.verify(d["hidden"], w_lm, d["draft_tok"], d["parent"], d["req_offsets"],
                     d["tau"], d["draft_logits"], k1_tile=tile)
    torch.cuda.synchronize()
    rep = compare(w, reference(w, w64), to_host(out))
    print(f"  clean {rep.clean_requests}, banded {rep.banded_requests}", flush=True)
