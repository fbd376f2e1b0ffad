"""Seeded synthetic inputs: determinism, tree validity, bf16 rounding, config shapes."""

import numpy as np
import pytest

from workloads import CONFIGS, bf16_normal, custom_workload, make_workload, round_to_bf16_bits
from workloads.synth import bf16_bits_to_f32


def test_rne_rounding_cases():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -8 + 2 ** -20, -2.5,
                  1.0 - 2 ** -9], dtype=np.float32)
    got = round_to_bf16_bits(x)
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7: even mantissa (1.0) wins; 1 + 3*2^-8 ties
    # between 1 + 2^-7 and 1 + 2^-6: even (1 + 2^-6) wins; just above a tie rounds up.
    want = np.array([0x3F80, 0x3F80, 0x3F82, 0x3F81, 0xC020, 0x3F80], dtype=np.uint16)
    assert np.array_equal(got, want), [hex(v) for v in got]
    assert np.array_equal(bf16_bits_to_f32(want[:2]), np.array([1.0, 1.0], np.float32))


def test_normal_statistics():
    rng = np.random.default_rng(0)
    v = bf16_bits_to_f32(bf16_normal(rng, (200000,), 0.02)).astype(np.float64)
    assert abs(v.mean()) < 3e-4 and abs(v.std() - 0.02) < 3e-4


def _check_tree(w):
    off = w.req_offsets
    assert off[0] == 0 and off[-1] == w.N and np.all(np.diff(off) >= 1)
    for b in range(w.B):
        lo, hi = off[b], off[b + 1]
        assert w.parent[lo] == -1 and w.depth[lo] == 0
        for c in range(lo + 1, hi):
            assert lo <= w.parent[c] < c
            assert w.depth[c] == w.depth[w.parent[c]] + 1
            assert w.kind[c] in (0, 1, 2) and 0 <= w.rank[c] < 8 and 0 <= w.uid[c] < w.V
        assert w.kind[lo] == -1


@pytest.mark.parametrize("cfg", [0, 1, 3])
def test_config_trees(cfg):
    w = make_workload(cfg)
    _check_tree(w)
    c = CONFIGS[cfg]
    assert w.B == c["B"] and w.hidden.shape == (w.N, c["H"])
    if cfg == 0:
        assert w.N == 8 and w.depth.max() <= 4
        assert max(np.bincount(w.parent[1:])) <= 3
    if cfg == 1:
        assert w.N == 60 and w.depth.max() == 6
        assert list(np.bincount(w.depth)) == [1, 10, 10, 10, 10, 10, 9]
    if cfg == 3:
        assert w.N == 2048 and w.depth.max() == 8


def test_adaptive_and_sweep_trees():
    w = make_workload(2, step=5)
    _check_tree(w)
    sizes = np.diff(w.req_offsets)
    assert w.B == 8 and sizes.min() >= 8 and sizes.max() <= 96
    assert w.draft_logits.shape == (w.N, w.V) and w.draft_logits.dtype == np.float32
    w4 = make_workload(4, tau=0.05)
    _check_tree(w4)
    sizes = np.diff(w4.req_offsets)
    assert np.all(sizes[0::2] == 17) and np.all((sizes[1::2] >= 34) & (sizes[1::2] <= 128))
    for b in range(1, w4.B, 2):
        lo = w4.req_offsets[b]
        assert np.sum(w4.parent == lo) == 32 and w4.depth[lo:w4.req_offsets[b + 1]].max() == 2
    assert np.all(w4.tau == np.float32(0.05))


def test_determinism():
    a, b = make_workload(2, step=3), make_workload(2, step=3)
    for f in ("req_offsets", "parent", "hidden", "kind", "rank", "uid", "draft_logits", "tau"):
        assert np.array_equal(getattr(a, f), getattr(b, f)), f
    c = make_workload(2, step=4)
    assert not np.array_equal(a.hidden[:8], c.hidden[:8])


def test_weights_deterministic_small():
    from workloads.synth import bf16_weights
    w1 = bf16_weights(5000, 64, 0.02, 7)
    bf16_weights.cache_clear()
    w2 = bf16_weights(5000, 64, 0.02, 7)
    assert np.array_equal(w1, w2) and w1.dtype == np.uint16 and not w1.flags.writeable


def test_resolve_drafts():
    w = custom_workload("t", 64, 100, [[-1, 0, 0, 1]], 0.3, seed=1)
    top8 = np.arange(w.N * 8, dtype=np.int32).reshape(w.N, 8) % 100
    w.with_drafts(top8)
    for c in range(1, w.N):
        p = w.parent[c]
        want = {0: top8[p, 0], 1: top8[p, w.rank[c]], 2: w.uid[c]}[int(w.kind[c])]
        assert w.draft_tok[c] == want
    assert w.draft_tok[0] == -1
