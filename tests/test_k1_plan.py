"""Host logic of the LM-head launch plan (asv_k1_plan): which tile family covers which slabs,
and each launch's K loop, weight copy policy and tile order. CPU only: no GPU call."""
import math

import numpy as np
import pytest

import paper_2609_02897_amd as asv
from paper_2609_02897_amd import _build

COST = {128: 62, 192: 80, 256: 98}      # per-round costs of the tile families (tile pick)


@pytest.fixture(scope="module", autouse=True)
def built():
    if not _build.is_built(_build.OUT):
        _build.build_library()


def _launch(tile_rows, slab0, n_slabs, row_tiles, k_loop, stream_w, blk_slabs=0, blk_rows=0):
    return dict(tile_rows=tile_rows, slab0=slab0, n_slabs=n_slabs, row_tiles=row_tiles,
                k_loop=k_loop, stream_w=stream_w, blk_slabs=blk_slabs, blk_rows=blk_rows)


@pytest.mark.parametrize("N,V,expected", [
    # the headline: 60 rows of Llama's vocabulary, 501 slabs, two 64-row tiles per CU
    (60, 128256, [_launch(64, 0, 501, 1, 0, 1)]),
    # Qwen's vocabulary: 594 slabs fit three per CU but not two: the one-slot ring
    (60, 151936, [_launch(64, 0, 594, 1, 1, 1)]),
    # 782 slabs fit neither: back to the two-slot burst ring
    (60, 200000, [_launch(64, 0, 782, 1, 0, 1)]),
    # 378 rows: 128-row tiles fill one round on 85 slabs (three row tiles: default policy),
    # 192-row tiles take the other 509 (two row tiles: non-temporal W)
    (378, 151936, [_launch(128, 0, 85, 3, 3, 0), _launch(192, 85, 509, 2, 2, 1)]),
    # 2048 rows: 23 slabs of 192-row tiles (11 row tiles: blocked order), then 256-row tiles
    (2048, 128256, [_launch(192, 0, 23, 11, 2, 0, 8, 4), _launch(256, 23, 478, 8, 2, 0)]),
    # 3048 rows: 256-row tiles only, twelve row tiles, blocks of 8 slabs x 4 row tiles
    (3048, 151936, [_launch(256, 0, 594, 12, 2, 0, 8, 4)]),
])
def test_documented_plans(N, V, expected):
    assert asv.k1_plan(N, V, 256) == expected


def _rounds(tiles, cus):
    return (tiles + cus - 1) // cus


def _estimate(launches, cus):
    return sum(_rounds(k["n_slabs"] * k["row_tiles"], cus) * COST[k["tile_rows"]]
               for k in launches)


def test_plan_invariants():
    """Over random shapes: the launches cover the slabs once, in order; every launch follows
    the stated rules; above 64 rows the plan's estimate is no worse than any single family's."""
    rng = np.random.default_rng(2609)
    for _ in range(3000):
        N = int(rng.choice([rng.integers(1, 65), rng.integers(65, 600), rng.integers(600, 6000)]))
        V = int(rng.integers(1, 300000))
        cus = int(rng.choice([8, 32, 80, 104, 256, 304]))
        forced = int(rng.choice([0, 0, 0, 64, 128, 192, 256]))
        got = asv.k1_plan(N, V, cus, forced)
        S = (V + 255) // 256
        c = max(1, cus // 8)
        assert 1 <= len(got) <= 2
        assert got[0]["slab0"] == 0 and sum(k["n_slabs"] for k in got) == S
        if len(got) == 2:
            assert got[1]["slab0"] == got[0]["n_slabs"] and got[0]["tile_rows"] != got[1]["tile_rows"]
        if forced:
            assert len(got) == 1 and got[0]["tile_rows"] == forced
        elif N <= 64:
            assert len(got) == 1 and got[0]["tile_rows"] == 64
        else:
            assert all(k["tile_rows"] in (128, 192, 256) for k in got)
            single = min(_rounds(S * math.ceil(N / r), cus) * COST[r] for r in COST)
            assert _estimate(got, cus) <= single, (N, V, cus, got)
        for k in got:
            rt = math.ceil(N / k["tile_rows"])
            assert k["row_tiles"] == rt
            tiles = k["n_slabs"] * rt
            if k["tile_rows"] == 64:
                assert k["k_loop"] == (1 if 2 * cus < tiles <= 3 * cus else 0)
            else:
                assert k["k_loop"] == (3 if k["tile_rows"] == 128 else 2)
            assert k["stream_w"] == (1 if rt <= 2 else 0)
            blocked = rt > 4 and c / rt + rt > c / 4 + 4
            assert (k["blk_slabs"], k["blk_rows"]) == ((max(1, c // 4), 4) if blocked else (0, 0))


def test_plan_of_the_largest_sizes_is_quick():
    """The two-family search is bounded: one CU and the largest accepted grid plan at once."""
    import time
    asv.k1_plan(100, 1000, 256)               # loads the library (runtime start-up) untimed
    t0 = time.perf_counter()
    got = asv.k1_plan((1 << 15) - 64, (1 << 30) - 1, 1)   # 2^22 slabs x 511 64-row tiles
    assert time.perf_counter() - t0 < 0.5
    assert sum(k["n_slabs"] for k in got) == ((1 << 30) - 1 + 255) // 256


@pytest.mark.parametrize("args", [(0, 1000, 256, 0), (10, 0, 256, 0), (10, 1000, 0, 0),
                                  (10, 1000, 256, 100)])
def test_plan_rejects(args):
    with pytest.raises(asv.AsvError):
        asv.k1_plan(*args)
