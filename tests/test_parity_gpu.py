"""GPU parity of the HIP path (through the C ABI) with the float64 CPU oracle.

Small and ragged shapes (several vocabulary slabs with a ragged last slab, one to three tree-row
tiles with a ragged last tile, every K1 tile family) and the degenerate cases the method has.
The oracle runs live on these sizes. Full-size configurations are in test_parity_full_gpu.py.
"""

import zlib

import numpy as np
import pytest

import oracle
from harness import TOL_F, SHAPE_BAND, compare, compare_state, device_inputs, follow_gpu_history, \
    reference, resolve_with_oracle, to_host
from workloads import build_tree, custom_workload, make_workload

pytestmark = pytest.mark.gpu


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


def _run(asv, w, W, dev, tau=None, state=None, params=None, out=None, k1_tile=0, packed=False):
    import torch
    d = device_inputs(w, W, dev, tau)
    w_lm = asv.pack_lm_head(d["w_lm"]) if packed else d["w_lm"]
    o = asv.verify(d["hidden"], w_lm, d["draft_tok"], d["parent"], d["req_offsets"],
                   d["tau"], d["draft_logits"], state=state, params=params, out=out,
                   k1_tile=k1_tile)
    torch.cuda.synchronize()
    return to_host(o)


def _trees(kind, n_req, seed):
    rng = np.random.default_rng(seed)
    return [build_tree(kind, rng, b) for b in range(n_req)]


def _rand_tree(rng, n, depth_max, branch_max):
    parent, depth, kids = [-1], [0], [0]
    while len(parent) < n:
        open_nodes = [i for i in range(len(parent)) if depth[i] < depth_max and
                      kids[i] < branch_max]
        p = int(open_nodes[rng.integers(len(open_nodes))])
        parent.append(p)
        depth.append(depth[p] + 1)
        kids.append(0)
        kids[p] += 1
    return parent


def _case(name):
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    if name == "tiny_config":
        return make_workload(0)
    if name == "rows64_eagle60_ragged_vocab":
        # one 60-node EAGLE-style tree, 17 slabs with a ragged last slab of 77 entries
        return custom_workload(name, 256, 16 * 256 + 77, _trees("eagle60", 1, 1), 0.3,
                               seed=1, w_std=0.08)
    if name == "rows128_mixed":
        trees = [_rand_tree(rng, int(rng.integers(1, 40)), 6, 4) for _ in range(5)]
        return custom_workload(name, 128, 3000, trees, 0.2, seed=2, w_std=0.11,
                               draft_logits=True)
    if name == "rows256_three_tiles":
        trees = _trees("adaptive", 9, 3)
        return custom_workload(name, 192, 2500, trees, 0.2, seed=3, w_std=0.09,
                               draft_logits=True)
    if name == "deep_chain_and_wide":
        trees = [[-1] + list(range(40)), [-1] + [0] * 100, [-1]]
        return custom_workload(name, 64, 1024, trees, 0.05, seed=4, w_std=0.16)
    if name == "root_only_requests":
        trees = [[-1], [-1, 0, 1, 1], [-1], [-1, 0]]
        return custom_workload(name, 64, 700, trees, 0.3, seed=5, w_std=0.16)
    if name == "many_tiny_requests":
        # 300 requests of 1 to 5 nodes: one merge workgroup completes several requests and
        # requests straddle workgroups (fused finishing kernel)
        trees = [_rand_tree(rng, int(rng.integers(1, 6)), 3, 3) for _ in range(300)]
        return custom_workload(name, 64, 900, trees, 0.3, seed=6, w_std=0.16)
    if name == "unfused_large_batch":
        # more requests than the fused finishing kernel takes: separate merge and walk kernels
        trees = [_rand_tree(rng, int(rng.integers(1, 4)), 2, 2) for _ in range(1100)]
        return custom_workload(name, 64, 600, trees, 0.3, seed=7, w_std=0.16,
                               draft_logits=True)
    if name == "request_over_lds_stage":
        # a 300-node request (walked from global memory) beside small ones, fused path
        trees = [_rand_tree(rng, 300, 12, 4), [-1, 0, 0], _rand_tree(rng, 40, 6, 3)]
        return custom_workload(name, 64, 800, trees, 0.3, seed=8, w_std=0.16,
                               draft_logits=True)
    if name == "unfused_with_large_request":
        # unfused path with one request above the LDS staging limit
        trees = [_rand_tree(rng, int(rng.integers(1, 4)), 2, 2) for _ in range(1030)]
        trees[517] = _rand_tree(rng, 290, 10, 4)
        return custom_workload(name, 64, 600, trees, 0.3, seed=9, w_std=0.16)
    if name == "single_row_single_slab":
        # N = 1 (a root-only request) and V < 256: one ragged vocabulary slab
        return custom_workload(name, 64, 100, [[-1]], 0.3, seed=10, w_std=0.16)
    if name == "vocab_over_one_merge_round":
        # V = 170000: 665 slabs, more than one round of record loads in the row merge
        trees = [_rand_tree(rng, 20, 5, 3), _rand_tree(rng, 11, 4, 3)]
        return custom_workload(name, 64, 170000, trees, 0.2, seed=11, w_std=0.16,
                               draft_logits=True)
    if name == "rows128_five_stages":
        # 128-row tiles (three-slot spread loop) over H = 320, five K stages: both ring wraps
        # and the tail copies past the last stage; two row tiles, the second ragged
        trees = [_rand_tree(rng, int(rng.integers(20, 60)), 7, 4) for _ in range(5)]
        return custom_workload(name, 320, 2000, trees, 0.2, seed=12, w_std=0.07)
    if name == "rows256_five_stages":
        # 256-row tiles (two-slot spread loop) over H = 320, five K stages; ragged last row tile
        # and ragged last slab
        trees = [_rand_tree(rng, int(rng.integers(40, 120)), 8, 4) for _ in range(9)]
        return custom_workload(name, 320, 1500, trees, 0.2, seed=13, w_std=0.07,
                               draft_logits=True)
    if name == "rows192_two_tiles":
        # 192-row tiles (two-slot spread loop) over H = 320: two row tiles, the second ragged
        trees = [_rand_tree(rng, int(rng.integers(30, 80)), 8, 4) for _ in range(6)]
        return custom_workload(name, 320, 1800, trees, 0.2, seed=14, w_std=0.07,
                               draft_logits=True)
    if name == "rows192_one_tile":
        # one ragged 192-row tile over H = 192 (three K stages)
        trees = [_rand_tree(rng, int(rng.integers(36, 48)), 6, 4) for _ in range(4)]
        return custom_workload(name, 192, 1300, trees, 0.3, seed=15, w_std=0.09)
    if name == "blocked_tile_order":
        # about 2600 rows: 11 row tiles of 256 (more than 8, so on 256 CUs the tiles run in
        # blocks of 8 slabs x 4 row tiles: row groups of 4, 4 and 3) over 11 slabs, the last
        # block of 3 slabs and a ragged last slab of 77 entries
        trees, n = [], 0
        while n < 2600:
            t = _rand_tree(rng, min(int(rng.integers(16, 120)), 2600 - n), 9, 4)
            trees.append(t)
            n += len(t)
        return custom_workload(name, 128, 10 * 256 + 77, trees, 0.2, seed=16, w_std=0.11,
                               draft_logits=True)
    raise KeyError(name)


# Cases that pin the LM-head tile, so that every tile family and both spread loops run with
# ragged row tiles and slabs and with one, two, three and five K stages (the other cases take the
# library's pick, which at these small vocabularies is the 128-row tile).
CASE_TILE = {"rows128_mixed": 128, "rows128_five_stages": 128, "rows192_one_tile": 192,
             "rows192_two_tiles": 192, "request_over_lds_stage": 192,
             "rows256_three_tiles": 256, "rows256_five_stages": 256, "many_tiny_requests": 256,
             "unfused_large_batch": 256}

CASES = ["tiny_config", "rows64_eagle60_ragged_vocab", "rows128_mixed", "rows256_three_tiles",
         "rows128_five_stages", "rows256_five_stages", "rows192_two_tiles", "rows192_one_tile",
         "deep_chain_and_wide", "root_only_requests", "many_tiny_requests",
         "unfused_large_batch", "request_over_lds_stage", "unfused_with_large_request",
         "single_row_single_slab", "vocab_over_one_merge_round"]


@pytest.mark.parametrize("tau", [None, 0.0, 0.05, 0.3, 1.0])
@pytest.mark.parametrize("name", CASES)
def test_parity_small(asv, dev, name, tau):
    print(f"[parity] case={name} tau={tau}", flush=True)
    w = _case(name)
    W = w.weights()
    w64 = oracle.widen_weights(W)
    resolve_with_oracle(w, w64)
    taus = None if tau is None else np.full(w.B, tau, dtype=np.float32)
    ref = reference(w, w64, tau=taus)
    got = _run(asv, w, W, dev, tau=taus, k1_tile=CASE_TILE.get(name, 0))
    rep = compare(w, ref, got, tag=f"{name} tau={tau}")
    print(f"  {rep}", flush=True)
    if tau == 0.0:
        assert np.all(got["accept"] == 1)
    if tau == 1.0:
        # strict verification: every accepted node is the argmax of its parent row
        for c in got["accepted_path"][got["accepted_path"] >= 0]:
            p = w.parent[c]
            assert w.draft_tok[c] == got["row_argmax"][p] or ref["row_gap"][p] < 1e-3


def test_determinism(asv, dev):
    w = _case("rows256_three_tiles")
    W = w.weights()
    resolve_with_oracle(w, oracle.widen_weights(W))
    a = _run(asv, w, W, dev, k1_tile=256)
    b = _run(asv, w, W, dev, k1_tile=256)
    for k in a:
        if a[k] is not None:
            assert np.array_equal(a[k], b[k], equal_nan=True), k


def test_every_tile_same_results(asv, dev):
    """Every K1 tile accumulates K in the same order, so the logits and every decision taken
    from them are the same bit for bit on all four tiles; row_lse may differ in the last bits
    (the slab records of a row are merged across a different number of waves)."""
    w = _case("rows192_two_tiles")
    W = w.weights()
    resolve_with_oracle(w, oracle.widen_weights(W))
    runs = {rows: _run(asv, w, W, dev, k1_tile=rows) for rows in (64, 128, 192, 256)}
    base = runs[64]
    nonroot = w.parent >= 0
    for rows, got in runs.items():
        for k in ("row_max", "row_argmax", "accept", "accepted_len", "accepted_path",
                  "bonus_token", "draft_conf"):
            assert np.array_equal(got[k], base[k], equal_nan=True), (rows, k)
        assert np.array_equal(got["drafted_logit"][nonroot], base["drafted_logit"][nonroot]), rows
        assert np.allclose(got["row_lse"], base["row_lse"], rtol=1e-6, atol=1e-6), rows


def test_blocked_tile_order(asv, dev):
    """Launches of many row tiles take their tiles in blocks of slabs x row tiles (ragged row
    groups and a ragged last block here, on every tile family: 11 to 41 row tiles). Every
    (slab, row tile) pair must run once: the records match the oracle's, and all four tile
    families agree bit for bit as in test_every_tile_same_results."""
    print("[blocked order] case=blocked_tile_order", flush=True)
    w = _case("blocked_tile_order")
    for rows in (256, 192, 128, 64):     # on a 256-CU GPU every family takes the blocked order
        assert asv.k1_plan(w.N, w.V, 256, rows)[0]["blk_rows"] == 4, rows
    W = w.weights()
    w64 = oracle.widen_weights(W)
    resolve_with_oracle(w, w64)
    ref = reference(w, w64)
    runs = {}
    for rows in (256, 192, 128, 64):
        runs[rows] = _run(asv, w, W, dev, k1_tile=rows, packed=rows == 256)
        compare(w, ref, runs[rows], tag=f"blocked order tile={rows}")
    base = runs[64]
    nonroot = w.parent >= 0
    for rows, got in runs.items():
        for k in ("row_max", "row_argmax", "accept", "accepted_len", "accepted_path",
                  "bonus_token", "draft_conf"):
            assert np.array_equal(got[k], base[k], equal_nan=True), (rows, k)
        assert np.array_equal(got["drafted_logit"][nonroot], base["drafted_logit"][nonroot]), rows
        assert np.allclose(got["row_lse"], base["row_lse"], rtol=1e-6, atol=1e-6), rows


@pytest.mark.parametrize("V,sizes,tile", [(140000, (30, 21, 4), 0),
                                          (80000, (40, 33, 27), 64)])
def test_one_slot_weight_stream(asv, dev, V, sizes, tile):
    """When a launch's 64-row tiles fit three per CU but not two (on a 256-CU GPU: 513-768
    tiles) the 64-row tile runs its one-slot ring: V = 140000 (547 slabs, one row tile) with
    the library's pick, and V = 80000 (313 slabs, two row tiles at 100 rows) with the 64-row
    tile forced. The records, drafted logits and walks match the oracle, and the other tile
    families bit for bit."""
    assert asv.k1_plan(sum(sizes), V, 256, tile)[0]["k_loop"] == 1
    print(f"[one-slot ring] V={V} N={sum(sizes)} tile={tile}", flush=True)
    rng = np.random.default_rng(V)
    trees = [_rand_tree(rng, n, 6, 4) for n in sizes]
    w = custom_workload(f"one_slot{V}", 256, V, trees, 0.2, seed=18, w_std=0.1,
                        draft_logits=True)
    W = w.weights()
    w64 = oracle.widen_weights(W)
    resolve_with_oracle(w, w64)
    ref = reference(w, w64)
    runs = {}
    for rows, packed in ((tile, True), (tile, False), (128, True), (256, True)):
        runs[(rows, packed)] = _run(asv, w, W, dev, k1_tile=rows, packed=packed)
        compare(w, ref, runs[(rows, packed)], tag=f"one-slot tile={rows} packed={packed}")
    base = runs[(tile, True)]
    nonroot = w.parent >= 0
    for key, got in runs.items():
        for k in ("row_max", "row_argmax", "accept", "accepted_len", "accepted_path",
                  "bonus_token", "draft_conf"):
            assert np.array_equal(got[k], base[k], equal_nan=True), (key, k)
        assert np.array_equal(got["drafted_logit"][nonroot], base["drafted_logit"][nonroot]), key
        assert np.allclose(got["row_lse"], base["row_lse"], rtol=1e-6, atol=1e-6), key


def test_long_hidden_16384(asv, dev):
    """H = 16384 (256 K stages, the hidden size of the largest Llama-3.1 model): every K loop
    (the burst ring of the 64-row tile, the three-slot loop of the 128-row tile and the two-slot
    loop of the 256-row tile) wraps its ring 128 times or more, on both weight layouts; the
    records, drafted logits and walks match the oracle."""
    print("[long hidden] H=16384", flush=True)
    rng = np.random.default_rng(16384)
    trees, n = [], 0
    while n < 300:
        t = _rand_tree(rng, min(int(rng.integers(10, 70)), 300 - n), 8, 4)
        trees.append(t)
        n += len(t)
    w = custom_workload("long_hidden", 16384, 6000 + 77, trees, 0.2, seed=17, w_std=0.02,
                        draft_logits=True)
    W = w.weights()
    w64 = oracle.widen_weights(W)
    resolve_with_oracle(w, w64)
    ref = reference(w, w64)
    for rows, packed in ((64, False), (128, True), (256, False), (256, True)):
        got = _run(asv, w, W, dev, k1_tile=rows, packed=packed)
        compare(w, ref, got, tag=f"long hidden tile={rows} packed={packed}")


@pytest.mark.parametrize("N", [150, 200, 378])
def test_two_family_plan(asv, dev, N):
    """At V = 151936 and these row counts the library splits the vocabulary slabs between two
    LM-head tile families in two launches (on 256 CUs: 128-row tiles on the first slabs, 192-
    or 256-row tiles on the rest), so that no round of workgroups runs a third empty. Every
    output equals the single-family runs' bit for bit (the same K order everywhere, and both
    families merge a slab's record across two waves), and the oracle's."""
    print(f"[two families] N={N}", flush=True)
    rng = np.random.default_rng(N)
    trees, n = [], 0
    while n < N:
        t = _rand_tree(rng, min(int(rng.integers(8, 97)), N - n), 8, 4)
        trees.append(t)
        n += len(t)
    w = custom_workload(f"plan{N}", 64, 151936, trees, 0.2, seed=20 + N, w_std=0.16)
    W = w.weights()
    w64 = oracle.widen_weights(W)
    resolve_with_oracle(w, w64)
    got = _run(asv, w, W, dev, packed=True)
    compare(w, reference(w, w64), got, tag=f"two families N={N}")
    nonroot = w.parent >= 0
    for rows in (128, 192, 256):
        base = _run(asv, w, W, dev, k1_tile=rows, packed=True)
        for k, v in base.items():
            if v is not None:
                sel = nonroot if k == "drafted_logit" else slice(None)
                assert np.array_equal(got[k][sel], v[sel], equal_nan=True), (rows, k)


@pytest.mark.parametrize("V,H", [(1, 64), (256, 64), (1000, 192), (2 * 256 + 77, 320),
                                 (151936, 4096)])
def test_pack_layout(asv, dev, V, H):
    """asv_pack_lm_head writes packed[((k S + s) 256 + r) 64 + c] = w[256 s + r][64 k + c],
    zero past V: checked against torch's reshape and permute of the zero-padded weight."""
    import torch
    print(f"[pack] V={V} H={H}", flush=True)
    g = torch.Generator(device=dev)
    g.manual_seed(V * 7919 + H)
    bits = torch.randint(-32768, 32768, (V, H), dtype=torch.int32, device=dev,
                         generator=g).to(torch.int16)
    w = bits.view(torch.bfloat16)
    p = asv.pack_lm_head(w)
    torch.cuda.synchronize()
    S, KT = -(-V // 256), H // 64
    assert (p.V, p.H) == (V, H) and p.data.numel() == S * 256 * H
    pad = torch.zeros((S * 256, H), dtype=torch.int16, device=dev)
    pad[:V] = bits
    ref = pad.view(S, 256, KT, 64).permute(2, 0, 1, 3).contiguous().view(-1)
    assert torch.equal(p.data.view(torch.int16), ref)


@pytest.mark.parametrize("name", ["rows64_eagle60_ragged_vocab", "rows128_five_stages",
                                  "rows192_one_tile", "rows256_five_stages",
                                  "single_row_single_slab", "vocab_over_one_merge_round"])
def test_packed_weight_same_results(asv, dev, name):
    """The packed weight feeds the MFMAs the same values in the same K order, so every output
    is bit for bit the row-major weight's; the packed run also meets the oracle."""
    w = _case(name)
    W = w.weights()
    w64 = oracle.widen_weights(W)
    resolve_with_oracle(w, w64)
    tile = CASE_TILE.get(name, 0)
    got = _run(asv, w, W, dev, k1_tile=tile, packed=True)
    compare(w, reference(w, w64), got)
    base = _run(asv, w, W, dev, k1_tile=tile)
    nonroot = w.parent >= 0                 # drafted_logit is unspecified at roots
    for k, v in base.items():
        if v is not None:
            sel = nonroot if k == "drafted_logit" else slice(None)
            assert np.array_equal(got[k][sel], v[sel], equal_nan=True), k


def test_packed_weight_every_tile(asv, dev):
    """Packed and row-major weights agree bit for bit on each of the four tile families."""
    w = _case("rows192_two_tiles")
    W = w.weights()
    resolve_with_oracle(w, oracle.widen_weights(W))
    for rows in (64, 128, 192, 256):
        got = _run(asv, w, W, dev, k1_tile=rows, packed=True)
        base = _run(asv, w, W, dev, k1_tile=rows)
        for k, v in base.items():
            if v is not None:
                sel = w.parent >= 0 if k == "drafted_logit" else slice(None)
                assert np.array_equal(got[k][sel], v[sel], equal_nan=True), (rows, k)


def test_packed_weight_past_2gib(asv, dev):
    """A 3.9 GiB packed weight (V = 128256, H = 16384: K-block offsets past 2^31, held in
    32-bit unsigned arithmetic) against the row-major weight, bit for bit, on the 64- and
    128-row tiles; the draft layout likewise at 2.1 GiB."""
    import torch
    V, H, N = 128256, 16384, 100
    g = torch.Generator(device=dev)
    g.manual_seed(7)
    w = (torch.randn((V, H), device=dev, generator=g) * 0.01).to(torch.bfloat16)
    hidden = torch.randn((N, H), device=dev, generator=g).to(torch.bfloat16)
    parent = torch.tensor([-1] + list(range(N - 1)), dtype=torch.int32, device=dev)
    tok = torch.randint(0, V, (N,), dtype=torch.int32, device=dev, generator=g)
    off = torch.tensor([0, N], dtype=torch.int32, device=dev)
    tau = torch.full((1,), 0.3, dtype=torch.float32, device=dev)
    p = asv.pack_lm_head(w)
    assert p.data.numel() * 2 >= 3.9 * 2**30
    for tile in (64, 128):
        n = 60 if tile == 64 else N
        args = (hidden[:n], None, tok[:n], parent[:n], torch.tensor([0, n], dtype=torch.int32,
                                                                     device=dev), tau)
        got = asv.verify(args[0], p, *args[2:], k1_tile=tile)
        ref = asv.verify(args[0], w, *args[2:], k1_tile=tile)
        torch.cuda.synchronize()
        assert torch.isfinite(ref.row_max).all()
        for f in ("row_max", "row_lse", "row_argmax", "accept", "accepted_len",
                  "accepted_path", "bonus_token"):
            assert torch.equal(getattr(got, f), getattr(ref, f)), (tile, f)
        assert torch.equal(got.drafted_logit[1:], ref.drafted_logit[1:]), tile
    del p
    # the draft layout at V = 64000, H = 16384 (2.1 GiB packed)
    wd = w[:64000]
    pd = asv.pack_draft_head(wd)
    x = hidden[:8]
    for weight_pair in ((wd, pd),):
        outs = []
        for weight in weight_pair:
            trees = asv.alloc_draft_trees(2, dev)
            outs.append(asv.draft_step(x, weight, trees, 0, shape=(3, 4, 4)))
        torch.cuda.synchronize()
        for f in outs[0]._fields:
            if getattr(outs[0], f) is not None:
                assert torch.equal(getattr(outs[0], f), getattr(outs[1], f)), f


@pytest.mark.parametrize("name", ["deep_chain_and_wide", "request_over_lds_stage"])
@pytest.mark.parametrize("max_promotions", [0, 1, 2])
def test_promotion_cap(asv, dev, max_promotions, name):
    w = _case(name)
    W = w.weights()
    w64 = oracle.widen_weights(W)
    resolve_with_oracle(w, w64)
    p = oracle.Params(max_promotions=max_promotions)
    ref = reference(w, w64, params=p)
    got = _run(asv, w, W, dev, params=asv.make_params(max_promotions=max_promotions))
    compare(w, ref, got)


@pytest.mark.parametrize("temperature", [0.5, 2.0])
@pytest.mark.parametrize("name", ["rows64_eagle60_ragged_vocab", "rows256_three_tiles"])
def test_margin_temperature(asv, dev, name, temperature):
    """The temperature variant of the margin rule: exp((z_d - z_max) / T) >= kappa."""
    print(f"[temperature] case={name} T={temperature}", flush=True)
    w = _case(name)
    W = w.weights()
    w64 = oracle.widen_weights(W)
    resolve_with_oracle(w, w64)
    ref = reference(w, w64, params=oracle.Params(temperature=temperature))
    got = _run(asv, w, W, dev, params=asv.make_params(temperature=temperature))
    rep = compare(w, ref, got)
    print(f"  {rep}", flush=True)
    base = reference(w, w64)
    if temperature > 1:
        assert ref["accept"].sum() >= base["accept"].sum()
    else:
        assert ref["accept"].sum() <= base["accept"].sum()


def test_exact_ties_lowest_index(asv, dev):
    """Bit-identical W rows give bit-identical logits in both implementations; the argmax, the
    bonus and the sibling choice must take the lowest index, across lanes, waves and slabs."""
    w = custom_workload("ties", 128, 2000, [[-1, 0, 0, 1, 1, 2]], 1.0, seed=9, w_std=0.11)
    W = np.array(w.weights())
    w64 = oracle.widen_weights(W)
    z = oracle.logits(oracle.widen_bf16(w.hidden), w64)
    a0 = int(np.argmax(z[0]))
    a1 = int(np.argmax(z[1]))
    # row 0's winner duplicated into a later slab and an earlier slab (the earlier one wins)
    W[min(a0 + 700, 1999)] = W[a0]
    lo_id = 3 if a0 != 3 else 5
    W[lo_id] = W[a0]
    # row 1's winner duplicated at the next index (same slab, neighbouring lanes)
    nxt = a1 + 1 if a1 + 1 < 2000 and a1 + 1 not in (a0, lo_id) else a1 - 1
    W[nxt] = W[a1]
    w64 = oracle.widen_weights(W)
    z = oracle.logits(oracle.widen_bf16(w.hidden), w64)
    top8 = oracle.row_top8(z)
    w.with_drafts(top8)
    # siblings 1 and 2 draft the two tied tokens of row 0: equal logits, lowest node id wins
    w.draft_tok[1] = lo_id
    w.draft_tok[2] = a0
    ref = reference(w, w64)
    got = _run(asv, w, W, dev)
    for r in (0, 1):
        ties = np.flatnonzero(z[r] == z[r].max())
        assert len(ties) >= 2
        assert got["row_argmax"][r] == ref["row_argmax"][r] == ties.min()
    assert got["drafted_logit"][1] == got["drafted_logit"][2]
    assert list(got["accepted_path"]) == list(ref["accepted_path"])
    assert got["bonus_token"][0] == ref["bonus_token"][0]


def test_exact_ties_lane_groups(asv, dev):
    """Exact ties laid across the accumulator layout of the 16x16 MFMA blocks: ids 558 (block
    34, lane group 3), 566 and 570 (block 35, groups 1 and 2), 582 (block 36), 694 (the other
    128-id half of slab 2, another wave) and 822 (slab 3) carry the same doubled weight row, so
    their logits are equal and the largest of row 0. Every LM-head tile family must report the
    lowest id, 558, as the oracle does, on the row-major and on the packed weight; the lowest id
    sits in the highest lane group of its block, so the lane-group merges decide it."""
    print("[ties across lane groups]", flush=True)
    w = custom_workload("ties16", 128, 2000, [[-1, 0, 0]], 1.0, seed=19, w_std=0.11)
    W = np.array(w.weights())
    x64 = oracle.widen_bf16(w.hidden)
    z = oracle.logits(x64, oracle.widen_weights(W))
    a0 = int(np.argmax(z[0]))
    assert z[0, a0] > 0
    doubled = (W[a0].astype(np.uint32) << 16).view(np.float32) * 2     # exact in bf16
    doubled = (doubled.view(np.uint32) >> 16).astype(np.uint16)
    ties = [558, 566, 570, 582, 694, 822]
    for v in ties:
        W[v] = doubled
    w64 = oracle.widen_weights(W)
    z = oracle.logits(x64, w64)
    assert list(np.flatnonzero(z[0] == z[0].max())) == ties
    w.with_drafts(oracle.row_top8(z))
    ref = reference(w, w64)
    assert ref["row_argmax"][0] == 558
    row_max = set()
    for packed in (False, True):
        for rows in (64, 128, 192, 256):
            got = _run(asv, w, W, dev, k1_tile=rows, packed=packed)
            assert got["row_argmax"][0] == 558, (rows, packed, int(got["row_argmax"][0]))
            row_max.add(float(got["row_max"][0]))
    assert len(row_max) == 1
    assert abs(row_max.pop() - ref["row_max"][0]) < TOL_F


@pytest.mark.parametrize("n_req", [3, 1030])
def test_history_state_over_steps(asv, dev, n_req):
    """20 steps through the policy state: EMA, ring wrap at 16, breaker (forced with kappa=1
    and non-argmax drafts on a stretch of steps). 1030 requests take the unfused path."""
    print(f"[history] n_req={n_req}", flush=True)
    H, V = 64, 900
    p = oracle.Params()
    st_ref = [oracle.state_init(p) for _ in range(n_req)]
    st_gpu = asv.state_init(n_req, asv.make_params(), device=dev)
    hi_size = 12 if n_req < 100 else 4
    for step in range(20):
        rng = np.random.default_rng(100 + step)
        trees = [_rand_tree(rng, int(rng.integers(2, hi_size)), 4, 3) for _ in range(n_req)]
        w = custom_workload(f"hist{step}", H, V, trees, 0.3, seed=200 + step, w_std=0.2,
                            draft_logits=True)
        W = w.weights()
        w64 = oracle.widen_weights(W)
        resolve_with_oracle(w, w64)
        if step < 6:
            w.tau[:] = 0.0      # accept everything: every streak is 0 before the stretch
        if 6 <= step < 13:
            # zero-accept steps: strict rule and drafts that are never the argmax
            z = oracle.logits(oracle.widen_bf16(w.hidden), w64)
            for c in range(w.N):
                if w.parent[c] >= 0:
                    w.draft_tok[c] = int(np.argsort(-z[w.parent[c]])[3])
            w.tau[:] = 1.0
        ref = reference(w, w64, state=st_ref, params=p)
        got = _run(asv, w, W, dev, state=st_gpu)
        tag = f"history n_req={n_req} step={step}"
        compare(w, ref, got, tag=tag)
        # A request whose walk passed a decision inside the float64 tolerance bands may
        # legitimately accept a different length; its expected state is the oracle's update
        # applied to the length the GPU accepted (listed, at most a tenth of the batch).
        st_ref = follow_gpu_history(tag, ref, got, st_ref, w, p, conf=ref["draft_conf"])
        compare_state(asv.state_fields(st_gpu), st_ref, params=p, tag=tag)
        if step == 10:   # fifth consecutive zero-accept step
            assert all(s.breaker == 1 for s in st_ref)
        if 6 <= step < 10:
            assert all(s.breaker == 0 and s.zero_streak == step - 5 for s in st_ref)


def test_tree_policy_entry_point(asv, dev):
    """asv_tree_policy against the float64 oracle (Sec. 3.3, Eq. (2)): fresh confidences
    including exact half-way points of the shape ranges (exact in both precisions, compared
    without bands), the stored confidence when none is given, a non-default divisor and range,
    and breaker-flagged requests. Elsewhere a shape within 1e-4 of a half-integer is banded."""
    import ctypes
    import torch
    B = 600
    rng = np.random.default_rng(31)
    conf = rng.uniform(0.0, 1.0, B).astype(np.float32)
    conf[:17] = np.arange(17, dtype=np.float32) / 32.0          # DCS = k/16 at RAR 1, d 0.5
    for params in (oracle.Params(),
                   oracle.Params(dcs_divisor=0.3, shape_lo=(2, 5, 3), shape_hi=(9, 1, 12),
                                 shape_start=(4, 2, 6))):
        cp = asv.make_params(dcs_divisor=params.dcs_divisor, shape_lo=params.shape_lo,
                             shape_hi=params.shape_hi, shape_start=params.shape_start)
        st = asv.state_init(B, cp, device=dev)
        raw = st.cpu().numpy().copy()
        # set RAR and the breaker flag on the host: rar is word 0, breaker word 20
        words = raw.view(np.int32).reshape(B, -1)
        fl = raw.view(np.float32).reshape(B, -1)
        rar = rng.uniform(0.0, 1.0, B).astype(np.float32)
        rar[:17] = 1.0
        fl[:, 0] = rar
        brk = (rng.random(B) < 0.1).astype(np.int32)
        brk[:17] = 0
        words[:, 20] = brk
        st.copy_(torch.from_numpy(raw).to(dev))
        asv.tree_policy(st, torch.from_numpy(conf).to(dev), cp)
        torch.cuda.synchronize()
        got = asv.state_fields(st)
        banded = []
        for b in range(B):
            dcs, shape = oracle.tree_shape(float(conf[b]), float(rar[b]), int(brk[b]), params)
            assert got[b].draft_conf == conf[b], b
            assert abs(got[b].dcs - dcs) <= 1e-6 * max(1.0, dcs), (b, got[b].dcs, dcs)
            if b >= 17 and oracle.tree_shape_slack(dcs, int(brk[b]), params) < SHAPE_BAND:
                banded.append(b)
                continue
            assert tuple(got[b].shape) == shape, (b, tuple(got[b].shape), shape)
        assert len(banded) <= B // 100, banded
        # without a fresh confidence the stored one is used
        asv.tree_policy(st, None, cp)
        torch.cuda.synchronize()
        again = asv.state_fields(st)
        assert all(tuple(a.shape) == tuple(g.shape) and a.dcs == g.dcs
                   for a, g in zip(again, got))
    assert ctypes.sizeof(asv.AsvReqState) == asv.STATE_BYTES == 112


def test_malformed_inputs_are_reported(asv, dev):
    """Bad trees, tokens, thresholds and offsets set req_status bits; other requests are
    unaffected and nothing faults."""
    trees = [[-1, 0, 1], [-1, 0, 0], [-1, 0], [-1, 0, 1], [-1, 0]]
    w = custom_workload("bad", 64, 500, trees, 0.3, seed=11, w_std=0.16)
    W = w.weights()
    w64 = oracle.widen_weights(W)
    resolve_with_oracle(w, w64)
    good_ref = reference(w, w64)
    off = w.req_offsets
    w.parent[off[0] + 2] = off[0] + 2          # request 0: parent not before the child
    w.draft_tok[off[1] + 1] = 500              # request 1: token out of range
    w.parent[off[2]] = 0                       # request 2: root with a parent
    tau = w.tau.copy()
    tau[3] = 1.5                               # request 3: threshold outside [0, 1]
    got = _run(asv, w, W, dev, tau=tau)
    assert got["req_status"][0] == asv.RS_BAD_PARENT
    assert got["req_status"][1] == asv.RS_BAD_TOKEN
    assert got["req_status"][2] == asv.RS_BAD_ROOT
    assert got["req_status"][3] == asv.RS_BAD_TAU
    assert got["req_status"][4] == 0
    for b in range(4):
        assert got["accepted_len"][b] == 0 and got["bonus_token"][b] == -1
        assert np.all(got["accepted_path"][off[b]:off[b + 1]] == -1)
    b = 4
    assert got["accepted_len"][b] == good_ref["accepted_len"][b]
    assert got["bonus_token"][b] == good_ref["bonus_token"][b]


@pytest.mark.parametrize("n_req", [2, 1030])
@pytest.mark.parametrize("fault", ["last_not_n", "first_not_zero", "decrease", "empty"])
def test_bad_offsets_reported(asv, dev, n_req, fault):
    """A malformed offsets array flags every request; the row statistics of all N rows are
    still produced (on both the fused and the unfused finishing path)."""
    import torch
    print(f"[bad offsets] n_req={n_req} fault={fault}", flush=True)
    rng = np.random.default_rng(12)
    trees = [[-1, 0], [-1, 0, 0]] + [_rand_tree(rng, 2, 1, 1) for _ in range(n_req - 2)]
    w = custom_workload("badoff", 64, 300, trees, 0.3, seed=12, w_std=0.16)
    W = w.weights()
    w64 = oracle.widen_weights(W)
    resolve_with_oracle(w, w64)
    ref = reference(w, w64)
    d = device_inputs(w, W, dev)
    off = d["req_offsets"]
    if fault == "last_not_n":
        off[n_req] = w.N - 1
    elif fault == "first_not_zero":
        off[0] = 1
    elif fault == "decrease":
        off[1] = off[2] + 1  # request 1 runs backwards, request 0 overlaps request 2
    else:
        off[1] = off[2]     # request 1 empty
    o = asv.verify(d["hidden"], d["w_lm"], d["draft_tok"], d["parent"], off, d["tau"])
    torch.cuda.synchronize()
    got = to_host(o)
    assert np.all(got["req_status"] == asv.RS_BAD_OFFSETS)
    assert np.all(got["accepted_len"] == 0) and np.all(got["bonus_token"] == -1)
    assert np.array_equal(got["row_argmax"], ref["row_argmax"]) or \
        np.all(ref["row_gap"][got["row_argmax"] != ref["row_argmax"]] < 1e-3)
    assert np.max(np.abs(got["row_max"] - ref["row_max"])) < 2e-3


def test_empty_batch(asv, dev):
    import torch
    e = dict(hidden=torch.empty((0, 64), dtype=torch.bfloat16, device=dev),
             w_lm=torch.zeros((10, 64), dtype=torch.bfloat16, device=dev),
             draft_tok=torch.empty(0, dtype=torch.int32, device=dev),
             parent=torch.empty(0, dtype=torch.int32, device=dev),
             req_offsets=torch.zeros(1, dtype=torch.int32, device=dev),
             tau=torch.empty(0, dtype=torch.float32, device=dev))
    o = asv.verify(**e)
    torch.cuda.synchronize()
    assert o.accepted_len.numel() == 0
