"""The entry points under HIP graph capture (torch.cuda.CUDAGraph on ROCm).

A verification step and a draft phase (three draft steps and the pruning) have static launch
shapes, so a serving loop can capture them once and replay them. Each graph is replayed several
times with fresh inputs copied into its static tensors, with eager work and synchronisations
between replays, and every replay is compared bit for bit with the same call run eagerly.
"""

import numpy as np
import pytest

from workloads import bf16_weights, custom_workload, draft_hidden

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


def _bf16(bits, dev):
    import torch
    return torch.from_numpy(np.array(bits, copy=True).view(np.int16)).to(dev).view(
        torch.bfloat16)


def _same(a, b):
    import torch
    if a is None:
        return b is None
    return torch.equal(a.view(torch.uint8) if a.dtype == torch.float32 else a,
                       b.view(torch.uint8) if b.dtype == torch.float32 else b)


def _same_trees(asv, a, b, tag):
    """Equal tree records: header, the filled frontier slots and the filled pool entries (the
    rest of a record is never written)."""
    for x, y in zip(asv.draft_tree_fields(a), asv.draft_tree_fields(b)):
        head = ("nsteps", "topk", "ndt", "steps", "n_pool", "n_front", "status")
        assert [getattr(x, f) for f in head] == [getattr(y, f) for f in head], tag
        nf, P = x.n_front, x.n_pool
        assert list(x.front[:nf]) == list(y.front[:nf]), tag
        assert bytes(x.front_score)[:4 * nf] == bytes(y.front_score)[:4 * nf], tag
        assert list(x.tok[:P]) == list(y.tok[:P]) and list(x.par[:P]) == list(y.par[:P]), tag
        assert bytes(x.score)[:4 * P] == bytes(y.score)[:4 * P], tag


def _chain_and_fans(n_req, size):
    """n_req requests of `size` nodes: a chain of four, the rest fanned out under its tip."""
    return [[-1, 0, 1, 2] + [3] * (size - 4) for _ in range(n_req)]


# one tree set per K1 tile family, the tile pinned: 20 rows (64-row tile, burst ring), 200 rows
# (128-row tile, three-slot spread loop), 300 rows (192-row tile) and 520 rows (256-row tile,
# both two-slot spread loop)
GRAPH_TREES = {
    "rows64": [[-1, 0, 0, 1, 1, 2, 3], [-1, 0, 1], [-1] + [0] * 9],
    "rows128": _chain_and_fans(5, 40),
    "rows192": _chain_and_fans(6, 50),
    "rows256": _chain_and_fans(8, 65),
}
GRAPH_TILE = {"rows64": 64, "rows128": 128, "rows192": 192, "rows256": 256}


@pytest.mark.parametrize("packed", [False, True])
@pytest.mark.parametrize("family", list(GRAPH_TREES))
def test_verify_graph_replays(asv, dev, family, packed):
    """The graph is captured on the row-major or the packed weight; every replay is compared
    with an eager call on the row-major weight."""
    import torch
    print(f"[graph] verify {family} packed={packed}", flush=True)
    trees = GRAPH_TREES[family]
    w = custom_workload("graph", 256, 3000, trees, 0.2, seed=41, w_std=0.1)
    rng = np.random.default_rng(5)
    w.draft_tok = rng.integers(0, 3000, w.N).astype(np.int32)
    W = _bf16(w.weights(), dev)
    Wg = asv.pack_lm_head(W) if packed else W
    hidden = _bf16(w.hidden, dev)
    tok = torch.from_numpy(w.draft_tok).to(dev)
    par = torch.from_numpy(w.parent.astype(np.int32)).to(dev)
    off = torch.from_numpy(w.req_offsets.astype(np.int32)).to(dev)
    tau = torch.from_numpy(w.tau).to(dev)
    out_g = asv.alloc_outputs(w.B, w.N, dev, False)
    ws_g = asv.alloc_workspace(w.B, w.N, w.H, w.V, dev)
    state_g = asv.state_init(w.B, device=dev)
    # warm-up on a side stream, as torch requires before capture
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    tile = GRAPH_TILE[family]
    with torch.cuda.stream(s):
        asv.verify(hidden, Wg, tok, par, off, tau, state=state_g, out=out_g, workspace=ws_g,
                   k1_tile=tile)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        asv.verify(hidden, Wg, tok, par, off, tau, state=state_g, out=out_g, workspace=ws_g,
                   k1_tile=tile)
    for r in range(4):
        x = np.random.default_rng([9, r]).standard_normal((w.N, w.H)).astype(np.float32)
        hidden.copy_(_bf16((x.view(np.uint32) >> 16).astype(np.uint16), dev))
        tok.copy_(torch.from_numpy(rng.integers(0, 3000, w.N).astype(np.int32)).to(dev))
        st0 = asv.state_init(w.B, device=dev)
        state_g.copy_(st0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        st_e = st0.clone()
        ref = asv.verify(hidden, W, tok, par, off, tau, state=st_e, k1_tile=tile)
        torch.cuda.synchronize()
        nonroot = torch.from_numpy(w.parent >= 0).to(dev)
        for f in ref._fields:
            a, b = getattr(ref, f), getattr(out_g, f)
            if f == "drafted_logit":            # unspecified at roots
                a, b = a[nonroot], b[nonroot]
            assert _same(a, b), (r, f)
        assert torch.equal(st_e, state_g), r


@pytest.mark.parametrize("packed", [False, True])
def test_draft_phase_graph_replays(asv, dev, packed):
    """Captured on the row-major or the packed draft weight; every replay is compared with
    eager calls on the row-major weight."""
    import torch
    print(f"[graph] draft phase packed={packed}", flush=True)
    B, H, V = 3, 128, 700
    Wd = _bf16(bf16_weights(V, H, 0.5, 42), dev)
    Wg = asv.pack_draft_head(Wd) if packed else Wd
    xs = [_bf16(draft_hidden(B, H, k, seed=11), dev) for k in range(3)]
    trees_g = asv.alloc_draft_trees(B, dev)
    ws = torch.empty(asv.draft_workspace_bytes(B, H, V), dtype=torch.uint8, device=dev)
    outs = [asv.draft_step(xs[k], Wg, trees_g, k, shape=(3, 3, 7), workspace=ws)
            for k in range(3)]
    n_cap = B * 7
    par_g = torch.empty(n_cap, dtype=torch.int32, device=dev)
    tok_g = torch.empty(n_cap, dtype=torch.int32, device=dev)
    off_g = torch.empty(B + 1, dtype=torch.int32, device=dev)
    st_g = torch.empty(B, dtype=torch.int32, device=dev)
    def prune():
        rc = asv.load().asv_draft_prune(trees_g.data_ptr(), B, None, n_cap, par_g.data_ptr(),
                                        tok_g.data_ptr(), off_g.data_ptr(), st_g.data_ptr(),
                                        torch.cuda.current_stream(dev).cuda_stream)
        assert rc == 0

    def phase():
        for k in range(3):
            asv.draft_step(xs[k], Wg, trees_g, k, shape=(3, 3, 7), out=outs[k], workspace=ws)
        prune()

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        phase()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        phase()
    for r in range(4):
        for k in range(3):
            xs[k].copy_(_bf16(draft_hidden(B, H, k, seed=100 + r), dev))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        trees_e = asv.alloc_draft_trees(B, dev)
        eager = [asv.draft_step(xs[k], Wd, trees_e, k, shape=(3, 3, 7)) for k in range(3)]
        pe, te, oe, se = asv.draft_prune(trees_e, n_cap)
        torch.cuda.synchronize()
        for k in range(3):
            for f in ("topk_id", "topk_logp", "row_lse", "front_tok"):
                assert _same(getattr(eager[k], f), getattr(outs[k], f)), (r, k, f)
        _same_trees(asv, trees_e, trees_g, r)
        n = int(oe[-1])
        assert torch.equal(oe, off_g) and torch.equal(se, st_g), r
        assert torch.equal(pe[:n], par_g[:n]) and torch.equal(te[:n], tok_g[:n]), r
