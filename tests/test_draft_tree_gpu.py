"""GPU parity of the draft side (asv_draft_step, asv_draft_prune) and of the steps around the
target forward (asv_tree_meta, asv_commit) with the CPU oracle, through the C ABI.

Draft top-4: ids bit-exact outside 1e-3 bands around the logit gaps that decide them (banded
rows must hold a valid top-4 within the band), log-probabilities and log-sum-exp within 2e-3.
Tree growth and pruning: the oracle grows its own trees from its own float64 top-4 and scores;
the GPU's trees (tokens, parents, frontier, pruned layout) must match them bit for bit, scores
within 2e-3 per level. Near-ties (0 < gap < 1e-3) in the oracle's values are handled like the
verification bands: where one orders a frontier row's topk + 1 best logits, the GPU's ranking,
checked to lie within the band, is taken for that row (listed); a tree whose best candidate
scores of a step, or whose pruning cut, sit on a near-tie is listed and no longer compared
(at most a tenth of the batch). Tree metadata and commit: bit-exact.
"""

import ctypes
import os

import numpy as np
import pytest

import oracle
from harness import BAND, MAX_BANDED_FRACTION, TOL_F, log_bands
from workloads import (bf16_weights, build_tree, draft_hidden, draft_shapes, draft_vocab_map,
                       root_tokens)

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


def _t(x, dev):
    import torch
    return torch.from_numpy(np.array(x, copy=True, order="C")).to(dev)


def _bf16(bits, dev):
    import torch
    return _t(np.asarray(bits, dtype=np.uint16).view(np.int16), dev).view(torch.bfloat16)


def _state_with_shapes(asv, shapes, dev):
    raw = b""
    for s in shapes:
        st = asv.AsvReqState()
        st.shape = (ctypes.c_int32 * 3)(*[int(v) for v in s])
        raw += bytes(st)
    return _t(np.frombuffer(raw, dtype=np.uint8).reshape(len(shapes), -1), dev)


def _check_topk(tag, x_bits, w64, vmap, ids, logp, lse):
    """GPU top-4 of every row against the oracle, banded where logits are within 1e-3."""
    x64 = oracle.widen_bf16(x_bits)
    ref = oracle.draft_topk(x64, w64, 4, vmap)
    z = oracle.logits(x64, w64)
    z = np.where(np.isnan(z), -np.inf, z)
    inv = None if vmap is None else {int(t): i for i, t in enumerate(vmap)}
    banded = 0
    # the oracle's float64 log-probabilities of the ids the GPU ranked, for rows whose ranking
    # a near-tie decides (the growth then follows the GPU's valid ranking there)
    ref["gpu_rank_logp"] = np.array(ref["logp"], copy=True)
    for r in range(x64.shape[0]):
        assert abs(lse[r] - ref["lse"][r]) <= TOL_F or lse[r] == ref["lse"][r], (tag, r)
        d_ids = [int(i) if inv is None else inv[int(i)] for i in ids[r]]
        assert len(set(d_ids)) == 4, (tag, r, d_ids)
        zs = ref["zs"][r]
        with np.errstate(invalid="ignore"):
            gaps = zs[:4] - zs[1:5]
        if np.all(gaps > BAND):
            assert list(ids[r]) == list(ref["ids"][r]), (tag, r, list(ids[r]),
                                                        list(ref["ids"][r]))
        else:
            banded += 1
            for j in range(4):
                assert abs(z[r, d_ids[j]] - zs[j]) <= BAND or z[r, d_ids[j]] == zs[j], (tag, r)
                with np.errstate(invalid="ignore"):
                    lp = z[r, d_ids[j]] - ref["lse"][r]
                ref["gpu_rank_logp"][r, j] = lp if np.isfinite(lp) else -np.inf
        for j in range(4):
            want = z[r, d_ids[j]] - ref["lse"][r]
            if np.isfinite(want):
                assert abs(logp[r, j] - want) <= TOL_F, (tag, r, j, logp[r, j], want)
            else:
                assert logp[r, j] == -np.inf, (tag, r, j)
    print(f"[{tag}] draft top-4: {x64.shape[0]} rows, {banded} banded")
    return ref


def _draft_host(out):
    return (out.topk_id.cpu().numpy(), out.topk_logp.cpu().numpy(), out.row_lse.cpu().numpy(),
            out.front_tok.cpu().numpy(),
            None if out.draft_conf is None else out.draft_conf.cpu().numpy())


# ----------------------------------------------------------------------------- draft top-4

@pytest.mark.parametrize("B,V,H,mapped", [(1, 1000, 256, False), (3, 1000, 256, True),
                                          (9, 1000, 256, False), (17, 1000, 256, True),
                                          (40, 777, 128, False), (2, 4, 64, False)])
def test_draft_topk(asv, dev, B, V, H, mapped):
    """Every draft tile family (4, 12 rows: 32-row tile; 36: 64-row; 68: 128-row; 160: two
    128-row tiles, the last ragged), ragged last vocabulary slabs, the id map, and a vocabulary
    of exactly four ids."""
    print(f"case B={B} V={V} H={H} mapped={mapped}", flush=True)
    W = bf16_weights(V, H, 0.5, 11)
    x = draft_hidden(B, H, 0, seed=V)
    vmap = draft_vocab_map(V, 5 * V) if mapped else None
    trees = asv.alloc_draft_trees(B, dev)
    out = asv.draft_step(_bf16(x, dev), _bf16(W, dev), trees, 0, shape=(3, 4, 4),
                         vocab_map=None if vmap is None else _t(vmap, dev))
    ids, logp, lse, _, _ = _draft_host(out)
    _check_topk(f"B{B}V{V}", x, oracle.widen_weights(W), vmap, ids, logp, lse)


@pytest.mark.parametrize("i", range(int(os.environ.get("ASV_RANDOM_DRAFT_CASES", "16"))))
def test_draft_topk_random_shapes(asv, dev, i):
    """Seeded random draft batches: B (every draft tile family), V (ragged slabs, down to the
    four ids of a top-4), H, the id map and the weight layout, against the oracle's top-4."""
    rng = np.random.default_rng([2609, 77, i])
    B = int(rng.integers(1, 49))
    V = int(rng.choice([int(rng.integers(4, 200)), int(rng.integers(200, 5000))]))
    H = 64 * int(rng.integers(1, 9))
    mapped, packed = bool(rng.integers(0, 2)), bool(rng.integers(0, 2))
    print(f"case {i}: B={B} V={V} H={H} mapped={mapped} packed={packed}", flush=True)
    W = bf16_weights(V, H, float(rng.uniform(0.2, 0.8)), 500 + i)
    x = draft_hidden(B, H, 0, seed=700 + i)
    vmap = draft_vocab_map(V, 3 * V + 11) if mapped else None
    w = _bf16(W, dev)
    trees = asv.alloc_draft_trees(B, dev)
    out = asv.draft_step(_bf16(x, dev), asv.pack_draft_head(w) if packed else w, trees, 0,
                         shape=(3, 4, 4), vocab_map=None if vmap is None else _t(vmap, dev))
    ids, logp, lse, _, _ = _draft_host(out)
    _check_topk(f"random{i}", x, oracle.widen_weights(W), vmap, ids, logp, lse)


def test_draft_topk_exact_ties_and_nan(asv, dev):
    """Bit-identical logits (duplicated W rows in different slabs, one in the ragged last slab)
    come out lowest id first without bands; a row holding a non-number ranks every id as -inf."""
    V, H, B = 1000, 128, 2
    W = bf16_weights(V, H, 0.02, 12).copy()
    half = np.uint16(0x3F00)                         # 0.5
    for v in (3, 700, 999):
        W[v] = half
    x = np.full((4 * B, H), np.uint16(0x3F80))      # 1.0: the tied logits are 64 exactly
    x[5, 7] = np.uint16(0x7FC0)                      # NaN in row 5
    trees = asv.alloc_draft_trees(B, dev)
    out = asv.draft_step(_bf16(x, dev), _bf16(W, dev), trees, 0, shape=(2, 3, 8))
    ids, logp, lse, _, _ = _draft_host(out)
    for r in range(4 * B):
        if r == 5:
            assert list(ids[r]) == [0, 1, 2, 3]
            assert np.all(logp[r] == -np.inf) and lse[r] == -np.inf
            continue
        assert list(ids[r][:3]) == [3, 700, 999], (r, list(ids[r]))
        assert logp[r, 0] == logp[r, 1] == logp[r, 2]
        assert abs(logp[r, 0] - (64.0 - lse[r])) < 1e-5


@pytest.mark.parametrize("B,V,H", [(1, 1000, 256), (9, 1000, 256), (17, 1000, 256),
                                   (40, 777, 128), (2, 4, 64), (32, 32000, 4096)])
def test_draft_packed_weight(asv, dev, B, V, H):
    """asv_pack_draft_head writes packed[((k T + s) 64 + r) 64 + c] = w[64 s + r][64 k + c]
    (64 T = V rounded up to a multiple of 128, zero rows past V), checked against torch's
    reshape and permute; draft_step then gives every output and tree bit for bit as with the
    row-major weight, on every draft tile family (4, 36, 68 and 160 rows)."""
    import torch
    print(f"case B={B} V={V} H={H}", flush=True)
    W = bf16_weights(V, H, 0.5, 13)
    x = draft_hidden(B, H, 0, seed=V + 1)
    w = _bf16(W, dev)
    p = asv.pack_draft_head(w)
    torch.cuda.synchronize()
    Vp, KT = -(-V // 128) * 128, H // 64
    assert p.kind == "draft" and p.data.numel() == Vp * H
    pad = torch.zeros((Vp, H), dtype=torch.int16, device=dev)
    pad[:V] = w.view(torch.int16)
    ref = pad.view(Vp // 64, 64, KT, 64).permute(2, 0, 1, 3).contiguous().view(-1)
    assert torch.equal(p.data.view(torch.int16), ref)
    runs = []
    for weight in (w, p):
        trees = asv.alloc_draft_trees(B, dev)
        out = asv.draft_step(_bf16(x, dev), weight, trees, 0, shape=(3, 4, 4), with_conf=True)
        torch.cuda.synchronize()
        runs.append((out, trees))
    (o0, t0), (o1, t1) = runs
    for f in o0._fields:
        assert torch.equal(getattr(o0, f), getattr(o1, f)), f
    for g0, g1 in zip(asv.draft_tree_fields(t0), asv.draft_tree_fields(t1)):
        n, F = g0.n_pool, g0.n_front            # pool entries past n_pool are never written
        assert (g0.nsteps, g0.topk, g0.ndt, g0.steps, g0.status, F, n) == \
               (g1.nsteps, g1.topk, g1.ndt, g1.steps, g1.status, g1.n_front, g1.n_pool)
        assert list(g0.front[:F]) == list(g1.front[:F])
        assert list(g0.front_score[:F]) == list(g1.front_score[:F])
        assert (list(g0.tok[:n]), list(g0.par[:n]), list(g0.score[:n])) == \
               (list(g1.tok[:n]), list(g1.par[:n]), list(g1.score[:n]))
    with pytest.raises(ValueError):
        asv.draft_step(_bf16(x, dev), asv.pack_lm_head(w), asv.alloc_draft_trees(B, dev), 0,
                       shape=(3, 4, 4))


# ----------------------------------------------------------------------------- tree growth

def _near_tie(values, upto):
    """True when two of the ``upto`` + 1 largest values (already sorted best first) differ by
    less than the band without being equal (equal values are ordered the same way on both
    sides: lowest id, earlier candidate)."""
    v = [float(x) for x in values[:upto + 1]]
    return any(0.0 < a - b < BAND for a, b in zip(v, v[1:]) if np.isfinite(a) and np.isfinite(b))


def _oracle_step(trees_ref, ref, gpu_ids, banded, adopted, step):
    """Advance the oracle trees with the oracle's own float64 top-4 of the frontier rows.

    Where a near-tie among a frontier row's topk + 1 best logits decides the ranking of its
    children, the GPU's ranking (checked to lie within the band) is taken, with the oracle's
    log-probabilities of those ids, and the row is listed in ``adopted``. A tree whose best
    candidate scores sit on a near-tie joins ``banded`` (with the reason) and is no longer
    compared."""
    out = []
    for b, t in enumerate(trees_ref):
        ids = np.array(ref["ids"][4 * b:4 * b + len(t.front)], copy=True)
        logp = np.array(ref["logp"][4 * b:4 * b + len(t.front)], copy=True)
        if t.steps < t.nsteps and b not in banded:
            for j in range(len(t.front)):
                r = 4 * b + j
                if _near_tie(ref["zs"][r], t.topk):
                    ids[j], logp[j] = gpu_ids[r], ref["gpu_rank_logp"][r]
                    adopted.append(dict(request=b, step=step, row=r))
            cand = sorted((t.front_score[j] + float(logp[j][c])
                           for j in range(len(t.front)) for c in range(t.topk)), reverse=True)
            if _near_tie(cand, t.topk):
                banded[b] = f"step {step}: near-tie among the best candidate scores"
        out.append(oracle.draft_tree_step(t, ids, logp))
    return out


def _compare_trees(asv, trees, trees_ref, front_tok, grew, banded, tag):
    got = asv.draft_tree_fields(trees)
    for b, (g, t) in enumerate(zip(got, trees_ref)):
        P = len(t.tok)
        assert (g.nsteps, g.topk, g.ndt) == (t.nsteps, t.topk, t.ndt), (tag, b)
        assert g.status == 0 and g.steps == t.steps and g.n_pool == P, (tag, b, g.n_pool, P)
        nf = len(t.front)
        assert g.n_front == nf, (tag, b)
        if b in banded:
            continue
        assert list(g.tok[:P]) == t.tok, (tag, b)
        assert list(g.par[:P]) == t.par, (tag, b)
        tol = TOL_F * max(1, t.steps)
        assert np.allclose(np.array(g.score[:P], np.float64), np.array(t.score), rtol=0,
                           atol=tol), (tag, b)
        assert list(g.front[:nf]) == t.front, (tag, b)
        assert np.allclose(np.array(g.front_score[:nf], np.float64), np.array(t.front_score),
                           rtol=0, atol=tol), (tag, b)
        # a tree that grew this step reports its new frontier's tokens, any other -1s
        want_tok = [t.tok[q] for q in t.front] if grew[b] else []
        exp = (want_tok + [-1] * 4)[:4]
        assert list(front_tok[b]) == exp, (tag, b, list(front_tok[b]), exp)


def _prune_tie(t):
    """True when the oracle's pruning cut (the ndt - 1 best pool nodes) separates two nodes
    whose scores are within the band without being equal. A node and its own descendant are
    not such a pair: log-probabilities are <= 0 in both precisions, so a descendant never
    scores above its ancestor and equal scores keep the earlier pool entry, the ancestor, on
    both sides (a peaked draft row gives a child a log-probability near 0, hence a score
    within 1e-6 of its parent's)."""
    P = len(t.tok)
    m = min(t.ndt - 1, P)
    if m == 0 or m == P:
        return False
    order = sorted(range(P), key=lambda q: (-float(t.score[q]), q))
    kept, dropped = order[:m], order[m:]

    def ancestors(q):
        out = set()
        while q >= 0:
            q = t.par[q]
            out.add(q)
        return out

    lo = float(t.score[kept[-1]])
    for q in dropped:
        if lo - float(t.score[q]) >= BAND:
            break
        anc = ancestors(q)
        for p in kept:
            d = float(t.score[p]) - float(t.score[q])
            if 0.0 < d < BAND and p not in anc:
                return True
    return False


def _grow_and_prune(asv, dev, B, V, H, shapes=None, shape=None, steps=None, vmap=None,
                    W=None, hidden=None, tag=""):
    import torch
    W = bf16_weights(V, H, 0.5, 13) if W is None else W
    w64 = oracle.widen_weights(W)
    trees = asv.alloc_draft_trees(B, dev)
    state = None if shapes is None else _state_with_shapes(asv, shapes, dev)
    all_shapes = shapes if shapes is not None else [shape] * B
    trees_ref = [oracle.draft_tree_init(s) for s in all_shapes]
    steps = steps or max(int(s[0]) for s in all_shapes) + 1
    wd = _bf16(W, dev)
    vm = None if vmap is None else _t(vmap, dev)
    banded, adopted = {}, []
    for s in range(steps):
        x = draft_hidden(B, H, s, seed=7) if hidden is None else hidden(s)
        out = asv.draft_step(_bf16(x, dev), wd, trees, s, state=state, shape=shape,
                             vocab_map=vm, with_conf=True)
        ids, logp, lse, ftok, conf = _draft_host(out)
        ref = _check_topk(f"{tag}s{s}", x, w64, vmap, ids, logp, lse)
        if s == 0:
            for b in range(B):
                want = oracle.draft_top1_prob(ref["logp"][4 * b, 0])
                assert abs(conf[b] - want) <= 2e-3 * max(want, 1e-3), (b, conf[b], want)
        before = [t.steps for t in trees_ref]
        trees_ref = _oracle_step(trees_ref, ref, ids, banded, adopted, s)
        grew = [t.steps > n for t, n in zip(trees_ref, before)]
        _compare_trees(asv, trees, trees_ref, ftok, grew, banded, f"{tag}s{s}")
    roots = root_tokens(B, 1000)
    n_cap = sum(t.ndt for t in trees_ref)
    parent, tok, off, status = asv.draft_prune(trees, n_cap, _t(roots, dev))
    torch.cuda.synchronize()
    for b, t in enumerate(trees_ref):
        if b not in banded and _prune_tie(t):
            banded[b] = "near-tie at the pruning cut"
    pruned = [oracle.draft_tree_prune(t, int(r)) for t, r in zip(trees_ref, roots)]
    par_ref, tok_ref, off_ref = oracle.draft_trees_to_batch(pruned)
    off = off.cpu().numpy()
    assert list(off) == list(off_ref), (tag, list(off), list(off_ref))   # sizes fix the layout
    par_g, tok_g = parent.cpu().numpy(), tok.cpu().numpy()
    for b in range(B):
        lo, hi = int(off[b]), int(off[b + 1])
        assert par_g[lo] == -1 and all(lo <= par_g[c] < c for c in range(lo + 1, hi)), (tag, b)
        if b in banded:
            continue
        assert list(par_g[lo:hi]) == list(par_ref[lo:hi]), (tag, b)
        assert list(tok_g[lo:hi]) == list(tok_ref[lo:hi]), (tag, b)
    assert not status.cpu().numpy().any()
    if banded or adopted:
        log_bands(tag, draft_trees=[dict(request=b, why=why) for b, why in banded.items()],
                  draft_rows_ranked_by_gpu=adopted)
        print(f"[{tag}] banded draft trees: {banded}; rows ranked within the band by the "
              f"GPU: {len(adopted)}", flush=True)
    assert len(banded) <= max(1, MAX_BANDED_FRACTION * B), (tag, banded)
    return trees, trees_ref


@pytest.mark.parametrize("B", [1, 6, 20])
def test_draft_tree_growth_per_request_shapes(asv, dev, B):
    """Per-request shapes from the policy state (the paper's range), one extra step after the
    deepest tree is done, then pruning to the verification layout."""
    print(f"case growth B={B}", flush=True)
    shapes = draft_shapes(B, seed=B)
    _grow_and_prune(asv, dev, B, 1000, 256, shapes=shapes, tag=f"grow{B}")


def test_draft_tree_growth_uniform_shape_with_map(asv, dev):
    vmap = draft_vocab_map(1000, 128256)
    _grow_and_prune(asv, dev, 3, 1000, 256, shape=(4, 4, 12), vmap=vmap, tag="uniform")


def test_draft_tree_growth_with_tied_scores(asv, dev):
    """Every row has three exactly tied best logits and all rows are equal, so candidates tie
    within and across frontier slots: the earlier candidate wins at every step and in pruning."""
    V, H, B = 1000, 128, 2
    W = bf16_weights(V, H, 0.02, 12).copy()
    for v in (3, 700, 999):
        W[v] = np.uint16(0x3F00)
    ones = np.full((4 * B, H), np.uint16(0x3F80))
    _grow_and_prune(asv, dev, B, V, H, shape=(3, 3, 9), W=W, hidden=lambda s: ones,
                    tag="ties")


def test_draft_bad_shape_and_prune_overflow(asv, dev):
    """A bad shape in the state leaves that tree root-only with ASV_DS_BAD_SHAPE; pruning into
    too small an output flags the requests that do not fit and writes none of their rows."""
    import torch
    V, H, B = 600, 128, 3
    W = bf16_weights(V, H, 0.5, 14)
    shapes = [(3, 4, 4), (2, 5, 4), (3, 2, 6)]       # topk 5 is out of range
    state = _state_with_shapes(asv, shapes, dev)
    trees = asv.alloc_draft_trees(B, dev)
    for s in range(3):
        out = asv.draft_step(_bf16(draft_hidden(B, H, s, 3), dev), _bf16(W, dev), trees, s,
                             state=state)
        ftok = out.front_tok.cpu().numpy()
        assert list(ftok[1]) == [-1] * 4
    f = asv.draft_tree_fields(trees)
    assert f[1].status == asv.DS_BAD_SHAPE and f[1].n_pool == 0
    parent, tok, off, status = asv.draft_prune(trees, 100)
    off, status = off.cpu().numpy(), status.cpu().numpy()
    n0 = 1 + min(3, f[0].n_pool)
    assert list(off) == [0, n0, n0 + 1, n0 + 1 + 1 + min(5, f[2].n_pool)]
    assert status[1] == asv.DS_BAD_SHAPE and status[0] == 0 and status[2] == 0
    assert parent.cpu().numpy()[n0] == -1          # the bad tree's root
    cap = n0 + 1                                    # the third tree does not fit
    p2, t2, off2, st2 = asv.draft_prune(trees, cap)
    torch.cuda.synchronize()
    assert list(off2.cpu().numpy()) == list(off)
    st2 = st2.cpu().numpy()
    assert st2[2] == asv.DS_OVERFLOW and st2[0] == 0 and st2[1] == asv.DS_BAD_SHAPE


# ----------------------------------------------------------------------------- tree metadata

def _pack_vis(vis, words):
    n = vis.shape[0]
    out = np.zeros((n, words), dtype=np.uint32)
    for c in range(n):
        for j in np.nonzero(vis[c])[0]:
            out[c, j >> 5] |= np.uint32(1) << np.uint32(j & 31)
    return out


def _random_batch(kinds, seed):
    rng = np.random.default_rng(seed)
    trees = [build_tree(k, rng, b) for b, k in enumerate(kinds)]
    off = np.cumsum([0] + [len(t) for t in trees])
    parent = np.concatenate([[p + off[b] if p >= 0 else -1 for p in t]
                             for b, t in enumerate(trees)]).astype(np.int32)
    return parent, off.astype(np.int32)


@pytest.mark.parametrize("kinds", [["eagle60"], ["tiny", "level8x8", "adaptive", "tiny"],
                                   ["chain_or_wide"] * 6])
def test_tree_meta(asv, dev, kinds):
    import torch
    parent, off = _random_batch(kinds, len(kinds))
    B = len(off) - 1
    n_max = int(np.diff(off).max())
    words = (n_max + 31) // 32 + 1                   # one spare word must come out zero
    base = np.arange(B, dtype=np.int32) * 1000 + 17
    pos, mask, status = asv.tree_meta(_t(parent, dev), _t(off, dev), _t(base, dev), words)
    torch.cuda.synchronize()
    depth, pos_ref, vis = oracle.tree_meta(parent, off, base)
    assert list(pos.cpu().numpy()) == list(pos_ref)
    m = mask.cpu().numpy().view(np.uint32)
    for b in range(B):
        assert np.array_equal(m[off[b]:off[b + 1]], _pack_vis(vis[b], words)), b
    assert not status.cpu().numpy().any()
    pos2, _, _ = asv.tree_meta(_t(parent, dev), _t(off, dev))          # positions only
    assert list(pos2.cpu().numpy()) == list(depth)


def test_tree_meta_large_request_and_status(asv, dev):
    """A 9000-node request (walked from global memory, past the LDS stage), a mask too narrow
    for it, a bad parent, a bad root, and malformed offsets."""
    import torch
    rng = np.random.default_rng(5)
    n = 9000
    big = np.array([-1] + [int(rng.integers(max(0, c - 40), c)) for c in range(1, n)])
    small = np.array([-1, 0, 0, 1])
    parent = np.concatenate([big, small + n]).astype(np.int32)
    parent[n] = -1
    off = np.array([0, n, n + 4], dtype=np.int32)
    words = (n + 31) // 32
    pos, mask, status = asv.tree_meta(_t(parent, dev), _t(off, dev), None, words)
    torch.cuda.synchronize()
    depth, _, vis = oracle.tree_meta(parent, off, np.zeros(2, np.int64))
    assert list(pos.cpu().numpy()) == list(depth)
    m = mask.cpu().numpy().view(np.uint32)
    packed = np.packbits(vis[0], axis=1, bitorder="little")
    packed = np.pad(packed, ((0, 0), (0, 4 * words - packed.shape[1])))
    assert np.array_equal(m[:n], packed.view(np.uint32)[:, :words])
    # a mask too small for the big request: positions only, status set
    _, _, st = asv.tree_meta(_t(parent, dev), _t(off, dev), None, 4)
    assert list(st.cpu().numpy()) == [asv.RS_MASK_SMALL, 0]
    bad = parent.copy()
    bad[n + 3] = n + 3                               # a node that is its own parent
    _, _, st = asv.tree_meta(_t(bad, dev), _t(off, dev), None, 1)
    assert list(st.cpu().numpy()) == [asv.RS_MASK_SMALL, asv.RS_BAD_PARENT]
    bad = parent.copy()
    bad[n] = 3
    _, _, st = asv.tree_meta(_t(bad, dev), _t(off, dev), None, 0)
    assert list(st.cpu().numpy()) == [0, asv.RS_BAD_ROOT]
    _, _, st = asv.tree_meta(_t(parent, dev), _t(np.array([0, n + 4, n], np.int32), dev))
    assert list(st.cpu().numpy()) == [asv.RS_BAD_OFFSETS] * 2


# ----------------------------------------------------------------------------- commit

def _accepted_paths(parent, off, rng):
    N, B = len(parent), len(off) - 1
    path = np.full(N, -1, dtype=np.int32)
    acc = np.zeros(B, dtype=np.int32)
    for b in range(B):
        cur, k = int(off[b]), 0
        while True:
            kids = [c for c in range(off[b] + 1, off[b + 1]) if parent[c] == cur]
            if not kids or rng.random() < 0.25:
                break
            cur = kids[int(rng.integers(len(kids)))]
            path[off[b] + k] = cur
            k += 1
        acc[b] = k
    return path, acc


def test_commit(asv, dev):
    import torch
    rng = np.random.default_rng(21)
    parent, off = _random_batch(["tiny", "eagle60", "level8x8", "tiny", "adaptive"], 3)
    N, B = len(parent), len(off) - 1
    tok = rng.integers(0, 128256, N).astype(np.int32)
    path, acc = _accepted_paths(parent, off, rng)
    bonus = rng.integers(0, 128256, B).astype(np.int32)
    rows16 = rng.integers(-2**31, 2**31, (N, 8)).astype(np.int32)     # 32-byte rows
    rows4 = rng.integers(-2**31, 2**31, (N, 3)).astype(np.int32)      # 12-byte rows
    ref = oracle.commit(path, acc, bonus, tok, off)
    total = int(ref["off"][-1])
    for rows in (rows16, rows4, None):
        c_off, c_tok, c_row, dst, status = asv.commit(
            _t(off, dev), _t(tok, dev), _t(acc, dev), _t(path, dev), _t(bonus, dev),
            None if rows is None else _t(rows, dev))
        torch.cuda.synchronize()
        assert list(c_off.cpu().numpy()) == list(ref["off"])
        assert list(c_tok.cpu().numpy()[:total]) == list(ref["tok"])
        assert list(c_row.cpu().numpy()[:total]) == list(ref["row"])
        assert not status.cpu().numpy().any()
        if rows is not None:
            assert np.array_equal(dst.cpu().numpy()[:total], rows[ref["row"]])


def test_commit_bad_path_and_offsets(asv, dev):
    import torch
    parent, off = _random_batch(["tiny", "tiny", "tiny"], 4)
    N, B = len(parent), len(off) - 1
    rng = np.random.default_rng(8)
    tok = rng.integers(0, 1000, N).astype(np.int32)
    path, acc = _accepted_paths(parent, off, rng)
    acc[0] = int(off[1] - off[0])                     # longer than the request allows
    path[off[2]] = off[0] + 1                         # a node of another request
    acc[2] = max(acc[2], 1)
    bonus = np.array([5, 6, 7], dtype=np.int32)
    c_off, c_tok, c_row, _, status = asv.commit(_t(off, dev), _t(tok, dev), _t(acc, dev),
                                                 _t(path, dev), _t(bonus, dev))
    torch.cuda.synchronize()
    st = status.cpu().numpy()
    assert st[0] == asv.RS_BAD_PATH and st[1] == 0 and st[2] == asv.RS_BAD_PATH
    c_off = c_off.cpu().numpy()
    assert c_off[1] == 1 and c_off[3] - c_off[2] == 1
    assert c_tok.cpu().numpy()[0] == 5 and c_row.cpu().numpy()[0] == off[0]
    assert c_tok.cpu().numpy()[c_off[2]] == 7 and c_row.cpu().numpy()[c_off[2]] == off[2]
    _, _, _, _, st = asv.commit(_t(np.array([0, 3, 2, N], np.int32), dev), _t(tok, dev),
                                _t(acc, dev), _t(path, dev), _t(bonus, dev))
    assert list(st.cpu().numpy()) == [asv.RS_BAD_OFFSETS] * 3


def test_commit_bad_path_on_first_request(asv, dev):
    """Request 0's accepted length is in range but its path holds a node of request 1: it
    commits its root row and bonus only, and requests 1 and 2 start right after it, with their
    own tokens and rows (the offsets of later requests use the same validated counts)."""
    import torch
    parent, off = _random_batch(["eagle60", "eagle60", "tiny"], 6)
    N = len(parent)
    rng = np.random.default_rng(9)
    tok = rng.integers(0, 1000, N).astype(np.int32)
    path, acc = _accepted_paths(parent, off, np.random.default_rng(10))
    # request 0: a three-node path whose last entry is a node of request 1
    deep = next(c for c in range(off[0] + 1, off[1]) if parent[c] != off[0])
    chain = [int(parent[deep]), int(deep)]
    path[off[0]:off[0] + 3] = chain + [int(off[1]) + 1]
    acc[0] = 3
    acc[1] = max(int(acc[1]), 1)
    if acc[1] == 1 and path[off[1]] < 0:
        path[off[1]] = [c for c in range(off[1] + 1, off[2]) if parent[c] == off[1]][0]
    bonus = np.array([5, 6, 7], dtype=np.int32)
    rows = rng.integers(-2**31, 2**31, (N, 4)).astype(np.int32)
    c_off, c_tok, c_row, dst, status = asv.commit(_t(off, dev), _t(tok, dev), _t(acc, dev),
                                                   _t(path, dev), _t(bonus, dev), _t(rows, dev))
    torch.cuda.synchronize()
    st = status.cpu().numpy()
    assert list(st) == [asv.RS_BAD_PATH, 0, 0], list(st)
    good_acc = acc.copy()
    good_acc[0] = 0
    ref = oracle.commit(path, good_acc, bonus, tok, off)
    total = int(ref["off"][-1])
    c_off = c_off.cpu().numpy()
    assert list(c_off) == list(ref["off"]) and c_off[1] == 1
    assert list(c_tok.cpu().numpy()[:total]) == list(ref["tok"])
    assert list(c_row.cpu().numpy()[:total]) == list(ref["row"])
    assert c_row.cpu().numpy()[1] == off[1] and c_tok.cpu().numpy()[0] == 5
    assert np.array_equal(dst.cpu().numpy()[:total], rows[ref["row"]])


# ----------------------------------------------------------------------------- full size

@pytest.mark.parametrize("name", ["llama31_8b_draft_b1", "llama31_8b_draft_b32"])
def test_draft_full_size(asv, dev, name):
    """The bench workloads (H=4096, 32000 draft ids mapped into the 128256-id target vocabulary,
    trees (3,4,4)) in bench.py's launch configuration: every row's top-4 against the oracle, then
    three growth steps and pruning bit-exact against the oracle's own trees."""
    from workloads import make_draft_workload
    dw = make_draft_workload(name)
    print(f"case {name}", flush=True)
    W = dw.weights()
    _grow_and_prune(asv, dev, dw.B, dw.V, dw.H, shape=(3, 4, 4), vmap=dw.vocab_map(), W=W,
                    hidden=lambda s: dw.hidden(s), tag=name)


def test_many_requests(asv, dev):
    """600 requests: the offset sums of pruning, tree metadata and commit run over several
    rounds of their workgroup; a 150-request draft batch spans five 128-row tiles."""
    import torch
    rng = np.random.default_rng(31)
    # draft side: 150 requests, per-request shapes, small vocabulary
    B, V, H = 150, 300, 64
    shapes = draft_shapes(B, seed=3)
    _grow_and_prune(asv, dev, B, V, H, shapes=shapes, tag="many")
    # tree metadata and commit: 600 requests of 1..40 nodes
    sizes = rng.integers(1, 41, 600)
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    parent = np.full(off[-1], -1, dtype=np.int32)
    for b, n in enumerate(sizes):
        for c in range(1, n):
            parent[off[b] + c] = off[b] + int(rng.integers(c))
    base = rng.integers(0, 5000, 600).astype(np.int32)
    pos, mask, st = asv.tree_meta(_t(parent, dev), _t(off, dev), _t(base, dev), 2)
    torch.cuda.synchronize()
    depth, pos_ref, vis = oracle.tree_meta(parent, off, base)
    assert list(pos.cpu().numpy()) == list(pos_ref) and not st.cpu().numpy().any()
    m = mask.cpu().numpy().view(np.uint32)
    for b in range(0, 600, 37):
        assert np.array_equal(m[off[b]:off[b + 1]], _pack_vis(vis[b], 2)), b
    tok = rng.integers(0, 1000, off[-1]).astype(np.int32)
    path, acc = _accepted_paths(parent, off, rng)
    bonus = rng.integers(0, 1000, 600).astype(np.int32)
    c_off, c_tok, c_row, _, cst = asv.commit(_t(off, dev), _t(tok, dev), _t(acc, dev),
                                             _t(path, dev), _t(bonus, dev))
    torch.cuda.synchronize()
    ref = oracle.commit(path, acc, bonus, tok, off)
    total = int(ref["off"][-1])
    assert list(c_off.cpu().numpy()) == list(ref["off"]) and not cst.cpu().numpy().any()
    assert list(c_tok.cpu().numpy()[:total]) == list(ref["tok"])
    assert list(c_row.cpu().numpy()[:total]) == list(ref["row"])
