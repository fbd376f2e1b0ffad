"""Checks that pin the draft-tree, tree-metadata and commit parts of the CPU oracle to the paper
and to mathematics, not to themselves.

Each ``check_*`` takes the ``oracle.tree_oracle`` module (or a stand-in with the same
functions) and raises AssertionError on a mismatch. ``test_tree_oracle_pins.py`` runs them on the
real oracle and ``test_tree_oracle_mutations.py`` on deliberately broken copies.
"""

from __future__ import annotations

import json
import os
from fractions import Fraction

import numpy as np
from scipy.special import logsumexp, softmax

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _bf16_values(rng, shape, std):
    x = (rng.standard_normal(shape) * std).astype(np.float32)
    return (x.view(np.uint32) & np.uint32(0xFFFF0000)).view(np.float32).astype(np.float64)


# ----------------------------------------------------------------------------- draft top-k

def check_topk_brute_force(tor):
    """Exact rational logits, a Python sort on (-logit, id) and the library log-sum-exp."""
    rng = np.random.default_rng(5)
    R, V, H, k = 4, 17, 5, 4
    x = _bf16_values(rng, (R, H), 1.0)
    w = _bf16_values(rng, (V, H), 0.6)
    w[9] = w[3]                                   # an exact tie in every row: ids 3 and 9
    out = tor.draft_topk(x, w, k)
    for r in range(R):
        z = [float(sum(Fraction(float(w[v, h])) * Fraction(float(x[r, h])) for h in range(H)))
             for v in range(V)]
        want = sorted(range(V), key=lambda v: (-z[v], v))[:k]
        assert list(out["ids"][r]) == want, (r, list(out["ids"][r]), want)
        lse = logsumexp(z)
        assert abs(out["lse"][r] - lse) < 1e-12
        for j, v in enumerate(want):
            assert abs(out["logp"][r, j] - (z[v] - lse)) < 1e-12
        srt = sorted(z, reverse=True)
        assert np.allclose(out["zs"][r], srt[:k + 1], rtol=0, atol=1e-12)


def check_topk_ties_and_argmax(tor):
    """k = 1 is the first-occurrence argmax; equal logits come out lowest id first."""
    rng = np.random.default_rng(6)
    x = _bf16_values(rng, (3, 8), 1.0)
    w = _bf16_values(rng, (40, 8), 0.5)
    out = tor.draft_topk(x, w, 1)
    assert list(out["ids"][:, 0]) == list(np.argmax(x @ w.T, axis=1))
    w_eq = np.tile(w[:1], (6, 1))                 # six identical vocabulary rows
    out = tor.draft_topk(x, w_eq, 4)
    for r in range(3):
        assert list(out["ids"][r]) == [0, 1, 2, 3]
        assert np.allclose(out["logp"][r], -np.log(6.0), rtol=0, atol=1e-12)


def check_topk_probabilities(tor):
    """With k = V the log-probabilities are the full log-softmax (library routine): their
    exponentials sum to one and the best one is the softmax maximum of Eq. (2)."""
    rng = np.random.default_rng(7)
    x = _bf16_values(rng, (2, 6), 1.0)
    w = _bf16_values(rng, (9, 6), 0.8)
    out = tor.draft_topk(x, w, 9)
    z = x @ w.T
    p = softmax(z, axis=1)
    for r in range(2):
        assert abs(np.exp(out["logp"][r]).sum() - 1.0) < 1e-12
        for j in range(9):
            assert abs(np.exp(out["logp"][r, j]) - p[r, out["ids"][r, j]]) < 1e-12
        assert abs(tor.draft_top1_prob(out["logp"][r, 0]) - p[r].max()) < 1e-6


def check_topk_map_and_nan(tor):
    """The draft-to-target id map applies after the ranking; a row of non-numbers ranks every
    id as -inf, so its top-k is the lowest ids with log-probability -inf."""
    rng = np.random.default_rng(8)
    x = _bf16_values(rng, (2, 4), 1.0)
    w = _bf16_values(rng, (12, 4), 0.5)
    vmap = np.arange(12) * 5 + 3
    plain = tor.draft_topk(x, w, 3)
    mapped = tor.draft_topk(x, w, 3, vocab_map=vmap)
    assert np.array_equal(mapped["ids"], vmap[plain["ids"]])
    assert np.array_equal(mapped["logp"], plain["logp"])
    x[1, 2] = np.nan
    out = tor.draft_topk(x, w, 3)
    assert list(out["ids"][1]) == [0, 1, 2]
    assert np.all(out["logp"][1] == -np.inf)
    assert np.array_equal(out["ids"][0], plain["ids"][0])


# ----------------------------------------------------------------------------- tree growth

def _grow(tor, shape, steps):
    t = tor.draft_tree_init(shape)
    for s in steps:
        t = tor.draft_tree_step(t, np.asarray(s["ids"]), np.asarray(s["logp"], np.float32))
    return t


def check_draft_tree_golden(tor):
    """The hand-worked example of tests/golden/draft_tree_example.json."""
    g = _golden("draft_tree_example.json")
    t = tor.draft_tree_init((g["nsteps"], g["topk"], 6))
    for s, front in zip(g["steps"], g["frontier_after_step"]):
        t = tor.draft_tree_step(t, np.asarray(s["ids"]), np.asarray(s["logp"], np.float32))
        assert list(t.front) == front, (list(t.front), front)
    assert [float(v) for v in t.score] == g["pool_score"]
    for ndt, want in g["expected"].items():
        t2 = tor.draft_tree_init((g["nsteps"], g["topk"], int(ndt)))
        for s in g["steps"]:
            t2 = tor.draft_tree_step(t2, np.asarray(s["ids"]),
                                     np.asarray(s["logp"], np.float32))
        out = tor.draft_tree_prune(t2, g["root_tok"])
        assert list(out["parent"]) == want["parent"], (ndt, list(out["parent"]))
        assert list(out["tok"]) == want["tok"], (ndt, list(out["tok"]))


def check_draft_tree_chain(tor):
    """topk = 1 is a chain: one node per step holding the top-1 token of the previous node's
    row, cut to ndt - 1 drafted nodes; extra steps past nsteps change nothing."""
    rng = np.random.default_rng(9)
    for nsteps, ndt in ((5, 8), (5, 3), (1, 4), (4, 1)):
        t = tor.draft_tree_init((nsteps, 1, ndt))
        toks = []
        for s in range(nsteps + 2):
            tok = int(rng.integers(1000))
            if s < nsteps:
                toks.append(tok)
            t = tor.draft_tree_step(t, np.array([[tok, 1]]),
                                    np.array([[-rng.random(), -5.0]], np.float32))
        out = tor.draft_tree_prune(t, 42)
        m = min(nsteps, ndt - 1)
        assert list(out["parent"]) == [-1] + list(range(m))
        assert list(out["tok"]) == [42] + toks[:m]


def _beam_by_levels(logp_of, nsteps, topk, ndt):
    """Independent statement of the growth on the complete topk-ary tree: a node is a tuple of
    child ranks, its score the sum of the log-probabilities along it; level d + 1 holds the
    children of the topk best nodes of level d; the result is the set of the ndt - 1 best
    nodes of all levels."""
    level = [((c,), float(logp_of(())[c])) for c in range(topk)]
    pool = list(level)
    for _ in range(1, nsteps):
        beam = sorted(level, key=lambda e: -float(e[1]))[:topk]
        level = [(node + (c,), s + float(logp_of(node)[c]))
                 for node, s in beam for c in range(topk)]
        pool += level
    keep = sorted(pool, key=lambda e: -float(e[1]))[:ndt - 1]
    return {node for node, _ in keep}, len(pool)


def check_draft_tree_levels(tor):
    """Random trees against the level-set statement above, plus the invariants of a pruned
    tree: parents first, ancestors kept, every kept node at least as good as every dropped one."""
    rng = np.random.default_rng(10)
    for trial in range(40):
        nsteps, topk = int(rng.integers(1, 5)), int(rng.integers(1, 4))
        ndt = int(rng.integers(1, 16))
        table = {}

        def logp_of(node):
            if node not in table:
                table[node] = np.sort(np.log(rng.random(4)).astype(np.float32))[::-1]
            return table[node]

        want, pool_size = _beam_by_levels(logp_of, nsteps, topk, ndt)
        t = tor.draft_tree_init((nsteps, topk, ndt))

        def path_of(q):
            out = []
            while q >= 0:
                out.append(t.tok[q])
                q = t.par[q]
            return tuple(reversed(out))

        for _ in range(nsteps):
            nodes = [() if f < 0 else path_of(f) for f in t.front]
            ids = np.array([[0, 1, 2, 3]] * len(nodes))          # token = child rank
            logp = np.array([logp_of(n) for n in nodes], np.float32)
            t = tor.draft_tree_step(t, ids, logp)
        out = tor.draft_tree_prune(t)
        par, tok = list(out["parent"]), list(out["tok"])
        assert len(par) == min(ndt, 1 + pool_size)
        got = set()
        for i in range(1, len(par)):
            assert 0 <= par[i] < i, (trial, par)
            path, j = [], i
            while j > 0:
                path.append(tok[j])
                j = par[j]
            got.add(tuple(reversed(path)))
        assert got == want, (trial, sorted(got), sorted(want))


def check_trees_to_batch(tor):
    """Per-request pruned trees laid out as verification reads them, against hand-built global
    parent ids: request b's local node i becomes row off[b] + i, roots keep -1."""
    pruned = [dict(parent=np.array([-1, 0, 0, 1]), tok=np.array([7, 3, 4, 5])),
              dict(parent=np.array([-1]), tok=np.array([9])),
              dict(parent=np.array([-1, 0, 1, 1, 0]), tok=np.array([1, 2, 3, 6, 8]))]
    par, tok, off = tor.draft_trees_to_batch(pruned)
    assert list(off) == [0, 4, 5, 10]
    assert list(par) == [-1, 0, 0, 1, -1, -1, 5, 6, 6, 5]
    assert list(tok) == [7, 3, 4, 5, 9, 1, 2, 3, 6, 8]
    par, tok, off = tor.draft_trees_to_batch([])
    assert list(off) == [0] and len(par) == len(tok) == 0
    # every row's parent lies in its own request, before it
    rng = np.random.default_rng(3)
    trees = []
    for n in rng.integers(1, 9, 12):
        trees.append(dict(parent=np.array([-1] + [int(rng.integers(c)) for c in range(1, n)]),
                          tok=rng.integers(0, 100, n)))
    par, tok, off = tor.draft_trees_to_batch(trees)
    for b, t in enumerate(trees):
        lo, hi = int(off[b]), int(off[b + 1])
        assert hi - lo == len(t["parent"]) and par[lo] == -1
        assert all(lo <= par[c] < c for c in range(lo + 1, hi))
        assert list(par[lo + 1:hi] - lo) == list(t["parent"][1:])
        assert list(tok[lo:hi]) == list(t["tok"])


# ----------------------------------------------------------------------------- tree metadata

def check_tree_meta_golden(tor):
    g = _golden("tree_meta_example.json")
    parent = np.array(g["parent"])
    depth, pos, vis = tor.tree_meta(parent, np.array([0, len(parent)]), np.array([g["pos_base"]]))
    assert list(depth) == g["depth"]
    assert list(pos) == [g["pos_base"] + d for d in g["depth"]]
    bits = [int(sum(1 << j for j in range(len(parent)) if vis[0][i, j]))
            for i in range(len(parent))]
    assert bits == g["mask_bits"], [hex(b) for b in bits]


def check_tree_meta_closure(tor):
    """Visibility is the reflexive-transitive closure of the parent relation, computed here by
    boolean matrix powers; depth is the number of strict ancestors; requests are independent."""
    rng = np.random.default_rng(12)
    sizes = [1, 2, 9, 30, 5]
    off = np.cumsum([0] + sizes)
    parent = np.full(off[-1], -1)
    for b, n in enumerate(sizes):
        for c in range(1, n):
            parent[off[b] + c] = off[b] + int(rng.integers(c))
    base = rng.integers(0, 1000, len(sizes))
    depth, pos, vis = tor.tree_meta(parent, off, base)
    for b, n in enumerate(sizes):
        lo = off[b]
        A = np.zeros((n, n), dtype=np.int64)
        for c in range(1, n):
            A[c, parent[lo + c] - lo] = 1
        reach = np.eye(n, dtype=np.int64)
        for _ in range(n):
            reach = np.minimum(1, reach + reach @ A)
        assert np.array_equal(vis[b], reach.astype(bool)), b
        for c in range(n):
            assert depth[lo + c] == reach[c].sum() - 1
            assert pos[lo + c] == base[b] + depth[lo + c]


# ----------------------------------------------------------------------------- commit

def check_commit_golden(tor):
    g = _golden("commit_example.json")
    out = tor.commit(np.array(g["accepted_path"]), np.array(g["accepted_len"]),
                     np.array(g["bonus"]), np.array(g["draft_tok"]), np.array(g["req_offsets"]))
    assert list(out["off"]) == g["off"]
    assert list(out["tok"]) == g["tok"]
    assert list(out["row"]) == g["row"]


def check_commit_is_root_prefix(tor):
    """Kept rows run from the root down one parent link at a time; tokens are the drafted
    tokens of all but the root followed by the bonus."""
    rng = np.random.default_rng(13)
    sizes = [4, 1, 7, 3]
    off = np.cumsum([0] + sizes)
    parent = np.full(off[-1], -1)
    for b, n in enumerate(sizes):
        for c in range(1, n):
            parent[off[b] + c] = off[b] + int(rng.integers(c))
    tok = rng.integers(0, 500, off[-1])
    path = np.full(off[-1], -1)
    acc = np.zeros(len(sizes), dtype=np.int64)
    for b in range(len(sizes)):
        cur, k = off[b], 0
        while True:
            kids = [c for c in range(off[b] + 1, off[b + 1]) if parent[c] == cur]
            if not kids or rng.random() < 0.3:
                break
            cur = kids[int(rng.integers(len(kids)))]
            path[off[b] + k] = cur
            k += 1
        acc[b] = k
    bonus = rng.integers(0, 500, len(sizes))
    out = tor.commit(path, acc, bonus, tok, off)
    assert list(np.diff(out["off"])) == list(acc + 1)
    for b in range(len(sizes)):
        rows = out["row"][out["off"][b]:out["off"][b + 1]]
        toks = out["tok"][out["off"][b]:out["off"][b + 1]]
        assert rows[0] == off[b]
        for i in range(1, len(rows)):
            assert parent[rows[i]] == rows[i - 1]
            assert toks[i - 1] == tok[rows[i]]
        assert toks[-1] == bonus[b]


ALL_TREE_CHECKS = [
    check_topk_brute_force, check_topk_ties_and_argmax, check_topk_probabilities,
    check_topk_map_and_nan, check_draft_tree_golden, check_draft_tree_chain,
    check_draft_tree_levels, check_trees_to_batch, check_tree_meta_golden,
    check_tree_meta_closure,
    check_commit_golden, check_commit_is_root_prefix,
]
