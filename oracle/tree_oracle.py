"""Float reference of the steps on either side of verification (test infrastructure only).

Draft side (Sec. 2, "Draft"; Sec. 1): the draft model runs ``nsteps`` forwards, each node of the
current frontier branches ``topk`` ways, and the tree is pruned to a verification budget of
``ndt`` tokens. The paper adopts the EAGLE-3 drafter, whose tree is grown the EAGLE-2 way: a
node's value is the product of the draft probabilities along its path, every step expands the
``topk`` most valuable nodes of the newest level, and the final tree keeps the most valuable
nodes of everything drafted. Here the value is kept in the log domain (a sum of log-probabilities),
which orders nodes identically in exact arithmetic.

Around the target forward (Sec. 2, "Verify"): the tree attention mask and position ids follow
from ``parent[]`` (a node sees itself and its ancestors; its position is the committed length plus
its depth), and after verification the accepted path is committed.

Readings of points the paper leaves open (listed with their reasons in the design notes):
  * top-k of a draft row: logits in descending order, lowest draft id on ties; a logit that is
    not a number counts as -inf; log-probabilities are taken against the row's log-sum-exp over
    the whole draft vocabulary; an optional map sends draft ids to target ids (EAGLE-3 drafts
    over a reduced vocabulary);
  * the score of a drafted node is the sum of the log-probabilities along its path (float64
    here); a log-probability that is not a number counts as -inf;
  * each step appends all frontier x topk children to the pool (frontier slot major, child rank
    minor) and takes the topk best of them as the next frontier, best first, earlier candidate
    on equal scores;
  * ``ndt`` counts the root: the kept tree is the root plus the ndt - 1 best pool nodes (earlier
    pool entry on equal scores), listed in pool order, so parents precede children;
  * the draft top-1 probability of Eq. (2) is exp of the root row's best log-probability;
  * committed tokens are the accepted drafted tokens followed by the bonus token; the rows kept
    for the next step are the root's and those of the accepted nodes.

Not fixed by the paper: the growth rule itself (scores, frontier choice, pruning) is the EAGLE-2
reading above; the paper names only its three parameters. The pins check the code against that reading
stated independently, not against numbers the paper prints.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

import numpy as np

from .asv_oracle import logits


# ----------------------------------------------------------------------------- draft top-k

def draft_topk(x64: np.ndarray, w64: np.ndarray, k: int,
               vocab_map: Optional[np.ndarray] = None) -> dict:
    """The k most probable draft tokens of every draft row and their log-probabilities.

    Sec. 2 ("Draft"): each node branches ``topk`` ways, i.e. takes the draft model's k most
    probable next tokens. z_r = W_d x_r is the draft LM head's logit row (the same contraction as
    the target's, ``logits``); ids are sorted by descending logit with the lowest draft id first
    among equal logits; logp = z - lse with lse = log sum_v exp(z_r[v]). Non-number logits count
    as -inf, and so does a non-number log-probability.

    Returns ids [R, k] (draft ids, or ``vocab_map[id]`` when a map is given), logp [R, k], lse
    [R] and ``zs`` [R, k + 1], the k + 1 largest logits of each row (to locate near-ties).
    """
    z = logits(x64, w64)
    z = np.where(np.isnan(z), -np.inf, z)
    R, V = z.shape
    assert 1 <= k <= V
    m = z.max(axis=1)
    lse = np.full(R, -np.inf)
    for r in range(R):
        if np.isfinite(m[r]):
            lse[r] = m[r] + np.log(np.exp(z[r] - m[r]).sum())
        elif m[r] == np.inf:
            lse[r] = np.inf
    order = np.argsort(-z, axis=1, kind="stable")       # stable: lower id first on ties
    ids = order[:, :k].astype(np.int64)
    top = np.take_along_axis(z, order[:, :k + 1], axis=1)
    with np.errstate(invalid="ignore"):
        logp = top[:, :k] - lse[:, None]
    logp = np.where(np.isnan(logp), -np.inf, logp)
    if vocab_map is not None:
        ids = np.asarray(vocab_map, dtype=np.int64)[ids]
    zs = np.full((R, k + 1), -np.inf)
    zs[:, :top.shape[1]] = top
    return dict(ids=ids, logp=logp, lse=lse, zs=zs)


def draft_top1_prob(root_logp: float) -> float:
    """p_draft(top1) of Eq. (2) from the root row's best log-probability."""
    return math.exp(float(root_logp))


# ----------------------------------------------------------------------------- tree growth

@dataclass
class DraftTree:
    """One request's draft tree while it grows (EAGLE-2 style dynamic tree, see module notes).

    Pool entry q holds a drafted token, the pool index of its parent (-1: the root) and its
    score. ``front`` lists the pool indices of the frontier slots, best first; before the first
    step the frontier is the root alone (index -1, score 0).
    """
    nsteps: int
    topk: int
    ndt: int
    tok: List[int] = field(default_factory=list)
    par: List[int] = field(default_factory=list)
    score: List[float] = field(default_factory=list)
    front: List[int] = field(default_factory=lambda: [-1])
    front_score: List[float] = field(default_factory=lambda: [0.0])
    steps: int = 0


def draft_tree_init(shape: Sequence[int]) -> DraftTree:
    nsteps, topk, ndt = (int(v) for v in shape)
    assert nsteps >= 1 and topk >= 1 and ndt >= 1
    return DraftTree(nsteps=nsteps, topk=topk, ndt=ndt)


def _logp(v) -> float:
    x = float(v)
    return -math.inf if math.isnan(x) else x


def draft_tree_step(t: DraftTree, ids: np.ndarray, logp: np.ndarray) -> DraftTree:
    """One draft forward's worth of growth (Sec. 2, "Draft": branch topk ways per node).

    ``ids[j]`` / ``logp[j]`` are the top-k (k >= topk) of frontier slot j's draft row, best first.
    Every frontier node gets its topk children, all of which join the pool; a child's score is
    its parent's score plus its log-probability. The topk best children become the next
    frontier. A tree that has taken its nsteps steps does not change.
    """
    if t.steps >= t.nsteps:
        return t
    cand = []                                         # (score, parent pool index, token)
    for j, f in enumerate(t.front):
        for c in range(t.topk):
            s = t.front_score[j] + _logp(logp[j][c])
            cand.append((s, f, int(ids[j][c])))
    base = len(t.tok)
    tok = t.tok + [c[2] for c in cand]
    par = t.par + [c[1] for c in cand]
    score = t.score + [c[0] for c in cand]
    best = sorted(range(len(cand)), key=lambda q: (-float(cand[q][0]), q))[:t.topk]
    return DraftTree(nsteps=t.nsteps, topk=t.topk, ndt=t.ndt, tok=tok, par=par, score=score,
                     front=[base + q for q in best], front_score=[cand[q][0] for q in best],
                     steps=t.steps + 1)


def draft_tree_prune(t: DraftTree, root_tok: int = -1) -> dict:
    """The verification tree: the root plus the ndt - 1 best pool nodes (Sec. 2: "pruning to a
    verify budget of ndt tokens").

    Nodes are kept in pool order, so every parent precedes its children and node 0 is the root.
    Returns ``parent`` (local ids, -1 at the root), ``tok`` (root_tok at the root) and ``pool``
    (the pool index of each kept node, -1 at the root).
    """
    P = len(t.tok)
    m = min(t.ndt - 1, P)
    best = sorted(range(P), key=lambda q: (-float(t.score[q]), q))[:m]
    kept = sorted(best)
    local = {-1: 0}
    for i, q in enumerate(kept):
        local[q] = i + 1
    parent = [-1] + [local[t.par[q]] for q in kept]   # a KeyError here would break closure
    tok = [root_tok] + [t.tok[q] for q in kept]
    return dict(parent=np.array(parent, dtype=np.int64), tok=np.array(tok, dtype=np.int64),
                pool=np.array([-1] + kept, dtype=np.int64))


def draft_trees_to_batch(pruned: Sequence[dict]) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Concatenate per-request trees into the batch layout of verification: global parent ids
    (-1 at each root), draft tokens and the request offsets."""
    off = [0]
    par, tok = [], []
    for p in pruned:
        lo = off[-1]
        par += [-1 if q < 0 else lo + int(q) for q in p["parent"]]
        tok += [int(v) for v in p["tok"]]
        off.append(lo + len(p["parent"]))
    return (np.array(par, dtype=np.int64), np.array(tok, dtype=np.int64),
            np.array(off, dtype=np.int64))


# ----------------------------------------------------------------------------- tree metadata

def tree_meta(parent: np.ndarray, req_offsets: np.ndarray, pos_base: np.ndarray):
    """Depth, position id and tree-attention visibility of every node (Sec. 1, Sec. 2: the
    target verifies the whole tree in one forward with tree attention).

    Node c of request b sees node j of the same request iff j is c or an ancestor of c; its
    depth is the number of parent links to the request's root and its position id is
    pos_base[b] + depth. Returns depth [N], pos [N] and a list of boolean [n_b, n_b] matrices
    ``vis`` with vis[b][c - lo, j - lo] = (c sees j).
    """
    N = len(parent)
    depth = np.zeros(N, dtype=np.int64)
    pos = np.zeros(N, dtype=np.int64)
    vis = []
    for b in range(len(req_offsets) - 1):
        lo, hi = int(req_offsets[b]), int(req_offsets[b + 1])
        v = np.zeros((hi - lo, hi - lo), dtype=bool)
        for c in range(lo, hi):
            j, d = c, 0
            v[c - lo, c - lo] = True
            while parent[j] >= 0:
                j = int(parent[j])
                v[c - lo, j - lo] = True
                d += 1
            depth[c] = d
            pos[c] = int(pos_base[b]) + d
        vis.append(v)
    return depth, pos, vis


# ----------------------------------------------------------------------------- commit

def commit(accepted_path: np.ndarray, accepted_len: np.ndarray, bonus: np.ndarray,
           draft_tok: np.ndarray, req_offsets: np.ndarray) -> dict:
    """What one verification step commits (Sec. 2, "Verify": the accepted tokens plus the target
    token at the last accepted node).

    Request b commits its accepted drafted tokens in path order followed by its bonus token;
    the tree rows that stay valid for the next step are the root's and those of the accepted
    nodes (the bonus token has no row yet). Returns ``off`` [B + 1] (prefix sums of
    accepted_len + 1), ``tok`` and ``row`` (global node ids), both [off[B]].
    """
    off, tok, row = [0], [], []
    for b in range(len(req_offsets) - 1):
        lo, n = int(req_offsets[b]), int(accepted_len[b])
        path = [int(p) for p in accepted_path[lo:lo + n]]
        row += [lo] + path
        tok += [int(draft_tok[p]) for p in path] + [int(bonus[b])]
        off.append(off[-1] + n + 1)
    return dict(off=np.array(off, dtype=np.int64), tok=np.array(tok, dtype=np.int64),
                row=np.array(row, dtype=np.int64))
