"""Plant plausible mistakes in the draft-tree, tree-metadata and commit oracle and check that the
pins of ``tree_pins.py`` catch each one (CPU only, through monkeypatch)."""

import numpy as np
import pytest

import oracle.tree_oracle as tor
from tree_pins import ALL_TREE_CHECKS

ORIG = {name: getattr(tor, name) for name in
        ("draft_topk", "draft_tree_step", "draft_tree_prune", "tree_meta", "commit",
         "draft_trees_to_batch")}


def _topk_highest_id_on_ties(x64, w64, k, vocab_map=None):
    out = ORIG["draft_topk"](x64, w64, k, vocab_map)
    z = x64 @ w64.T
    V = z.shape[1]
    order = V - 1 - np.argsort(-z[:, ::-1], axis=1, kind="stable")
    ids = order[:, :k]
    out["ids"] = ids if vocab_map is None else np.asarray(vocab_map)[ids]
    return out


def _topk_logp_against_max(x64, w64, k, vocab_map=None):
    out = ORIG["draft_topk"](x64, w64, k, vocab_map)
    out["logp"] = out["logp"] - out["logp"][:, :1]
    return out


def _topk_map_before_ranking(x64, w64, k, vocab_map=None):
    out = ORIG["draft_topk"](x64, w64, k, None)
    return out                                    # the map is forgotten


def _step_own_logp_only(t, ids, logp):
    zero = tor.DraftTree(nsteps=t.nsteps, topk=t.topk, ndt=t.ndt, tok=t.tok, par=t.par,
                         score=t.score, front=t.front,
                         front_score=[0.0] * len(t.front), steps=t.steps)
    return ORIG["draft_tree_step"](zero, ids, logp)


def _step_frontier_first_candidates(t, ids, logp):
    out = ORIG["draft_tree_step"](t, ids, logp)
    if out is t:
        return out
    base = len(t.tok)
    out.front = [base + q for q in range(t.topk)]
    out.front_score = [out.score[q] for q in out.front]
    return out


def _step_keeps_frontier_only(t, ids, logp):
    out = ORIG["draft_tree_step"](t, ids, logp)
    if out is t:
        return out
    base = len(t.tok)
    keep = set(out.front)
    idx = list(range(base)) + [q for q in range(base, len(out.tok)) if q in keep]
    remap = {q: i for i, q in enumerate(idx)}
    remap[-1] = -1
    out.tok = [out.tok[q] for q in idx]
    out.par = [out.par[q] for q in idx]
    out.score = [out.score[q] for q in idx]
    out.front = [remap[q] for q in out.front]
    return out


def _prune_keeps_ndt(t, root_tok=-1):
    bigger = tor.DraftTree(nsteps=t.nsteps, topk=t.topk, ndt=t.ndt + 1, tok=t.tok, par=t.par,
                           score=t.score, front=t.front, front_score=t.front_score,
                           steps=t.steps)
    return ORIG["draft_tree_prune"](bigger, root_tok)


def _prune_score_order(t, root_tok=-1):
    P = len(t.tok)
    m = min(t.ndt - 1, P)
    best = sorted(range(P), key=lambda q: (-float(t.score[q]), q))[:m]
    local = {-1: 0}
    for i, q in enumerate(best):
        local[q] = i + 1
    parent = [-1] + [local.get(t.par[q], 0) for q in best]
    return dict(parent=np.array(parent), tok=np.array([root_tok] + [t.tok[q] for q in best]),
                pool=np.array([-1] + best))


def _meta_excludes_self(parent, req_offsets, pos_base):
    depth, pos, vis = ORIG["tree_meta"](parent, req_offsets, pos_base)
    for v in vis:
        np.fill_diagonal(v, False)
    return depth, pos, vis


def _meta_depth_counts_self(parent, req_offsets, pos_base):
    depth, pos, vis = ORIG["tree_meta"](parent, req_offsets, pos_base)
    return depth + 1, pos + 1, vis


def _commit_without_bonus(path, acc, bonus, tok, off):
    out = ORIG["commit"](path, acc, bonus, tok, off)
    keep = np.ones(len(out["tok"]), dtype=bool)
    keep[out["off"][1:] - 1] = False
    out["tok"] = out["tok"][keep]
    return out


def _commit_drops_root_row(path, acc, bonus, tok, off):
    out = ORIG["commit"](path, acc, bonus, tok, off)
    keep = np.ones(len(out["row"]), dtype=bool)
    keep[out["off"][:-1]] = False
    out["row"] = np.concatenate([out["row"][keep], [-1] * int((~keep).sum())])
    return out


def _batch_local_parents(pruned):
    par, tok, off = ORIG["draft_trees_to_batch"](pruned)
    lo = np.repeat(off[:-1], np.diff(off))
    return np.where(par >= 0, par - lo, -1), tok, off      # parents left request-local


def _batch_offsets_shifted(pruned):
    par, tok, off = ORIG["draft_trees_to_batch"](pruned)
    return par, tok, np.concatenate([off[1:], [off[-1]]])  # offsets one request late


MUTANTS = {
    "topk_highest_id_on_ties": ("draft_topk", _topk_highest_id_on_ties),
    "topk_logp_against_max": ("draft_topk", _topk_logp_against_max),
    "topk_forgets_map": ("draft_topk", _topk_map_before_ranking),
    "step_drops_parent_score": ("draft_tree_step", _step_own_logp_only),
    "step_frontier_first_candidates": ("draft_tree_step", _step_frontier_first_candidates),
    "step_pools_frontier_only": ("draft_tree_step", _step_keeps_frontier_only),
    "prune_keeps_ndt_nodes": ("draft_tree_prune", _prune_keeps_ndt),
    "prune_lists_by_score": ("draft_tree_prune", _prune_score_order),
    "meta_excludes_self": ("tree_meta", _meta_excludes_self),
    "meta_depth_counts_self": ("tree_meta", _meta_depth_counts_self),
    "commit_without_bonus": ("commit", _commit_without_bonus),
    "commit_drops_root_row": ("commit", _commit_drops_root_row),
    "batch_parents_left_local": ("draft_trees_to_batch", _batch_local_parents),
    "batch_offsets_shifted": ("draft_trees_to_batch", _batch_offsets_shifted),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_tree_mutant_is_caught(name, monkeypatch):
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(tor, attr, fn)
    failures = 0
    for check in ALL_TREE_CHECKS:
        try:
            check(tor)
        except (AssertionError, ValueError, IndexError, KeyError):
            failures += 1
    assert failures > 0, f"no pin caught the planted mistake {name}"
