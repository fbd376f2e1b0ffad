"""Write the tolerance-band lists of the full-size synthetic configurations (run on the CPU).

The bands of the parity comparison are decided on the oracle's float64 values alone: a row
whose top-2 logit gap is below 1e-3, a node whose margin g - M lies within 1e-3 of T ln kappa
(or whose parent row is such a row), a request whose walk crosses such a decision or a sibling
choice between distinct tokens within 1e-3, and (configuration 2, whose policy state runs over
32 steps) a request whose tree-shape decision lies within 1e-4 of a half-integer. This script
lists every such row, node and request by id, from the oracle tables of make_oracle_tables.py
and the seeded trees; it calls only the oracle.

    python tests/golden/make_band_lists.py
"""

from __future__ import annotations

import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from oracle.asv_oracle import finish  # noqa: E402
from workloads import CONFIGS, make_trees, make_workload  # noqa: E402

OUT = os.path.join(HERE, "band_lists.json")
SHAPE_BAND = 1e-4


def load_table(cfg: int) -> dict:
    with np.load(os.path.join(HERE, f"oracle_cfg{cfg}.npz"), allow_pickle=False) as t:
        return {k: t[k] for k in t.files}


def walk_bands(tab: dict, step: int, off, parent, tau: float, draft_logits=None, state=None,
               params=oracle.Params()):
    """Banded rows, nodes and requests of one verify call, from the oracle table's values."""
    s = f"_s{step}"
    tok = tab["draft_tok" + s].astype(np.int64)
    B = len(off) - 1
    taus = np.full(B, tau, dtype=np.float32)
    ref = finish(tab["row_max" + s], tab["row_lse" + s], tab["row_argmax" + s].astype(np.int64),
                 tab["row_gap" + s], tab["drafted_logit" + s], tok, parent, off, taus,
                 draft_logits, state, params)
    gap = ref["row_gap"]
    rows = np.flatnonzero(gap < oracle.LN_BAND)
    kappa = float(np.float32(tau))
    nodes = []
    for c in range(len(parent)):
        p = int(parent[c])
        if p < 0:
            continue
        if gap[p] < oracle.LN_BAND:
            nodes.append(c)
        elif kappa > 0 and tok[c] != ref["row_argmax"][p]:
            delta = ref["drafted_logit"][c] - ref["row_max"][p]
            if abs(delta - params.temperature * np.log(kappa)) < oracle.LN_BAND:
                nodes.append(c)
    requests = []
    for b in range(B):
        at = int(ref["band_at"][b])
        if at >= 0:
            lo = int(off[b])
            path = [lo] + [int(v) for v in ref["accepted_path"][lo:lo + ref["accepted_len"][b]]]
            requests.append([b, at, path[at]])
    return dict(rows=[int(r) for r in rows], nodes=nodes, requests=requests,
                n_rows=int(len(parent)), n_requests=B), ref


def make() -> dict:
    out = {}
    for cfg in (1, 3, 4):
        tab = load_table(cfg)
        off, parent, _ = make_trees(cfg, 0)
        for tau in CONFIGS[cfg]["taus"]:
            out[f"cfg{cfg}_tau{tau}"], _ = walk_bands(tab, 0, off, parent, tau)
    tab = load_table(2)
    p = oracle.Params()
    state = [oracle.state_init(p) for _ in range(CONFIGS[2]["B"])]
    for step in range(int(tab["steps"])):
        w = make_workload(2, step)
        bands, ref = walk_bands(tab, step, w.req_offsets, w.parent, CONFIGS[2]["taus"][0],
                                w.draft_logits, state, p)
        state = ref["state"]
        bands["shape"] = [[b, float(oracle.tree_shape_slack(st.dcs, st.breaker, p))]
                          for b, st in enumerate(state)
                          if oracle.tree_shape_slack(st.dcs, st.breaker, p) < SHAPE_BAND]
        bands["shapes"] = [list(st.shape) for st in state]
        out[f"cfg2_step{step}"] = bands
        print(f"cfg2 step {step}: {len(bands['requests'])} banded requests", flush=True)
    return out


if __name__ == "__main__":
    lists = make()
    with open(OUT, "w") as f:
        json.dump(lists, f, indent=0, sort_keys=True)
    for k, v in lists.items():
        print(k, {f: len(v[f]) for f in ("rows", "nodes", "requests")})
    print(f"wrote {OUT}")
