"""Shared helpers of the GPU tests: device transfer, oracle reference, banded comparison.

Bands. The parity bar puts a 1e-3 band around every floating-point decision the path takes: a row's
argmax (its top-2 gap), a node's margin (|g - M - T ln kappa|) and the walk's choice between
siblings with distinct tokens. Where the oracle's float64 values put a decision inside a band,
the GPU's float32 decision may legitimately differ. Every banded row, node and request is
recorded by id in BAND_LOG (tests/conftest.py writes it to parity_bands.json at the end of the
session) together with what the GPU did there, and callers cap how many requests
of a full-size workload may be banded.
"""

from __future__ import annotations

import dataclasses
import math
import os
from typing import List, Optional

import numpy as np

import oracle
from workloads import Workload

BAND = oracle.LN_BAND
TOL_F = 2e-3          # |max|, |lse|, |drafted logit| tolerance (bf16 inputs, fp32 accumulation)
TOL_STATE = 1e-5      # float fields of the policy state (fp32 EMA / ring mean)
# Band of the tree-shape decision (Sec. 3.3, Eq. (2)): members lo + (hi - lo) * DCS within this
# distance of a half-integer may round differently from the float32 score. The float fields
# agree within TOL_STATE, so a member moves by at most |hi - lo| * TOL_STATE (4e-5 at the
# paper's ranges).
SHAPE_BAND = 1e-4
MAX_BANDED_FRACTION = 0.1   # banded requests allowed in a full-size workload

BAND_LOG: List[dict] = []


def _test_id() -> str:
    return os.environ.get("PYTEST_CURRENT_TEST", "").split(" ")[0]


def log_bands(tag: str, **info):
    """Record banded decisions of the current test (written out at the end of the session)."""
    BAND_LOG.append(dict(test=_test_id(), tag=tag, **info))


def resolve_with_oracle(w: Workload, w64: np.ndarray) -> dict:
    """Drafted tokens from the oracle's top-8 and the full float64 reference of the step."""
    x64 = oracle.widen_bf16(w.hidden)
    top8 = np.empty((w.N, 8), dtype=np.int32)
    for r0 in range(0, w.N, 256):
        top8[r0:r0 + 256] = oracle.row_top8(oracle.logits(x64[r0:r0 + 256], w64))
    w.with_drafts(top8)
    return top8


def reference(w: Workload, w64: np.ndarray, tau=None, state=None,
              params: Optional[oracle.Params] = None) -> dict:
    tau = w.tau if tau is None else tau
    return oracle.verify(w64, w.hidden, w.draft_tok, w.parent, w.req_offsets, tau,
                         w.draft_logits, state, params or oracle.Params())


def device_inputs(w: Workload, W: np.ndarray, dev, tau=None):
    import torch

    def t(x):
        return torch.from_numpy(np.array(x, copy=True, order="C")).to(dev)

    return dict(
        hidden=t(w.hidden.view(np.int16)).view(torch.bfloat16),
        w_lm=t(W.view(np.int16)).view(torch.bfloat16),
        draft_tok=t(w.draft_tok.astype(np.int32)),
        parent=t(w.parent.astype(np.int32)),
        req_offsets=t(w.req_offsets.astype(np.int32)),
        tau=t(np.asarray(w.tau if tau is None else tau, dtype=np.float32)),
        draft_logits=None if w.draft_logits is None else t(w.draft_logits),
    )


def to_host(out) -> dict:
    return {f: (None if getattr(out, f) is None else getattr(out, f).cpu().numpy())
            for f in out._fields}


@dataclasses.dataclass
class Report:
    banded_rows: int = 0
    banded_nodes: int = 0
    banded_requests: int = 0
    clean_requests: int = 0
    requests: list = dataclasses.field(default_factory=list)    # [b, decision, node id]

    @property
    def banded_ids(self):
        return {r[0] for r in self.requests}


def compare(w: Workload, ref: dict, got: dict, rows=None, tag: str = "") -> Report:
    """Assert GPU outputs match the oracle: floats within TOL_F, integer outputs bit-exact
    except where the oracle's float64 values put a decision inside the 1e-3 bands. Banded rows,
    nodes and requests are recorded by id with the GPU's outcome there. ``rows`` restricts the
    per-row/per-node checks to a sample of row ids."""
    rep = Report()
    N = w.N
    rows = np.arange(N) if rows is None else np.asarray(rows)
    assert np.all(got["req_status"] == 0), got["req_status"]
    dm = np.abs(got["row_max"][rows] - ref["row_max"][rows])
    dl = np.abs(got["row_lse"][rows] - ref["row_lse"][rows])
    assert dm.max() < TOL_F, ("row_max", float(dm.max()), int(rows[dm.argmax()]))
    assert dl.max() < TOL_F, ("row_lse", float(dl.max()), int(rows[dl.argmax()]))
    gap = ref["row_gap"]
    clean_rows = rows[gap[rows] >= BAND]
    banded_rows = rows[gap[rows] < BAND]
    rep.banded_rows = int(len(banded_rows))
    bad = clean_rows[got["row_argmax"][clean_rows] != ref["row_argmax"][clean_rows]]
    assert len(bad) == 0, ("row_argmax", bad[:10])
    rowset = set(rows.tolist())
    nodes = np.array([c for c in range(N) if w.parent[c] >= 0 and int(w.parent[c]) in rowset],
                     dtype=np.int64)
    banded_nodes = np.zeros(0, dtype=np.int64)
    if len(nodes):
        dg = np.abs(got["drafted_logit"][nodes] - ref["drafted_logit"][nodes])
        assert dg.max() < TOL_F, ("drafted_logit", float(dg.max()), int(nodes[dg.argmax()]))
        p = w.parent[nodes]
        kappa = ref["tau_node"][nodes]
        with np.errstate(divide="ignore"):
            lnk = np.log(kappa)
        delta = ref["drafted_logit"][nodes] - ref["row_max"][p]
        lnk = lnk * ref.get("temperature", 1.0)
        in_band = (gap[p] < BAND) | ((kappa > 0) & (np.abs(delta - lnk) < BAND) &
                                     (w.draft_tok[nodes] != ref["row_argmax"][p]))
        rep.banded_nodes = int(in_band.sum())
        banded_nodes = nodes[in_band]
        clean = nodes[~in_band]
        badn = clean[got["accept"][clean].astype(bool) != ref["accept"][clean]]
        assert len(badn) == 0, ("accept", badn[:10])
    roots = w.req_offsets[:-1]
    assert np.all(got["accept"][roots] == 1)
    req_log = []
    for b in range(w.B):
        lo, hi = int(w.req_offsets[b]), int(w.req_offsets[b + 1])
        k_ref = int(ref["accepted_len"][b])
        path_ref = list(ref["accepted_path"][lo:lo + k_ref])
        k_got = int(got["accepted_len"][b])
        path_got = list(got["accepted_path"][lo:lo + k_got])
        assert np.all(got["accepted_path"][lo + k_got:hi] == -1), ("path padding", b)
        band_at = int(ref["band_at"][b])
        if band_at < 0:
            rep.clean_requests += 1
            assert k_got == k_ref and path_got == path_ref, ("walk", b, path_got, path_ref)
            assert int(got["bonus_token"][b]) == int(ref["bonus_token"][b]), ("bonus", b)
        else:
            rep.banded_requests += 1
            assert path_got[:band_at] == path_ref[:band_at], ("walk prefix", b, band_at)
            node = ([lo] + [int(v) for v in path_ref])[band_at]
            rep.requests.append([b, band_at, node])
            req_log.append(dict(request=b, decision=band_at, node=node,
                                gpu_len=k_got, oracle_len=k_ref,
                                same_walk=path_got == path_ref and int(got["bonus_token"][b]) ==
                                int(ref["bonus_token"][b])))
        # whatever the bands decide, the GPU path is a root prefix of accepted nodes
        cur = lo
        for c in path_got:
            assert w.parent[c] == cur and got["accept"][c] == 1, ("root prefix", b, c)
            cur = c
    if ref.get("draft_conf") is not None and got.get("draft_conf") is not None and \
            not np.all(np.isnan(ref["draft_conf"])):
        dc = np.abs(got["draft_conf"] - ref["draft_conf"])
        assert dc.max() < 1e-5 * max(1.0, float(np.abs(ref["draft_conf"]).max())) + 1e-6, \
            ("draft_conf", float(dc.max()))
    if len(banded_rows) or len(banded_nodes) or req_log:
        log_bands(tag, rows=[dict(row=int(r), gap=float(gap[r]),
                                  gpu_argmax=int(got["row_argmax"][r]),
                                  oracle_argmax=int(ref["row_argmax"][r]))
                             for r in banded_rows],
                  nodes=[dict(node=int(c), gpu_accept=int(got["accept"][c]),
                              oracle_accept=int(ref["accept"][c])) for c in banded_nodes],
                  requests=req_log)
    return rep


def compare_state(gpu_states, ref_states, banded_requests=(), params=None, tag: str = ""):
    """The GPU's policy state against the oracle's own state chain (Sec. 3.3): counters exact,
    floats within TOL_STATE, and the tree shape of Eq. (2) exact unless the oracle's shape
    decision lies within SHAPE_BAND of a half-integer (recorded). Requests in
    ``banded_requests`` carry a history the bands allow to differ and are skipped."""
    p = params or oracle.Params()
    shape_banded = []
    for b, (g, r) in enumerate(zip(gpu_states, ref_states)):
        if b in banded_requests:
            continue
        assert g.steps == r.steps and g.hist_count == r.hist_count, b
        assert g.hist_head == r.hist_head and g.zero_streak == r.zero_streak, b
        assert g.breaker == r.breaker, b
        assert abs(g.rar - r.rar) < TOL_STATE, (b, g.rar, r.rar)
        assert abs(g.hist_mean - r.hist_mean) < TOL_STATE, (b, g.hist_mean, r.hist_mean)
        for i in range(16):
            assert abs(g.hist[i] - r.hist[i]) < TOL_STATE, (b, i)
        assert abs(g.draft_conf - r.draft_conf) < 1e-5, (b, g.draft_conf, r.draft_conf)
        assert abs(g.dcs - r.dcs) < TOL_STATE, (b, g.dcs, r.dcs)
        slack = oracle.tree_shape_slack(r.dcs, r.breaker, p)
        if slack < SHAPE_BAND:
            shape_banded.append(dict(request=b, slack=slack, gpu=list(g.shape),
                                     oracle=list(r.shape)))
            continue
        assert tuple(g.shape) == tuple(r.shape), (b, tuple(g.shape), tuple(r.shape))
    if shape_banded:
        log_bands(tag, shape=shape_banded)
    return shape_banded


def follow_gpu_history(tag: str, ref: dict, got: dict, st_before, w, params, conf=None,
                       max_fraction: float = MAX_BANDED_FRACTION):
    """The oracle's next state for a step whose walks were banded: a banded request may accept
    another length, so its history takes the GPU's length (the oracle's update applied to it).
    Such requests are recorded and may be at most ``max_fraction`` of the batch."""
    new = list(ref["state"])
    banded = [int(b) for b in np.flatnonzero(ref["band_at"] >= 0)]
    for b in banded:
        n_b = int(w.req_offsets[b + 1] - w.req_offsets[b])
        c = None if conf is None else float(conf[b])
        new[b] = oracle.state_update(st_before[b], int(got["accepted_len"][b]), n_b, c, params)
    if banded:
        log_bands(tag, history_follows_gpu=[dict(request=b,
                                                 gpu_len=int(got["accepted_len"][b]),
                                                 oracle_len=int(ref["accepted_len"][b]))
                                            for b in banded])
    assert len(banded) <= max(1, math.floor(max_fraction * len(st_before))), (tag, banded)
    return new
