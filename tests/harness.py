"""Shared helpers of the GPU tests: device transfer, oracle reference, banded comparison."""

from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

import oracle
from workloads import Workload

BAND = oracle.LN_BAND
TOL_F = 2e-3          # |max|, |lse|, |drafted logit| tolerance (bf16 inputs, fp32 accumulation)
TOL_STATE = 1e-5      # float fields of the policy state (fp32 EMA / ring mean)


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


def compare(w: Workload, ref: dict, got: dict, rows=None) -> Report:
    """Assert GPU outputs match the oracle: floats within TOL_F, integer outputs bit-exact
    except where the oracle's float64 values put a decision inside the 1e-3 bands (reported).
    ``rows`` restricts the per-row/per-node checks to a sample of row ids."""
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
    rep.banded_rows = int(len(rows) - len(clean_rows))
    bad = clean_rows[got["row_argmax"][clean_rows] != ref["row_argmax"][clean_rows]]
    assert len(bad) == 0, ("row_argmax", bad[:10])
    rowset = set(rows.tolist())
    nodes = np.array([c for c in range(N) if w.parent[c] >= 0 and int(w.parent[c]) in rowset],
                     dtype=np.int64)
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
        clean = nodes[~in_band]
        badn = clean[got["accept"][clean].astype(bool) != ref["accept"][clean]]
        assert len(badn) == 0, ("accept", badn[:10])
    roots = w.req_offsets[:-1]
    assert np.all(got["accept"][roots] == 1)
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
    return rep


def compare_state(gpu_states, ref_states, banded_requests=(), params=None):
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
        # Eq. (2): the score within tolerance of the float64 state's; the integer shape is
        # the oracle's float32 decision taken on the library's own confidence and RAR
        assert abs(g.dcs - r.dcs) < TOL_STATE, (b, g.dcs, r.dcs)
        assert tuple(g.shape) == oracle.tree_shape(g.draft_conf, g.rar, g.breaker,
                                                   params or oracle.Params())[1], (b,)
