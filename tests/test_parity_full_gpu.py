"""GPU parity at the full synthetic sizes, in the launch configuration bench.py times.

The float64 oracle values for these sizes (every row's max / argmax / log-sum-exp / top-2 gap
and every node's drafted logit) come from tests/golden/make_oracle_tables.py, which calls only
the oracle. Flags, walks, bonus tokens, draft confidence and the policy state are recomputed
here by the oracle from those values; a sample of rows is recomputed live by the oracle from
the raw inputs and compared with both the table and the GPU.
"""

import hashlib
import json
import os

import numpy as np
import pytest

import oracle
from oracle.asv_oracle import finish
from harness import MAX_BANDED_FRACTION, TOL_F, compare, compare_state, device_inputs, to_host
from workloads import CONFIGS, make_workload

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
_W64 = {}
_WSHA = {}


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


def _sha(a):
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()


def _table(cfg):
    path = os.path.join(GOLDEN, f"oracle_cfg{cfg}.npz")
    with np.load(path, allow_pickle=False) as t:
        return {k: t[k] for k in t.files}


def _workload(cfg, step, tab):
    w = make_workload(cfg, step)
    s = f"_s{step}"
    assert tab["sha_hidden" + s] == _sha(w.hidden)
    assert tab["sha_parent" + s] == _sha(w.parent)
    assert tab["sha_offsets" + s] == _sha(w.req_offsets)
    assert tab["sha_choice" + s] == _sha(np.concatenate([w.kind.astype(np.int32), w.rank,
                                                        w.uid]))
    W = w.weights()
    key = (w.V, w.H)
    if key not in _WSHA:
        _WSHA[key] = _sha(W)
    assert tab["sha_w"] == _WSHA[key], "seeded weights differ from the tables' inputs"
    w.draft_tok = tab["draft_tok" + s].astype(np.int32)
    return w, W


def _ref(w, tab, step, tau=None, state=None, params=oracle.Params()):
    s = f"_s{step}"
    return finish(tab["row_max" + s], tab["row_lse" + s], tab["row_argmax" + s].astype(np.int64),
                  tab["row_gap" + s], tab["drafted_logit" + s], w.draft_tok, w.parent,
                  w.req_offsets, w.tau if tau is None else tau, w.draft_logits, state, params)


def _gpu(asv, w, W, dev, tau=None, state=None, packed=False):
    import torch
    d = device_inputs(w, W, dev, tau)
    w_lm = asv.pack_lm_head(d["w_lm"]) if packed else d["w_lm"]
    o = asv.verify(d["hidden"], w_lm, d["draft_tok"], d["parent"], d["req_offsets"],
                   d["tau"], d["draft_logits"], state=state)
    torch.cuda.synchronize()
    return to_host(o)


def _live_rows(w, W, rows):
    """The oracle from raw inputs for a few rows: (M, a, L, logits)."""
    key = (w.V, w.H)
    if key not in _W64:
        _W64.clear()
        _W64[key] = oracle.widen_weights(W)
    z = oracle.logits(oracle.widen_bf16(w.hidden[rows]), _W64[key])
    M, a, L, gap = oracle.row_stats(z)
    return M, a, L, z


def _report(name, rep, B):
    print(f"[full] {name}: clean requests {rep.clean_requests}, banded requests "
          f"{rep.requests} (request, decision, node), banded rows {rep.banded_rows}, banded "
          f"nodes {rep.banded_nodes}", flush=True)
    assert rep.banded_requests <= MAX_BANDED_FRACTION * B, (name, rep.requests)


def _band_list(key):
    with open(os.path.join(GOLDEN, "band_lists.json")) as f:
        return json.load(f)[key]


@pytest.mark.parametrize("tau", [0.1, 0.3])
def test_full_llama_b1(asv, dev, tau):
    tab = _table(1)
    w, W = _workload(1, 0, tab)
    taus = np.full(w.B, tau, dtype=np.float32)
    got = _gpu(asv, w, W, dev, taus)
    rep = compare(w, _ref(w, tab, 0, taus), got, tag=f"cfg1 tau={tau}")
    _report(f"cfg1 tau={tau}", rep, w.B)
    assert rep.requests == _band_list(f"cfg1_tau{tau}")["requests"]


def test_full_compute_b32x64(asv, dev):
    tab = _table(3)
    w, W = _workload(3, 0, tab)
    got = _gpu(asv, w, W, dev)
    rep = compare(w, _ref(w, tab, 0), got, tag="cfg3")
    _report("cfg3", rep, w.B)
    assert rep.requests == _band_list("cfg3_tau0.3")["requests"]


@pytest.mark.parametrize("tau", [0.05, 0.1, 0.3, 1.0])
def test_full_sweep_b64(asv, dev, tau):
    tab = _table(4)
    w, W = _workload(4, 0, tab)
    taus = np.full(w.B, tau, dtype=np.float32)
    got = _gpu(asv, w, W, dev, taus)
    rep = compare(w, _ref(w, tab, 0, taus), got, tag=f"cfg4 tau={tau}")
    _report(f"cfg4 tau={tau}", rep, w.B)
    assert rep.requests == _band_list(f"cfg4_tau{tau}")["requests"]


def test_full_qwen_b8_32_steps(asv, dev):
    """Adaptive trees with draft logits over 32 steps: the window-16 history wraps twice. The
    GPU's policy state is compared with the oracle's own state chain (its own walks, its own
    float64 confidence and score) after every step. After step 16 the state bytes are copied
    to the host and into a fresh device tensor, and the remaining steps run on both states:
    the resumed run must give the uninterrupted run's outputs and state bit for bit (the
    per-request state of Sec. 3.3 is plain bytes that a serving engine may checkpoint)."""
    import torch
    tab = _table(2)
    p = oracle.Params()
    st_ref = None
    st_gpu = asv.state_init(CONFIGS[2]["B"], asv.make_params(), device=dev)
    st_resumed = None
    banded = set()
    banded_steps = 0
    steps = int(tab["steps"])
    for step in range(steps):
        w, W = _workload(2, step, tab)
        if st_ref is None:
            st_ref = [oracle.state_init(p) for _ in range(w.B)]
        ref = _ref(w, tab, step, state=st_ref, params=p)
        got = _gpu(asv, w, W, dev, state=st_gpu)
        rep = compare(w, ref, got, tag=f"cfg2 step={step}")
        assert rep.requests == _band_list(f"cfg2_step{step}")["requests"], step
        banded_steps += rep.banded_requests
        banded |= rep.banded_ids
        st_ref = ref["state"]
        # a request whose walk was ever banded may legitimately carry a different history
        compare_state(asv.state_fields(st_gpu), st_ref, banded_requests=banded, params=p,
                      tag=f"cfg2 step={step}")
        if st_resumed is not None:
            again = _gpu(asv, w, W, dev, state=st_resumed)
            for k, v in got.items():
                if v is not None:
                    sel = w.parent >= 0 if k == "drafted_logit" else slice(None)
                    assert np.array_equal(again[k][sel], v[sel], equal_nan=True), (step, k)
            assert torch.equal(st_resumed, st_gpu), step
        if step == steps // 2 - 1:
            # checkpoint: the state's bytes through host memory into a fresh device tensor
            saved = st_gpu.cpu().numpy().tobytes()
            st_resumed = torch.from_numpy(
                np.frombuffer(saved, dtype=np.uint8).reshape(w.B, -1).copy()).to(dev)
        print(f"[full] cfg2 step {step}: N={w.N} len={list(got['accepted_len'])} "
              f"banded={rep.requests}", flush=True)
    assert st_resumed is not None
    assert banded_steps <= MAX_BANDED_FRACTION * steps * CONFIGS[2]["B"], banded_steps


@pytest.mark.parametrize("cfg", [1, 3, 4, 2])
def test_full_live_sample(asv, dev, cfg):
    """Rows recomputed from the raw inputs by the oracle agree with the table and the GPU."""
    tab = _table(cfg)
    w, W = _workload(cfg, 0, tab)
    got = _gpu(asv, w, W, dev)
    rng = np.random.default_rng(cfg)
    rows = np.unique(np.concatenate([w.req_offsets[:-1][:3], rng.choice(w.N, 5, replace=False)]))
    M, a, L, z = _live_rows(w, W, rows)
    assert np.allclose(M, tab["row_max_s0"][rows], atol=1e-9)
    assert np.allclose(L, tab["row_lse_s0"][rows], atol=1e-9)
    assert np.all(a == tab["row_argmax_s0"][rows])
    assert np.all(np.abs(got["row_max"][rows] - M) < TOL_F)
    assert np.all(np.abs(got["row_lse"][rows] - L) < TOL_F)
    for i, r in enumerate(rows):
        kids = np.nonzero(w.parent == r)[0]
        for c in kids:
            assert abs(z[i, w.draft_tok[c]] - tab["drafted_logit_s0"][c]) < 1e-9
            assert abs(got["drafted_logit"][c] - z[i, w.draft_tok[c]]) < TOL_F


@pytest.mark.parametrize("cfg,tau", [(1, None), (3, None), (2, None), (4, 0.05), (4, 0.1),
                                     (4, 0.3), (4, 1.0)])
def test_full_packed_weight(asv, dev, cfg, tau):
    """The packed LM-head weight at full size, as bench.py times it: parity with the oracle's
    tables, and every output bit for bit equal to the row-major weight's."""
    tab = _table(cfg)
    w, W = _workload(cfg, 0, tab)
    taus = None if tau is None else np.full(w.B, tau, dtype=np.float32)
    got = _gpu(asv, w, W, dev, taus, packed=True)
    rep = compare(w, _ref(w, tab, 0, taus), got, tag=f"cfg{cfg} tau={tau} packed")
    _report(f"cfg{cfg} tau={tau} packed weight", rep, w.B)
    base = _gpu(asv, w, W, dev, taus)
    nonroot = w.parent >= 0                 # drafted_logit is unspecified at roots
    for k, v in base.items():
        if v is not None:
            sel = nonroot if k == "drafted_logit" else slice(None)
            assert np.array_equal(got[k][sel], v[sel], equal_nan=True), k
