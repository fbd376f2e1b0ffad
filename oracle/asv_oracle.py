"""Float64 reference of the AdaptiveSpec verification path (test infrastructure only).

Notation follows the paper: for a draft-tree node c with drafted token d_c, the target
distribution that judges it is the one predicted at its parent p (the row of p's hidden state);
p_target(top1) is that row's softmax maximum and p_target(draft) the probability of d_c
(Sec. 3.2, Eq. (1)). The threshold is kappa (called ``tau`` at the library boundary).

Readings of points the paper leaves open (each one is listed with its reason in the design notes):
  * row of node c's verdict = the row of its parent (draft-then-verify in one pass, Sec. 1/2);
  * the rule is applied at every mismatch along the walk, not only the first one, unless
    ``max_promotions`` caps it (Sec. 3.2 speaks of "the first mismatch position");
  * among siblings the walk takes the child with the highest target logit, lowest node id on
    ties (reading R3: the paper does not fix the choice);
  * an exact match is always accepted (redundant in exact arithmetic: margin = 1 >= kappa);
  * kappa = 0 accepts everything; kappa must lie in [0, 1] (margin lies in [0, 1], Eq. (1));
  * argmax ties break to the lowest vocabulary id; the bonus token is the argmax of the last
    accepted node's row (greedy decoding, Sec. 4.1).
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field, replace
from typing import Dict, List, Optional

import numpy as np

# Width of the tolerance bands around floating-point decisions (margin, argmax, sibling).
LN_BAND = 1e-3

HIST_WINDOW = 16


# ----------------------------------------------------------------------------- inputs

def widen_bf16(bits: np.ndarray) -> np.ndarray:
    """bf16 raw bits -> float64, exactly (bf16 is the top half of an IEEE float32)."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def widen_weights(w_bits: np.ndarray) -> np.ndarray:
    """W[V, H] as float64 (exact), converted in slices to bound temporary memory."""
    V = w_bits.shape[0]
    out = np.empty(w_bits.shape, dtype=np.float64)
    step = 8192
    for v0 in range(0, V, step):
        out[v0:v0 + step] = widen_bf16(w_bits[v0:v0 + step])
    return out


# ----------------------------------------------------------------------------- logits

def logits(x64: np.ndarray, w64: np.ndarray) -> np.ndarray:
    """Target LM-head logits z_r[v] = sum_h W[v, h] * x_r[h] for every given row (float64).

    The verify pass of speculative decoding scores every draft-tree token in one target forward
    (Sec. 1, Sec. 2 "Verify"); the LM head is its last layer. ``x64`` is [R, H], ``w64`` [V, H].
    Products of two bf16 values are exact in float64, so z is the exact dot product up to the
    float64 rounding of the sum.
    """
    return x64 @ w64.T


def row_stats(z: np.ndarray):
    """Per row: max logit M, argmax a (lowest id among ties), log-sum-exp L and top-2 gap.

    p_target(top1) = exp(M - L) is the softmax maximum used in Eq. (1). ``gap`` (M minus the
    largest logit at any other id) is kept to locate near-ties for the tolerance bands.
    """
    z = np.atleast_2d(z)
    M = z.max(axis=1)
    a = z.argmax(axis=1)                      # first occurrence = lowest id among ties
    L = M + np.log(np.exp(z - M[:, None]).sum(axis=1))
    rest = z.copy()
    rest[np.arange(z.shape[0]), a] = -np.inf
    gap = M - rest.max(axis=1)
    return M, a.astype(np.int64), L, gap


def row_top8(z: np.ndarray) -> np.ndarray:
    """The eight highest-logit vocabulary ids of each row, best first, lowest id on ties."""
    z = np.atleast_2d(z)
    out = np.empty((z.shape[0], 8), dtype=np.int32)
    for i, row in enumerate(z):
        thr = np.partition(row, -8)[-8]
        cand = np.nonzero(row >= thr)[0]
        order = np.lexsort((cand, -row[cand]))
        out[i] = cand[order[:8]]
    return out


# ----------------------------------------------------------------------------- margin rule

def accept_flags(g: np.ndarray, M: np.ndarray, a: np.ndarray, parent: np.ndarray,
                 draft_tok: np.ndarray, tau_node: np.ndarray,
                 temperature: float = 1.0) -> np.ndarray:
    """Margin rule of Sec. 3.2, Eq. (1), for every non-root node c with parent p.

    margin(c) = p_target(d_c) / p_target(top1) = exp(g_c - M_p), which lies in (0, 1]. The node
    is promoted when margin >= kappa, i.e. g_c - M_p >= ln kappa. An exact match d_c = a_p is
    accepted outright and kappa = 0 accepts every node. Roots are marked accepted.
    With a temperature T the target distribution is softmax(z / T), so the margin is
    exp((g_c - M_p) / T) (the paper's variant at T != 1; T = 1 is Eq. (1)).
    ``M`` and ``a`` are indexed by row id; ``tau_node`` is kappa of each node's request.
    """
    acc = np.ones(len(parent), dtype=bool)
    for c in range(len(parent)):
        p = parent[c]
        if p < 0:
            continue
        kappa = float(tau_node[c])
        if draft_tok[c] == a[p] or kappa == 0.0:
            acc[c] = True
        else:
            acc[c] = (g[c] - M[p]) / temperature >= math.log(kappa)
    return acc


# ----------------------------------------------------------------------------- walk

def _children(parent: np.ndarray, lo: int, hi: int) -> Dict[int, List[int]]:
    kids: Dict[int, List[int]] = {i: [] for i in range(lo, hi)}
    for c in range(lo + 1, hi):
        kids[int(parent[c])].append(c)
    return kids


def walk(root: int, end: int, parent: np.ndarray, draft_tok: np.ndarray, g: np.ndarray,
         accept: np.ndarray, a: np.ndarray, max_promotions: int = -1):
    """Accepted path and bonus token of one request whose nodes are rows [root, end).

    Starting at the root (the last committed token), repeatedly take the child with the highest
    target logit g (lowest node id on ties) and keep it while the margin rule accepts it. A
    child whose token differs from the current row's argmax is a promotion (Sec. 3.2: the rule
    "promotes drafted tokens at the first mismatch position"); with ``max_promotions >= 0`` the
    walk stops instead of exceeding that many promotions. The bonus token is the target argmax
    at the last accepted node (greedy decoding, Sec. 4.1). The child choice and the repeated
    promotion are readings the paper does not fix (R3, R2); the pins check the walk against
    them stated independently.

    Returns (path as global node ids, accepted_len, bonus_token).
    """
    kids = _children(parent, root, end)
    cur, path, promos = root, [], 0
    while kids[cur]:
        best = kids[cur][0]
        for c in kids[cur][1:]:
            if g[c] > g[best]:
                best = c
        if not accept[best]:
            break
        if draft_tok[best] != a[cur]:
            if max_promotions >= 0 and promos >= max_promotions:
                break
            promos += 1
        path.append(best)
        cur = best
    return path, len(path), int(a[cur])


def walk_bands(root: int, end: int, parent: np.ndarray, draft_tok: np.ndarray,
               g: np.ndarray, M: np.ndarray, a: np.ndarray, gap: np.ndarray, kappa: float,
               path: List[int], band: float = LN_BAND, temperature: float = 1.0):
    """Index of the first walk decision that falls inside a tolerance band, or -1.

    Decision i (0 <= i <= len(path)) is the step taken at node path[i-1] (the root for i=0):
    the sibling choice, the accept test of the chosen child, and for the last one the bonus.
    A decision is banded when the current row's top-2 gap is below ``band`` (its argmax could
    differ at float32), when the two best children with distinct tokens are within ``band``,
    or when the chosen mismatched child's logit gap g - M is within ``band`` of T ln kappa.
    """
    kids = _children(parent, root, end)
    nodes = [root] + list(path)
    for i, cur in enumerate(nodes):
        if gap[cur] < band:
            return i
        ch = kids[cur]
        if not ch:
            continue
        best = max(ch, key=lambda c: (g[c], -c))
        others = [g[c] for c in ch if draft_tok[c] != draft_tok[best]]
        if others and g[best] - max(others) < band:
            return i
        if draft_tok[best] != a[cur] and kappa > 0.0:
            if abs((g[best] - M[cur]) - temperature * math.log(kappa)) < band:
                return i
    return -1


# ----------------------------------------------------------------------------- Eq. (2) signals

def draft_confidence(q: np.ndarray) -> float:
    """p_draft(top1) of Sec. 3.3, Eq. (2): the softmax maximum of one row of draft logits,
    1 / sum_v exp(q_v - max q)."""
    q = np.asarray(q, dtype=np.float64)
    return float(1.0 / np.exp(q - q.max()).sum())


@dataclass
class Params:
    alpha: float = 0.3          # EMA weight of the newest observation (Sec. 3.3)
    rar0: float = 1.0           # initial rolling acceptance rate (not given by the paper)
    breaker_n: int = 5          # consecutive zero-accept steps that trip the breaker (Sec. 3.3)
    max_promotions: int = -1    # -1: no cap on promotions along one walk
    temperature: float = 1.0    # T of the margin exp((z_d - z_max) / T); 1 is Eq. (1)
    dcs_divisor: float = 0.5    # d of Sec. 3.3 (d = 0.5 for every run of Sec. 4)
    shape_lo: tuple = (3, 4, 4)     # (nsteps, topk, ndt) at DCS = 0: wide and shallow
    shape_hi: tuple = (7, 1, 8)     # at DCS = 1: deep and narrow (Sec. 3.3, Table of configs)
    shape_start: tuple = (3, 4, 4)  # the starting configuration a breaker trip reverts to


@dataclass
class ReqState:
    rar: float = 1.0
    hist: List[float] = field(default_factory=lambda: [0.0] * HIST_WINDOW)
    hist_head: int = 0
    hist_count: int = 0
    zero_streak: int = 0
    breaker: int = 0
    steps: int = 0
    hist_mean: float = 1.0
    draft_conf: float = 0.0
    dcs: float = 0.0
    shape: tuple = (0, 0, 0)


def state_init(p: Params) -> ReqState:
    """Before the first step a request drafts with the starting configuration."""
    return ReqState(rar=p.rar0, hist_mean=p.rar0, shape=tuple(p.shape_start))


def state_update(s: ReqState, accepted_len: int, n_nodes: int, conf: Optional[float],
                 p: Params) -> ReqState:
    """Per-request acceptance history after one step (Sec. 3.3).

    RAR is an exponential moving average (alpha = 0.3) of the fraction of drafted tokens the
    target accepted, here x = accepted_len / (n_nodes - 1) (reading R10: the paper names
    the fraction, not its denominator). A 16-slot ring keeps the last observations and their
    mean. A request with ``breaker_n`` consecutive zero-accept steps trips the circuit breaker:
    the flag is raised and RAR, the ring and the streak restart (the reset itself is reading R13,
    not fixed by the paper). A root-only tree drafts nothing and only advances ``steps``.
    Finally the next step's tree shape is chosen from the latest draft confidence (this step's
    when draft logits were given, else the last one stored) and the updated RAR (Eq. (2),
    :func:`tree_shape`).
    """
    s = replace(s, hist=list(s.hist))
    if n_nodes > 1:
        x = accepted_len / (n_nodes - 1)
        s.rar = s.rar + p.alpha * (x - s.rar)
        s.hist[s.hist_head] = x
        s.hist_head = (s.hist_head + 1) % HIST_WINDOW
        s.hist_count = min(s.hist_count + 1, HIST_WINDOW)
        s.hist_mean = _ring_mean(s)
        s.zero_streak = s.zero_streak + 1 if accepted_len == 0 else 0
        s.breaker = 1 if s.zero_streak >= p.breaker_n else 0
        if s.breaker:
            s.rar = p.rar0
            s.hist = [0.0] * HIST_WINDOW
            s.hist_head = 0
            s.hist_count = 0
            s.hist_mean = p.rar0
            s.zero_streak = 0
    else:
        s.breaker = 0
    s.steps += 1
    if conf is not None:
        s.draft_conf = conf
    s.dcs, s.shape = tree_shape(s.draft_conf, s.rar, s.breaker, p)
    return s


def tree_shape(conf: float, rar: float, breaker: int, p: Params):
    """Draft Confidence Score and the tree shape it selects (Sec. 3.3, Eq. (2)).

    DCS = p_draft(top1) * RAR, rescaled by the divisor d so that it saturates at 1 once the
    product reaches d: DCS = min(1, p_draft(top1) * RAR / d). Each member of the triplet
    (nsteps, topk, ndt) moves linearly from ``shape_lo`` at DCS = 0 to ``shape_hi`` at DCS = 1
    (depth grows with DCS, branching with 1 - DCS), rounded to the nearest integer with halves
    going to the lower one (a reading: the paper selects among pre-captured integer triplets
    without naming the rounding; reading R23). A request whose breaker tripped reverts to
    ``shape_start`` (Sec. 3.3; which triplet is "the starting configuration" is reading R24,
    not fixed by the paper). Evaluated in float64.
    """
    dcs = min(1.0, float(conf) * float(rar) / float(p.dcs_divisor))
    if breaker:
        return dcs, tuple(int(v) for v in p.shape_start)
    shape = []
    for lo, hi in zip(p.shape_lo, p.shape_hi):
        x = lo + (hi - lo) * dcs
        shape.append(int(math.ceil(x - 0.5)))
    return dcs, tuple(shape)


def tree_shape_slack(dcs: float, breaker: int, p: Params) -> float:
    """How far the tree-shape decision of score ``dcs`` is from changing: the smallest distance
    of any member lo + (hi - lo) * dcs from a half-integer (infinite after a breaker trip, whose
    shape does not depend on the score). Used to band the integer shape where the library's
    float32 score and the float64 one may round to different integers."""
    if breaker:
        return math.inf
    out = math.inf
    for lo, hi in zip(p.shape_lo, p.shape_hi):
        x = lo + (hi - lo) * float(dcs)
        out = min(out, abs(x - math.floor(x) - 0.5))
    return out


def _ring_mean(s: ReqState) -> float:
    # Slots written so far are the hist_count slots ending just before hist_head.
    vals = [s.hist[(s.hist_head - 1 - i) % HIST_WINDOW] for i in range(s.hist_count)]
    return sum(vals) / len(vals)


# ----------------------------------------------------------------------------- full call

def verify(w64: np.ndarray, hidden_bits: np.ndarray, draft_tok: np.ndarray,
           parent: np.ndarray, req_offsets: np.ndarray, tau: np.ndarray,
           draft_logits: Optional[np.ndarray] = None,
           state: Optional[List[ReqState]] = None, params: Params = Params(),
           row_chunk: int = 256):
    """Every output of one verify call, from the definitions (float64).

    Computes the logits of all rows (in independent slices of ``row_chunk`` rows to bound
    memory), the row statistics, the drafted logits, the margin flags, each request's walk and
    bonus, the draft confidence of each request's root row and the updated history.
    """
    N = hidden_bits.shape[0]
    M = np.empty(N)
    L = np.empty(N)
    gap = np.empty(N)
    a = np.empty(N, dtype=np.int64)
    g = np.full(N, np.nan)
    x64 = widen_bf16(hidden_bits)
    for r0 in range(0, N, row_chunk):
        z = logits(x64[r0:r0 + row_chunk], w64)
        M[r0:r0 + len(z)], a[r0:r0 + len(z)], L[r0:r0 + len(z)], gap[r0:r0 + len(z)] = \
            row_stats(z)
        rows = {r0 + i: z[i] for i in range(len(z))}
        for c in range(N):
            if parent[c] in rows:
                g[c] = rows[parent[c]][draft_tok[c]]
    return finish(M, L, a, gap, g, draft_tok, parent, req_offsets, tau, draft_logits, state,
                  params)


def finish(M, L, a, gap, g, draft_tok, parent, req_offsets, tau, draft_logits=None,
           state=None, params: Params = Params()):
    """The part of :func:`verify` after the logits: flags, walks, confidence and history."""
    N = len(parent)
    B = len(req_offsets) - 1
    tau_node = np.empty(N)
    for b in range(B):
        tau_node[req_offsets[b]:req_offsets[b + 1]] = float(np.float32(tau[b]))
    acc = accept_flags(g, M, a, parent, draft_tok, tau_node, params.temperature)
    out_len = np.zeros(B, dtype=np.int64)
    bonus = np.zeros(B, dtype=np.int64)
    path_arr = np.full(N, -1, dtype=np.int64)
    band_at = np.full(B, -1, dtype=np.int64)
    conf = np.full(B, np.nan)
    new_state = None if state is None else list(state)
    for b in range(B):
        lo, hi = int(req_offsets[b]), int(req_offsets[b + 1])
        path, n_acc, bon = walk(lo, hi, parent, draft_tok, g, acc, a, params.max_promotions)
        out_len[b], bonus[b] = n_acc, bon
        path_arr[lo:lo + n_acc] = path
        band_at[b] = walk_bands(lo, hi, parent, draft_tok, g, M, a, gap,
                                float(np.float32(tau[b])), path,
                                temperature=params.temperature)
        if draft_logits is not None:
            conf[b] = draft_confidence(draft_logits[lo])
        if new_state is not None:
            new_state[b] = state_update(state[b], n_acc, hi - lo,
                                        None if draft_logits is None else conf[b], params)
    return dict(row_max=M, row_lse=L, row_argmax=a, row_gap=gap, drafted_logit=g,
                accept=acc, accepted_len=out_len, accepted_path=path_arr, bonus_token=bonus,
                band_at=band_at, draft_conf=conf, state=new_state, tau_node=tau_node,
                temperature=params.temperature)
