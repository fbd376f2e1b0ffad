"""Checks that pin the CPU oracle to the paper and to mathematics, not to itself.

Each ``check_*`` takes the oracle module (or a stand-in with the same functions) and raises
AssertionError on a mismatch. ``test_oracle_pins.py`` runs them against the real oracle, and
``test_oracle_mutations.py`` runs them against deliberately broken copies to show that a
plausible mistake (wrong row, sign, index, transposed operand, dropped term) is caught.
"""

from __future__ import annotations

import math
from fractions import Fraction

import numpy as np
from scipy.special import logsumexp, softmax


def _bf16_values(rng, shape, std):
    """Random bf16-representable float64 values (truncate float32 bits, exact in float64)."""
    x = (rng.standard_normal(shape) * std).astype(np.float32)
    b = (x.view(np.uint32) & np.uint32(0xFFFF0000)).view(np.float32)
    return b.astype(np.float64), (x.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


# ----------------------------------------------------------------------------- widening

def check_widen(orc):
    bits = np.array([0x3F80, 0xC000, 0x3F81, 0x0001, 0x7F7F, 0x8000, 0x4049], dtype=np.uint16)
    want = [1.0, -2.0, 1.0 + 2.0 ** -7, 2.0 ** -133, (2 - 2.0 ** -7) * 2.0 ** 127, -0.0,
            3.140625]
    got = orc.widen_bf16(bits)
    assert got.dtype == np.float64
    for g, w in zip(got, want):
        assert g == w, (g, w)
    assert math.copysign(1.0, got[5]) == -1.0


# ----------------------------------------------------------------------------- logits

def check_logits_exact(orc):
    """Oracle logits against exact rational dot products (brute force, tiny shapes)."""
    rng = np.random.default_rng(11)
    R, V, H = 3, 13, 7
    xv, xb = _bf16_values(rng, (R, H), 1.0)
    wv, wb = _bf16_values(rng, (V, H), 0.5)
    z = orc.logits(orc.widen_bf16(xb), orc.widen_weights(wb))
    assert z.shape == (R, V)
    for r in range(R):
        for v in range(V):
            exact = sum(Fraction(float(wv[v, h])) * Fraction(float(xv[r, h])) for h in range(H))
            assert abs(z[r, v] - float(exact)) <= 1e-15 * max(1.0, abs(float(exact))), (r, v)


# ----------------------------------------------------------------------------- row stats

def check_row_stats(orc):
    # z_v = ln(v + 1): M = ln n, a = n - 1, L = ln(n (n + 1) / 2), gap = ln n - ln(n - 1).
    n = 50
    z = np.log(np.arange(1, n + 1, dtype=np.float64))[None, :]
    M, a, L, gap = orc.row_stats(z)
    assert abs(M[0] - math.log(n)) < 1e-15
    assert a[0] == n - 1
    assert abs(L[0] - math.log(n * (n + 1) / 2)) < 1e-13
    assert abs(gap[0] - (math.log(n) - math.log(n - 1))) < 1e-13
    # All equal: L = c + ln V, lowest id wins, gap 0.
    V, c = 37, -1.25
    M, a, L, gap = orc.row_stats(np.full((1, V), c))
    assert M[0] == c and a[0] == 0 and gap[0] == 0.0
    assert abs(L[0] - (c + math.log(V))) < 1e-13
    # Ties below the max do not move the argmax; a tie at the max picks the lowest id.
    row = np.array([[0.5, 2.0, -1.0, 2.0, 1.9]])
    M, a, L, gap = orc.row_stats(row)
    assert a[0] == 1 and gap[0] == 0.0
    # Random rows against the library log-sum-exp and a Python-loop max/argmax.
    rng = np.random.default_rng(5)
    z = rng.standard_normal((6, 301)) * 3.0
    M, a, L, gap = orc.row_stats(z)
    for r in range(6):
        best, arg = -math.inf, -1
        for v in range(z.shape[1]):
            if z[r, v] > best:
                best, arg = z[r, v], v
        second = max(z[r, v] for v in range(z.shape[1]) if v != arg)
        assert M[r] == best and a[r] == arg
        assert abs(gap[r] - (best - second)) < 1e-15
        assert abs(L[r] - logsumexp(z[r])) < 1e-12
        assert M[r] <= L[r] <= M[r] + math.log(z.shape[1])


def check_top8(orc):
    rng = np.random.default_rng(9)
    z = rng.standard_normal((4, 200))
    z[2, 17] = z[2, 40] = z[2].max() + 1.0      # exact tie at the top: 17 before 40
    t = orc.row_top8(z)
    for r in range(4):
        want = sorted(range(200), key=lambda v: (-z[r, v], v))[:8]
        assert list(t[r]) == want, (r, list(t[r]), want)


# ----------------------------------------------------------------------------- margin rule

def _random_rows_tree(rng, n_nodes, V):
    parent = np.array([-1] + [int(rng.integers(0, c)) for c in range(1, n_nodes)])
    return parent


def check_margin_is_probability_ratio(orc):
    """Eq. (1): margin = p_target(draft) / p_target(top1), promote iff margin >= kappa.

    Probabilities come from the library softmax of the *parent's* row; the test uses rows that
    differ strongly so that judging a node by its own row (or by any other row) fails.
    """
    rng = np.random.default_rng(21)
    N, V = 40, 23
    z = rng.standard_normal((N, V)) * 2.0
    parent = _random_rows_tree(rng, N, V)
    d = rng.integers(0, V, size=N)
    d[0] = -1
    M, a, L, gap = orc.row_stats(z)
    g = np.array([np.nan] + [z[parent[c], d[c]] for c in range(1, N)])
    probs = softmax(z, axis=1)
    checked = 0
    for kappa in (0.05, 0.1, 0.2, 0.3, 0.5, 0.9, 1.0):
        acc = orc.accept_flags(g, M, a, parent, d, np.full(N, kappa))
        assert acc[0]
        for c in range(1, N):
            p = parent[c]
            margin = probs[p, d[c]] / probs[p].max()
            assert 0.0 < margin <= 1.0 + 1e-12
            if abs(margin - kappa) < 1e-9:
                continue
            assert acc[c] == (margin >= kappa), (kappa, c, margin)
            checked += 1
    assert checked > 200
    # kappa = 0 promotes every node (ln 0 = -inf).
    assert orc.accept_flags(g, M, a, parent, d, np.zeros(N)).all()


def check_margin_with_temperature(orc):
    """The temperature variant: the target distribution is softmax(z / T), so a node passes iff
    p_T(draft) / p_T(top1) >= kappa; T = 1 is Eq. (1), a large T accepts more, a small T fewer."""
    rng = np.random.default_rng(23)
    N, V = 40, 23
    z = rng.standard_normal((N, V)) * 2.0
    parent = _random_rows_tree(rng, N, V)
    d = rng.integers(0, V, size=N)
    d[0] = -1
    M, a, L, gap = orc.row_stats(z)
    g = np.array([np.nan] + [z[parent[c], d[c]] for c in range(1, N)])
    checked = 0
    for T in (0.25, 0.7, 1.0, 2.0, 5.0):
        probs = softmax(z / T, axis=1)
        for kappa in (0.05, 0.2, 0.5, 0.9):
            acc = orc.accept_flags(g, M, a, parent, d, np.full(N, kappa), T)
            for c in range(1, N):
                p = parent[c]
                margin = probs[p, d[c]] / probs[p].max()
                if abs(margin - kappa) < 1e-9:
                    continue
                want = d[c] == a[p] or margin >= kappa
                assert acc[c] == want, (T, kappa, c)
                checked += 1
    assert checked > 500
    base = orc.accept_flags(g, M, a, parent, d, np.full(N, 0.3), 1.0)
    hot = orc.accept_flags(g, M, a, parent, d, np.full(N, 0.3), 3.0)
    cold = orc.accept_flags(g, M, a, parent, d, np.full(N, 0.3), 0.3)
    assert (hot >= base).all() and (cold <= base).all() and hot.sum() > base.sum() > cold.sum()


def check_exact_match_always_accepted(orc):
    # d_c is the parent's argmax: accepted for every kappa in [0, 1], including kappa = 1.
    rng = np.random.default_rng(3)
    N, V = 12, 31
    z = rng.standard_normal((N, V))
    parent = _random_rows_tree(rng, N, V)
    M, a, L, gap = orc.row_stats(z)
    d = np.array([-1] + [int(a[parent[c]]) for c in range(1, N)])
    g = np.array([np.nan] + [z[parent[c], d[c]] for c in range(1, N)])
    for kappa in (0.0, 0.5, 1.0):
        assert orc.accept_flags(g, M, a, parent, d, np.full(N, kappa)).all()


# ----------------------------------------------------------------------------- walk

def _tree_and_logits(rng, n, V, branch_max=3, depth_max=6, distinct_siblings=True):
    parent, depth, kids = [-1], [0], [0]
    while len(parent) < n:
        open_nodes = [i for i in range(len(parent)) if depth[i] < depth_max and
                      kids[i] < branch_max]
        p = int(open_nodes[rng.integers(len(open_nodes))])
        parent.append(p)
        depth.append(depth[p] + 1)
        kids.append(0)
        kids[p] += 1
    parent = np.array(parent)
    z = rng.standard_normal((n, V)) * 1.5
    a = z.argmax(axis=1)
    d = np.full(n, -1)
    for c in range(1, n):
        p = parent[c]
        used = {d[s] for s in range(1, c) if parent[s] == p} if distinct_siblings else set()
        while True:
            u = rng.random()
            if u < 0.55:
                tok = int(a[p])
            elif u < 0.85:
                tok = int(np.argsort(-z[p])[rng.integers(1, 4)])
            else:
                tok = int(rng.integers(V))
            if tok not in used:
                break
        d[c] = tok
    return parent, z, d


def _greedy_by_paths(parent, z, d):
    """Textbook greedy tree verification by enumerating every root-to-leaf path: the longest
    prefix whose every token equals the argmax of the previous node's row."""
    n = len(parent)
    kids = {i: [c for c in range(1, n) if parent[c] == i] for i in range(n)}
    paths, stack = [], [[0]]
    while stack:
        p = stack.pop()
        if not kids[p[-1]]:
            paths.append(p)
        for c in kids[p[-1]]:
            stack.append(p + [c])
    best_len, best_end = 0, 0
    for p in paths:
        k = 0
        while k + 1 < len(p) and d[p[k + 1]] == int(np.argmax(z[p[k]])):
            k += 1
        if k > best_len:
            best_len, best_end = k, p[k]
    return best_len, int(np.argmax(z[best_end]))


def _walk_with_oracle(orc, parent, z, d, kappa, max_promotions=-1):
    n = len(parent)
    M, a, L, gap = orc.row_stats(z)
    g = np.array([np.nan] + [z[parent[c], d[c]] for c in range(1, n)])
    acc = orc.accept_flags(g, M, a, parent, d, np.full(n, kappa))
    path, k, bonus = orc.walk(0, n, parent, d, g, acc, a, max_promotions)
    return path, k, bonus, acc


def check_kappa_one_is_strict(orc):
    """kappa = 1 reduces the margin rule to strict token-match greedy verification (Sec. 3.2:
    lossless decoding accepts only exact matches)."""
    rng = np.random.default_rng(31)
    for trial in range(60):
        parent, z, d = _tree_and_logits(rng, int(rng.integers(2, 16)), 17)
        path, k, bonus, _ = _walk_with_oracle(orc, parent, z, d, 1.0)
        want_len, want_bonus = _greedy_by_paths(parent, z, d)
        assert (k, bonus) == (want_len, want_bonus), (trial, k, bonus, want_len, want_bonus)


def check_kappa_zero_reaches_leaf(orc):
    rng = np.random.default_rng(41)
    for trial in range(40):
        n = int(rng.integers(2, 20))
        parent, z, d = _tree_and_logits(rng, n, 19)
        path, k, bonus, acc = _walk_with_oracle(orc, parent, z, d, 0.0)
        assert acc.all()
        last = path[-1] if path else 0
        assert not any(parent[c] == last for c in range(1, n)), "walk must end at a leaf"
        depth = 0
        node = last
        while node != 0:
            node = parent[node]
            depth += 1
        assert k == depth and bonus == int(np.argmax(z[last]))


def check_walk_properties(orc):
    """For any kappa the accepted path is a root prefix whose every step takes the sibling with
    the largest target probability and satisfies Eq. (1); the walk stops at a leaf or at a best
    child that fails the rule; the bonus is the argmax of the last node's row."""
    rng = np.random.default_rng(51)
    for trial in range(80):
        n = int(rng.integers(2, 24))
        parent, z, d = _tree_and_logits(rng, n, 13, distinct_siblings=False)
        kappa = float(rng.choice([0.05, 0.1, 0.2, 0.3, 0.6, 1.0]))
        path, k, bonus, acc = _walk_with_oracle(orc, parent, z, d, kappa)
        probs = softmax(z, axis=1)
        assert k == len(path)
        cur = 0
        for c in path:
            assert parent[c] == cur, "not a root prefix"
            sib = [s for s in range(1, n) if parent[s] == cur]
            best = min(sib, key=lambda s: (-probs[cur, d[s]], s))
            assert c == best
            assert probs[cur, d[c]] / probs[cur].max() >= kappa - 1e-12
            cur = c
        sib = [s for s in range(1, n) if parent[s] == cur]
        if sib:
            best = min(sib, key=lambda s: (-probs[cur, d[s]], s))
            margin = probs[cur, d[best]] / probs[cur].max()
            assert margin < kappa + 1e-12 and d[best] != int(np.argmax(z[cur]))
        assert bonus == int(np.argmax(z[cur]))


def check_len_monotone_in_kappa(orc):
    rng = np.random.default_rng(61)
    for trial in range(40):
        parent, z, d = _tree_and_logits(rng, int(rng.integers(2, 20)), 11)
        lens = [_walk_with_oracle(orc, parent, z, d, kp)[1]
                for kp in (0.0, 0.05, 0.1, 0.3, 0.6, 1.0)]
        assert all(x >= y for x, y in zip(lens, lens[1:])), lens


def check_promotion_cap(orc):
    """With at most one promotion the path holds at most one mismatched token; with none it is
    strict verification."""
    rng = np.random.default_rng(71)
    for trial in range(40):
        parent, z, d = _tree_and_logits(rng, int(rng.integers(2, 16)), 9)
        path, k, bonus, _ = _walk_with_oracle(orc, parent, z, d, 0.05, max_promotions=1)
        mism = sum(1 for c in path if d[c] != int(np.argmax(z[parent[c]])))
        assert mism <= 1
        path0, k0, b0, _ = _walk_with_oracle(orc, parent, z, d, 0.05, max_promotions=0)
        assert (k0, b0) == _greedy_by_paths(parent, z, d)


def _band_enumeration(parent, z, d, path, kappa, T, band):
    """The quantities behind every decision of a walk, computed by brute force: at each node of
    [root] + path, the row's top-2 logit gap (second largest over all other ids, Python
    loops), the gap between the best child's logit and the best logit among children whose
    token differs from it, and, when the best child's token is not the row argmax and
    kappa > 0, |g - M - T ln kappa|. Returns (the first decision index with any of them below
    ``band``, which one it was), or (-1, None)."""
    n = len(parent)
    nodes = [0] + list(path)
    for i, cur in enumerate(nodes):
        row = [float(v) for v in z[cur]]
        top, arg = -math.inf, -1
        for v, x in enumerate(row):
            if x > top:
                top, arg = x, v
        second = max(x for v, x in enumerate(row) if v != arg)
        quantities = [(top - second, "row")]
        kids = [c for c in range(1, n) if parent[c] == cur]
        if kids:
            gs = {c: row[d[c]] for c in kids}
            best = kids[0]
            for c in kids:
                if gs[c] > gs[best]:
                    best = c
            rivals = [gs[c] for c in kids if d[c] != d[best]]
            if rivals:
                quantities.append((gs[best] - max(rivals), "sibling"))
            if d[best] != arg and kappa > 0.0:
                quantities.append((abs(gs[best] - top - T * math.log(kappa)), "margin"))
        for q, kind in quantities:
            if q < band:
                return i, kind
    return -1, None


def check_walk_bands(orc):
    """The band finder against a brute-force enumeration of what each walk decision hangs on:
    row top-2 gaps, sibling gaps between distinct tokens and the margin's distance to T ln
    kappa, on trees with planted near-ties (inside and outside 1e-3) and planted near-threshold
    margins, at several kappa and temperatures."""
    rng = np.random.default_rng(97)
    band = 1e-3
    hits = {"none": 0, "root": 0, "deeper": 0, "row": 0, "sibling": 0, "margin": 0}
    for trial in range(400):
        n = int(rng.integers(2, 14))
        parent, z, d = _tree_and_logits(rng, n, 12, distinct_siblings=False)
        kappa = float(rng.choice([0.0, 0.05, 0.3, 1.0]))
        T = float(rng.choice([1.0, 0.5, 2.0]))
        z = z.copy()
        for cur in range(n):
            kids = [c for c in range(1, n) if parent[c] == cur]
            u = float(rng.choice([0.0, 4e-4, 8e-4, 1.5e-3, 3e-3]))
            kind = rng.choice(["row", "sibling", "margin", "margin"])
            best = max(kids, key=lambda c: (z[cur, d[c]], -c)) if kids else None
            if kind == "row" and rng.random() < 0.5:        # a near-tie at the top of the row
                a = int(np.argmax(z[cur]))
                other = (a + 1 + int(rng.integers(11))) % 12
                z[cur, other] = z[cur, a] - u
            elif kind == "sibling" and len(kids) >= 2:      # a rival sibling just below
                # distinct tokens other than the row argmax, so the row's own gap stays wide
                a = int(np.argmax(z[cur]))
                toks = rng.permutation([v for v in range(12) if v != a])[:len(kids)]
                for c, v in zip(kids, toks):
                    d[c] = int(v)
                best = max(kids, key=lambda c: (z[cur, d[c]], -c))
                c2 = [c for c in kids if c != best][int(rng.integers(len(kids) - 1))]
                z[cur, d[c2]] = z[cur, d[best]] - max(u, 1e-4)
            elif kind == "margin" and best is not None and kappa > 0.0:
                # the best child's margin next to the threshold, its token made a mismatch
                # (another child may then be the best)
                a = int(np.argmax(z[cur]))
                if d[best] == a:
                    d[best] = int((a + 1 + rng.integers(11)) % 12)
                target = z[cur].max() + T * math.log(kappa) + float(rng.choice([-1, 1])) * u
                if target < z[cur].max():
                    z[cur, d[best]] = target
        M, a, L, gap = orc.row_stats(z)
        g = np.array([np.nan] + [z[parent[c], d[c]] for c in range(1, n)])
        acc = orc.accept_flags(g, M, a, parent, d, np.full(n, kappa), T)
        path, k, bonus = orc.walk(0, n, parent, d, g, acc, a)
        got = orc.walk_bands(0, n, parent, d, g, M, a, gap, kappa, path, band, T)
        want, why = _band_enumeration(parent, z, d, path, kappa, T, band)
        assert got == want, (trial, got, want, why, path, kappa, T)
        hits["none" if want < 0 else ("root" if want == 0 else "deeper")] += 1
        if why:
            hits[why] += 1
    # the planted cases put decisions on both sides of the band, at the root and deeper, and
    # each of the three quantities decides some of them
    assert min(hits.values()) >= 20, hits


# ----------------------------------------------------------------------------- Eq. (2) signals

def check_draft_confidence(orc):
    V = 1000
    assert abs(orc.draft_confidence(np.full(V, 0.7)) - 1.0 / V) < 1e-15
    q = np.zeros(V)
    q[3] = 50.0
    assert abs(orc.draft_confidence(q) - 1.0 / (1.0 + (V - 1) * math.exp(-50.0))) < 1e-15
    rng = np.random.default_rng(2)
    for _ in range(5):
        q = rng.standard_normal(V) * 2.0
        c = orc.draft_confidence(q)
        assert abs(c - softmax(q).max()) < 1e-14
        assert 1.0 / V <= c <= 1.0


def check_ema_closed_form(orc):
    """RAR is an EMA with alpha = 0.3 (Sec. 3.3): a constant observation x gives
    r_k = x + (1 - alpha)^k (r_0 - x)."""
    p = orc.Params()
    s = orc.state_init(p)
    n_nodes, acc_len = 9, 3          # x = 3/8
    x = acc_len / (n_nodes - 1)
    for k in range(1, 40):
        s = orc.state_update(s, acc_len, n_nodes, None, p)
        want = x + (1.0 - p.alpha) ** k * (p.rar0 - x)
        assert abs(s.rar - want) < 1e-12, (k, s.rar, want)
        assert s.steps == k
    assert abs(p.alpha - 0.3) < 1e-15 and p.breaker_n == 5


def check_ring_mean(orc):
    p = orc.Params()
    s = orc.state_init(p)
    rng = np.random.default_rng(8)
    seen = []
    for k in range(45):
        n = int(rng.integers(2, 12))
        ln = int(rng.integers(1, n))
        s = orc.state_update(s, ln, n, None, p)
        seen.append(ln / (n - 1))
        window = seen[-16:]
        assert s.hist_count == len(window)
        assert abs(s.hist_mean - sum(window) / len(window)) < 1e-12


def check_breaker(orc):
    """Five consecutive zero-accept steps trip the circuit breaker (Sec. 3.3)."""
    p = orc.Params()
    s = orc.state_init(p)
    s = orc.state_update(s, 2, 5, None, p)
    for k in range(4):
        s = orc.state_update(s, 0, 5, None, p)
        assert s.breaker == 0 and s.zero_streak == k + 1
    s = orc.state_update(s, 1, 1 + 1, None, p)          # an accept resets the streak
    assert s.zero_streak == 0 and s.breaker == 0
    for k in range(5):
        s = orc.state_update(s, 0, 1, None, p)          # root-only trees draft nothing
        assert s.zero_streak == 0 and s.breaker == 0
    for k in range(5):
        s = orc.state_update(s, 0, 4, None, p)
        assert s.breaker == (1 if k == 4 else 0), k
    assert s.rar == p.rar0 and s.hist_count == 0 and s.zero_streak == 0
    s = orc.state_update(s, 0, 4, None, p)
    assert s.breaker == 0 and s.zero_streak == 1


def _shape_by_fractions(conf, rar, d, lo, hi):
    """Eq. (2) mapping in exact rationals of the inputs: DCS = min(1, conf * rar / d), each
    member lo + (hi - lo) * DCS, nearest integer with halves down."""
    f = lambda v: Fraction(float(v))
    dcs = min(Fraction(1), f(conf) * f(rar) / f(d))
    out = []
    for a, b in zip(lo, hi):
        x = a + (b - a) * dcs
        n = math.floor(x)
        out.append(n if x - n <= Fraction(1, 2) else n + 1)
    return dcs, tuple(out)


def check_tree_shape(orc):
    """Sec. 3.3, Eq. (2): DCS = min(1, p_draft(top1) * RAR / d); depth and node count grow
    linearly with DCS, branching with 1 - DCS, over (3,4,4) <-> (7,1,8); the breaker returns
    the starting configuration."""
    p = orc.Params()
    assert p.dcs_divisor == 0.5 and tuple(p.shape_lo) == (3, 4, 4) and tuple(p.shape_hi) == (7, 1, 8)
    # the two ends and saturation at p_draft * RAR >= d
    assert orc.tree_shape(0.0, 1.0, 0, p) == (0.0, (3, 4, 4))
    for conf, rar in ((0.5, 1.0), (1.0, 0.5), (0.9, 0.9), (1.0, 1.0)):
        dcs, shape = orc.tree_shape(conf, rar, 0, p)
        assert dcs == 1.0 and shape == (7, 1, 8), (conf, rar, shape)
    # the lattice DCS = k/8 (exact in float32) hits every half-way point of the three ranges
    for k in range(9):
        conf = k / 8 * 0.5
        dcs, shape = orc.tree_shape(conf, 1.0, 0, p)
        want_dcs, want = _shape_by_fractions(conf, 1.0, 0.5, (3, 4, 4), (7, 1, 8))
        assert dcs == float(want_dcs) == k / 8 and shape == want, (k, shape, want)
    assert orc.tree_shape(0.25, 1.0, 0, p)[1] == (5, 2, 6)      # topk 2.5 -> 2
    # random points against the rational formula, and monotonicity along the score
    rng = np.random.default_rng(21)
    prev = None
    for prod in sorted(rng.uniform(0.0, 0.6, 200)):
        conf, rar = float(prod), 1.0
        dcs, shape = orc.tree_shape(conf, rar, 0, p)
        want_dcs, want = _shape_by_fractions(conf, rar, 0.5, (3, 4, 4), (7, 1, 8))
        assert shape == want and abs(dcs - float(want_dcs)) < 1e-15, (conf, shape, want)
        # the slack is the distance of the nearest member to a half-integer
        slack = min(abs(float(a + (b - a) * want_dcs) % 1.0 - 0.5)
                    for a, b in zip((3, 4, 4), (7, 1, 8)))
        assert abs(orc.tree_shape_slack(dcs, 0, p) - slack) < 1e-12
        if prev is not None:
            assert shape[0] >= prev[0] and shape[2] >= prev[2] and shape[1] <= prev[1]
        prev = shape
    # a smaller divisor saturates sooner; the breaker reverts to the starting configuration
    q = orc.Params(dcs_divisor=0.25)
    assert orc.tree_shape(0.25, 1.0, 0, q)[1] == (7, 1, 8)
    assert orc.tree_shape(0.9, 0.9, 1, p)[1] == tuple(p.shape_start)
    assert orc.tree_shape_slack(0.3, 1, p) == math.inf
    assert orc.tree_shape_slack(0.125, 0, p) == 0.0           # 3.5, 3.625, 4.5: two halves
    assert abs(orc.tree_shape_slack(0.1, 0, p) - 0.1) < 1e-12  # 3.4, 3.7, 4.4
    # the state update picks the shape from the latest confidence and the updated RAR
    s = orc.state_init(p)
    s = orc.state_update(s, 2, 9, 0.4, p)
    assert s.shape == orc.tree_shape(0.4, s.rar, 0, p)[1] and s.draft_conf == 0.4
    s = orc.state_update(s, 0, 9, None, p)                # no new confidence: keep the last
    assert s.shape == orc.tree_shape(0.4, s.rar, 0, p)[1]


def check_verify_end_to_end(orc):
    """The composed call against brute force on a tiny batch: exact rational logits, a
    Python-loop max / argmax, the library log-sum-exp and softmax, the walk properties of
    Eq. (1) and the confidence of Eq. (2)."""
    rng = np.random.default_rng(77)
    H, V = 6, 11
    trees = [[-1, 0, 0, 1, 1, 2], [-1], [-1, 0, 1, 2], [-1, 0, 0, 0, 3, 3, 4]]
    off = np.cumsum([0] + [len(t) for t in trees])
    N = int(off[-1])
    parent = np.concatenate([[p + off[b] if p >= 0 else -1 for p in t]
                             for b, t in enumerate(trees)]).astype(np.int64)
    xv, xb = _bf16_values(rng, (N, H), 1.0)
    wv, wb = _bf16_values(rng, (V, H), 0.7)
    z = np.array([[float(sum(Fraction(float(wv[v, h])) * Fraction(float(xv[r, h]))
                             for h in range(H))) for v in range(V)] for r in range(N)])
    d = np.array([-1 if parent[c] < 0 else
                  (int(np.argmax(z[parent[c]])) if rng.random() < 0.5 else int(rng.integers(V)))
                  for c in range(N)])
    tau = np.array([0.3, 0.3, 1.0, 0.05], dtype=np.float32)
    q = rng.standard_normal((N, V)) * 2.0
    p = orc.Params()
    st = [orc.state_init(p) for _ in trees]
    out = orc.verify(orc.widen_weights(wb), xb, d, parent, off, tau, q, st, p)
    probs = softmax(z, axis=1)
    for r in range(N):
        assert abs(out["row_max"][r] - z[r].max()) < 1e-14
        assert out["row_argmax"][r] == min(v for v in range(V) if z[r, v] == z[r].max())
        assert abs(out["row_lse"][r] - logsumexp(z[r])) < 1e-12
    for c in range(N):
        if parent[c] >= 0:
            assert abs(out["drafted_logit"][c] - z[parent[c], d[c]]) < 1e-14
    for b, t in enumerate(trees):
        lo, hi = int(off[b]), int(off[b + 1])
        k = int(out["accepted_len"][b])
        path = list(out["accepted_path"][lo:lo + k])
        assert all(x == -1 for x in out["accepted_path"][lo + k:hi])
        cur = lo
        for c in path:
            assert parent[c] == cur
            sib = [s for s in range(lo + 1, hi) if parent[s] == cur]
            assert c == min(sib, key=lambda s: (-probs[cur, d[s]], s))
            assert probs[cur, d[c]] / probs[cur].max() >= float(tau[b]) - 1e-12
            cur = c
        assert out["bonus_token"][b] == int(np.argmax(z[cur]))
        assert abs(out["draft_conf"][b] - softmax(q[lo]).max()) < 1e-14
        s = out["state"][b]
        assert s.steps == 1
        if hi - lo > 1:
            assert abs(s.rar - (p.rar0 + p.alpha * (k / (hi - lo - 1) - p.rar0))) < 1e-12


ALL_CHECKS = [
    check_widen, check_logits_exact, check_row_stats, check_top8,
    check_margin_is_probability_ratio, check_margin_with_temperature,
    check_exact_match_always_accepted,
    check_kappa_one_is_strict, check_kappa_zero_reaches_leaf, check_walk_properties,
    check_len_monotone_in_kappa, check_promotion_cap, check_walk_bands, check_draft_confidence,
    check_ema_closed_form, check_ring_mean, check_breaker, check_tree_shape,
    check_verify_end_to_end,
]
