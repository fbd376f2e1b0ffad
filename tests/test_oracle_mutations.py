"""Plant plausible mistakes in the CPU oracle and check that the pins catch each one.

Every mutant replaces one oracle function (on the CPU, through monkeypatch) with a copy that
carries a single mistake; at least one pin must then fail.
"""

import math

import numpy as np
import pytest

import oracle.asv_oracle as orc
from oracle_pins import ALL_CHECKS


def _accept_own_row(g, M, a, parent, d, tau_node, temperature=1.0):
    acc = np.ones(len(parent), dtype=bool)
    for c in range(len(parent)):
        if parent[c] < 0:
            continue
        k = float(tau_node[c])
        acc[c] = d[c] == a[c] or k == 0.0 or (g[c] - M[c]) / temperature >= math.log(k)
    return acc


def _accept_sign(g, M, a, parent, d, tau_node, temperature=1.0):
    acc = np.ones(len(parent), dtype=bool)
    for c in range(len(parent)):
        p = parent[c]
        if p < 0:
            continue
        k = float(tau_node[c])
        acc[c] = d[c] == a[p] or k == 0.0 or (M[p] - g[c]) / temperature >= math.log(k)
    return acc


def _accept_strict_gt(g, M, a, parent, d, tau_node, temperature=1.0):
    acc = np.ones(len(parent), dtype=bool)
    for c in range(len(parent)):
        p = parent[c]
        if p < 0:
            continue
        k = float(tau_node[c])
        acc[c] = k == 0.0 or (g[c] - M[p]) / temperature > math.log(k)   # no exact-match clause
    return acc


def _accept_ignores_temperature(g, M, a, parent, d, tau_node, temperature=1.0):
    return ORIG["accept_flags"](g, M, a, parent, d, tau_node, 1.0)


def _accept_temperature_inverted(g, M, a, parent, d, tau_node, temperature=1.0):
    return ORIG["accept_flags"](g, M, a, parent, d, tau_node, 1.0 / temperature)


def _logits_transposed(x64, w64):
    return (w64 @ x64.T)


def _row_stats_last_argmax(z):
    M, a, L, gap = ORIG["row_stats"](z)
    z = np.atleast_2d(z)
    a = z.shape[1] - 1 - np.argmax(z[:, ::-1], axis=1)
    return M, a, L, gap


def _row_stats_no_shift(z):
    M, a, L, gap = ORIG["row_stats"](z)
    return M, a, np.log(np.exp(np.atleast_2d(z) - M[:, None]).sum(axis=1)), gap


def _walk_lowest_id(root, end, parent, d, g, accept, a, max_promotions=-1):
    kids = orc._children(parent, root, end)
    cur, path = root, []
    while kids[cur]:
        best = kids[cur][0]
        if not accept[best]:
            break
        path.append(best)
        cur = best
    return path, len(path), int(a[cur])


def _walk_root_bonus(root, end, parent, d, g, accept, a, max_promotions=-1):
    path, k, _ = ORIG["walk"](root, end, parent, d, g, accept, a, max_promotions)
    return path, k, int(a[root])


def _walk_ignores_accept(root, end, parent, d, g, accept, a, max_promotions=-1):
    return ORIG["walk"](root, end, parent, d, g, np.ones_like(accept), a, max_promotions)


def _conf_min(q):
    q = np.asarray(q, dtype=np.float64)
    return float(1.0 / np.exp(q - q.min()).sum())


def _update_alpha_swapped(s, acc_len, n, conf, p):
    q = orc.Params(alpha=1.0 - p.alpha, rar0=p.rar0, breaker_n=p.breaker_n,
                   max_promotions=p.max_promotions)
    return ORIG["state_update"](s, acc_len, n, conf, q)


def _update_breaker_early(s, acc_len, n, conf, p):
    q = orc.Params(alpha=p.alpha, rar0=p.rar0, breaker_n=p.breaker_n - 1,
                   max_promotions=p.max_promotions)
    return ORIG["state_update"](s, acc_len, n, conf, q)


def _update_counts_depth(s, acc_len, n, conf, p):
    # observation = accepted / all nodes (root included) instead of drafted nodes
    return ORIG["state_update"](s, acc_len, n + 1 if n > 1 else n, conf, p)


def _shape_uses_ring_mean(s, acc_len, n, conf, p):
    s = ORIG["state_update"](s, acc_len, n, conf, p)
    s.dcs, s.shape = orc.tree_shape(s.draft_conf, s.hist_mean, s.breaker, p)
    return s


def _shape_halves_up(conf, rar, breaker, p):
    dcs = min(1.0, conf * rar / p.dcs_divisor)
    if breaker:
        return dcs, tuple(p.shape_start)
    return dcs, tuple(int(math.floor(lo + (hi - lo) * dcs + 0.5))
                      for lo, hi in zip(p.shape_lo, p.shape_hi))


def _shape_ends_swapped(conf, rar, breaker, p):
    return ORIG["tree_shape"](conf, rar, breaker,
                              orc.Params(shape_lo=p.shape_hi, shape_hi=p.shape_lo,
                                         shape_start=p.shape_start,
                                         dcs_divisor=p.dcs_divisor))


def _shape_no_saturation(conf, rar, breaker, p):
    dcs = conf * rar / p.dcs_divisor
    if breaker:
        return dcs, tuple(p.shape_start)
    return dcs, tuple(int(math.ceil(lo + (hi - lo) * dcs - 0.5))
                      for lo, hi in zip(p.shape_lo, p.shape_hi))


def _slack_from_integers(dcs, breaker, p):
    # distance to the nearest integer instead of the nearest half-integer
    if breaker:
        return math.inf
    return min(abs(x - round(x)) for x in (lo + (hi - lo) * dcs
                                           for lo, hi in zip(p.shape_lo, p.shape_hi)))


def _bands_always_first(root, end, parent, d, g, M, a, gap, kappa, path, band=1e-3,
                        temperature=1.0):
    return 0


def _bands_never(root, end, parent, d, g, M, a, gap, kappa, path, band=1e-3, temperature=1.0):
    return -1


def _bands_off_by_one(root, end, parent, d, g, M, a, gap, kappa, path, band=1e-3,
                      temperature=1.0):
    i = ORIG["walk_bands"](root, end, parent, d, g, M, a, gap, kappa, path, band, temperature)
    return i + 1 if i >= 0 else -1


def _bands_no_sibling_check(root, end, parent, d, g, M, a, gap, kappa, path, band=1e-3,
                            temperature=1.0):
    kids = orc._children(parent, root, end)
    for i, cur in enumerate([root] + list(path)):
        if gap[cur] < band:
            return i
        if not kids[cur]:
            continue
        best = max(kids[cur], key=lambda c: (g[c], -c))
        if d[best] != a[cur] and kappa > 0.0:
            if abs((g[best] - M[cur]) - temperature * math.log(kappa)) < band:
                return i
    return -1


def _bands_ignore_temperature(root, end, parent, d, g, M, a, gap, kappa, path, band=1e-3,
                              temperature=1.0):
    return ORIG["walk_bands"](root, end, parent, d, g, M, a, gap, kappa, path, band, 1.0)


def _widen_truncating(bits):
    return np.asarray(bits, dtype=np.uint16).astype(np.float64)


ORIG = {name: getattr(orc, name) for name in
        ("row_stats", "walk", "state_update", "accept_flags", "logits", "tree_shape",
         "walk_bands")}

MUTANTS = {
    "accept_uses_own_row": ("accept_flags", _accept_own_row),
    "accept_sign_flipped": ("accept_flags", _accept_sign),
    "accept_drops_exact_match": ("accept_flags", _accept_strict_gt),
    "accept_ignores_temperature": ("accept_flags", _accept_ignores_temperature),
    "accept_temperature_inverted": ("accept_flags", _accept_temperature_inverted),
    "logits_transposed": ("logits", _logits_transposed),
    "argmax_last_occurrence": ("row_stats", _row_stats_last_argmax),
    "lse_drops_max_term": ("row_stats", _row_stats_no_shift),
    "walk_takes_lowest_id": ("walk", _walk_lowest_id),
    "walk_bonus_from_root": ("walk", _walk_root_bonus),
    "walk_ignores_accept": ("walk", _walk_ignores_accept),
    "conf_uses_min": ("draft_confidence", _conf_min),
    "ema_alpha_swapped": ("state_update", _update_alpha_swapped),
    "breaker_one_early": ("state_update", _update_breaker_early),
    "observation_counts_root": ("state_update", _update_counts_depth),
    "widen_as_integer": ("widen_bf16", _widen_truncating),
    "shape_from_ring_mean": ("state_update", _shape_uses_ring_mean),
    "shape_halves_up": ("tree_shape", _shape_halves_up),
    "shape_ends_swapped": ("tree_shape", _shape_ends_swapped),
    "shape_not_saturated": ("tree_shape", _shape_no_saturation),
    "shape_slack_to_integers": ("tree_shape_slack", _slack_from_integers),
    "bands_always_first_decision": ("walk_bands", _bands_always_first),
    "bands_never": ("walk_bands", _bands_never),
    "bands_off_by_one": ("walk_bands", _bands_off_by_one),
    "bands_without_sibling_check": ("walk_bands", _bands_no_sibling_check),
    "bands_ignore_temperature": ("walk_bands", _bands_ignore_temperature),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, monkeypatch):
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(orc, attr, fn)
    failures = 0
    for check in ALL_CHECKS:
        try:
            check(orc)
        except (AssertionError, ValueError, IndexError):
            failures += 1
    assert failures > 0, f"no pin caught the planted mistake {name}"
