"""Cost-aware pruning (oracle, fp64) -- Sec. IV-B, steps 1-4, using the
layer cost of Sec. IV-A.

Test infrastructure only; see the package docstring.

Cost model (Sec. IV-A): each expert e placed on device d costs R(e,d)*C(e,d);
the layer cost is the maximum over devices of the summed cost of its active
experts.  Here the product R*C is one non-negative number per expert,
``cost[e]`` (0 for an expert that is already resident), and devices are
``n_bins`` bins given by ``bins[e]`` (None: one bin).

Three mandatory rules, selected by ``rule``:
  * "max": I(e) is the largest normalised gate weight that any token of the
    batch gives e, and A_must = {e : I(e) >= tau}.  Sec. IV-B leaves I(e)
    open; this reading makes "no expert whose gate weight reaches the
    threshold is pruned" hold token by token.
  * "sum": I(e) = sum over tokens of G(t)_e, the definition of the
    on-device experiments (Sec. V-C), and A_must = {e : I(e) >= tau}.  The
    sum runs over tokens in ascending order.
  * "cir": the retention rule of the offloading experiments (Sec. V-B):
    each token keeps its minimal number m* of top experts (by gate weight)
    whose cumulative importance ratio CIR(m) = sum_{i<=m} G_i / sum_{j<=k} G_j
    reaches tau (theta_imp); A_must is the union over tokens.  The ratio is
    formed from the router scores s (G is s normalised), added in gate order.
    Candidates are visited by their largest gate weight.

Readings taken where the paper is silent or inconsistent:
  * the candidate set is the activated experts that are not mandatory (the
    text writes the complement in all experts, but the final set must lie in
    the activated set);
  * step 1 is taken as written: A_must holds only the experts the rule makes
    mandatory.  The one case the paper leaves undefined is an empty A_trans
    (no mandatory expert and no candidate the expansion can keep for free):
    the final top-k of Sec. IV-C would then have nothing to choose from.
    Only then, steps 1-4 run again with every token's own top expert (largest
    G, lower index on ties) made mandatory.  ``keep_top1=True`` makes those
    top experts mandatory in every call (a stricter variant, not the paper's
    step 1);
  * expansion visits candidates by importance, highest first, ties to the
    lower index, and keeps F_base fixed at its step-2 value while bin loads
    grow; "does not increase above F_base" is tested as load + cost <= F_base.
Bin sums are float64 additions in a fixed order: ascending expert index for
the step-2 loads, visiting order for the expansion.
"""
from __future__ import annotations

import numpy as np


def importance_max(orig_ids: np.ndarray, g: np.ndarray, E: int):
    """A_act = union of the tokens' K_t; I(e) = max over tokens t with
    e in K_t of G(t)_e (0 for inactive experts).  Also returns each token's
    top expert (largest G, ties to the lower index)."""
    act = np.zeros(E, dtype=bool)
    imp = np.zeros(E, dtype=np.float64)
    top1 = []
    for t in range(orig_ids.shape[0]):
        best_e, best_g = None, None
        for e, gv in zip(orig_ids[t].tolist(), g[t].tolist()):
            act[e] = True
            imp[e] = max(imp[e], gv)
            if best_g is None or gv > best_g or (gv == best_g and e < best_e):
                best_e, best_g = e, gv
        top1.append(best_e)
    return act, imp, top1


def importance_sum(orig_ids: np.ndarray, g: np.ndarray, E: int) -> np.ndarray:
    """I(e) = sum over tokens t (ascending) with e in K_t of G(t)_e."""
    imp = np.zeros(E, dtype=np.float64)
    for t in range(orig_ids.shape[0]):
        for e, gv in zip(orig_ids[t].tolist(), g[t].tolist()):
            imp[e] = imp[e] + gv
    return imp


def cir_mandatory(orig_ids: np.ndarray, s: np.ndarray, theta_imp: float, E: int) -> np.ndarray:
    """Per token: experts of K_t in gate order (score descending, lower index
    first on ties); keep the shortest prefix whose cumulative ratio
    (prefix sum of s) / (sum of s over K_t) reaches theta_imp."""
    must = np.zeros(E, dtype=bool)
    for t in range(orig_ids.shape[0]):
        order = sorted(orig_ids[t].tolist(), key=lambda e: (-float(s[t, e]), e))
        total = 0.0
        for e in order:
            total += float(s[t, e])
        cum = 0.0
        for e in order:
            cum += float(s[t, e])
            must[e] = True
            if cum / total >= float(theta_imp):
                break
    return must


def mandatory_split(act: np.ndarray, imp: np.ndarray, tau: float, forced=(), extra=None):
    """Step 1: A_must = {e in A_act : I(e) >= tau}, plus the experts listed
    in ``forced`` and the mask ``extra``; A_cand = A_act minus A_must.
    Pass tau = inf to skip the threshold."""
    must = act & (imp >= float(tau))
    for e in forced:
        must[e] = True
    if extra is not None:
        must |= extra
    cand = act & ~must
    return must, cand


def bin_loads(member: np.ndarray, cost: np.ndarray, bins, n_bins: int) -> np.ndarray:
    """Per-bin load: sum over e in ``member`` placed in bin b of cost[e],
    added in ascending e (float64)."""
    loads = np.zeros(n_bins, dtype=np.float64)
    for e in range(member.shape[0]):
        if member[e]:
            b = 0 if bins is None else int(bins[e])
            loads[b] = loads[b] + float(cost[e])
    return loads


def cost_aware_greedy(must: np.ndarray, cand: np.ndarray, imp: np.ndarray,
                      cost: np.ndarray, bins, n_bins: int):
    """Steps 2-4.  F_base = max_b load_b(A_must).  Each candidate, in
    (importance desc, index asc) order, is promoted iff the load of its bin
    plus its cost stays <= F_base; the bin load then grows by its cost.
    Returns (trans, promoted, must_loads, final_loads, F_base, order)."""
    must_loads = bin_loads(must, cost, bins, n_bins)
    f_base = float(must_loads.max()) if n_bins > 0 else 0.0
    loads = must_loads.copy()
    order = sorted(np.flatnonzero(cand).tolist(), key=lambda e: (-float(imp[e]), e))
    promoted = np.zeros_like(must)
    for e in order:
        b = 0 if bins is None else int(bins[e])
        if loads[b] + float(cost[e]) <= f_base:
            promoted[e] = True
            loads[b] = loads[b] + float(cost[e])
    trans = must | promoted
    return trans, promoted, must_loads, loads, f_base, order


def prune_batch(orig_ids: np.ndarray, g: np.ndarray, E: int, tau: float,
                cost: np.ndarray, bins, n_bins: int, rule: str = "max", s=None,
                keep_top1: bool = False) -> dict:
    """Steps 1-4 for a routed batch under mandatory ``rule`` ("max", "sum"
    or "cir"; "cir" needs the router scores ``s`` [T][E]).  Returns every set
    as a bool[E] mask plus the loads, F_base and ``fallback`` (True when
    A_trans came out empty and the steps were rerun with each token's top
    expert mandatory)."""
    act, imp, top1 = importance_max(orig_ids, g, E)
    if rule == "max":
        thr, extra = tau, None
    elif rule == "sum":
        imp = importance_sum(orig_ids, g, E)
        thr, extra = tau, None
    elif rule == "cir":
        thr, extra = float("inf"), cir_mandatory(orig_ids, s, tau, E)
    else:
        raise ValueError(rule)
    must, cand = mandatory_split(act, imp, thr, top1 if keep_top1 else (), extra)
    trans, promoted, must_loads, final_loads, f_base, order = cost_aware_greedy(
        must, cand, imp, cost, bins, n_bins)
    fallback = bool(act.any() and not trans.any())
    if fallback:
        must, cand = mandatory_split(act, imp, thr, top1, extra)
        trans, promoted, must_loads, final_loads, f_base, order = cost_aware_greedy(
            must, cand, imp, cost, bins, n_bins)
    return dict(act=act, imp=imp, top1=top1, must=must, cand=cand,
                promoted=promoted, trans=trans, pruned=act & ~trans,
                act_loads=bin_loads(act, cost, bins, n_bins),
                must_loads=must_loads, trans_loads=final_loads,
                f_base=f_base, cand_order=order, fallback=fallback)
