"""Pins for the oracle's cost-aware pruning (Sec. IV-B): a hand-computed
example, the paper's literal expansion test re-evaluated from scratch,
invariants and special cases."""
import math

import numpy as np
import pytest

from oracle import cost_aware_greedy, mandatory_split, prune_batch, route_batch


def _mask(E, ids):
    m = np.zeros(E, dtype=bool)
    m[list(ids)] = True
    return m


def test_hand_example(golden):
    g = golden("greedy_hand_example.json")
    E = g["E"]
    act = _mask(E, g["act"])
    imp = np.array(g["importance"])
    cost = np.array(g["cost"], dtype=np.float32)
    bins = np.array(g["bins"], dtype=np.int32)
    must, cand = mandatory_split(act, imp, g["tau"], [])
    assert np.flatnonzero(must).tolist() == g["expected_must"]
    trans, promoted, must_loads, loads, f_base, order = cost_aware_greedy(
        must, cand, imp, cost, bins, g["n_bins"])
    assert must_loads.tolist() == g["expected_must_loads"]
    assert f_base == g["expected_f_base"]
    assert order == g["expected_order"]
    assert np.flatnonzero(promoted).tolist() == g["expected_promoted"]
    assert np.flatnonzero(trans).tolist() == g["expected_trans"]
    assert np.flatnonzero(act & ~trans).tolist() == g["expected_pruned"]
    assert loads.tolist() == g["expected_final_loads"]
    trans1, *_ = cost_aware_greedy(must, cand, imp, cost, None, 1)
    assert np.flatnonzero(trans1).tolist() == g["expected_trans_one_bin"]


def _literal_expansion(must, cand, imp, cost, bins, n_bins):
    """The expansion test as the paper writes it, recomputed from the sets
    each time with exact sums: promote e iff max over devices of the summed
    cost of (A_must + {e}) on that device equals F_base."""
    def f_cost(members):
        per = [[] for _ in range(n_bins)]
        for e in np.flatnonzero(members):
            per[0 if bins is None else bins[e]].append(float(cost[e]))
        return max(math.fsum(p) for p in per)
    cur = must.copy()
    f_base = f_cost(cur)
    for e in sorted(np.flatnonzero(cand), key=lambda e: (-imp[e], e)):
        trial = cur.copy()
        trial[e] = True
        if f_cost(trial) == f_base:
            cur = trial
    return cur, f_base


def _random_batch(rng, T, E, G, tg, k):
    logits = rng.standard_normal((T, E)).astype(np.float32)
    return route_batch(logits, None, G, tg, k)


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("n_bins", [1, 2, 4])
def test_literal_form_and_invariants(seed, n_bins):
    rng = np.random.default_rng(seed)
    E = 16
    s, keys, ids, g = _random_batch(rng, 12, E, 4, 2, 4)
    # integer costs: every sum is exact, so the literal form is unambiguous
    cost = rng.integers(0, 9, E).astype(np.float32)
    bins = None if n_bins == 1 else (np.arange(E) // (E // n_bins)).astype(np.int32)
    tau = [0.0, 0.15, 0.2, 0.3][seed % 4]
    pr = prune_batch(ids, g, E, tau, cost, bins, n_bins)
    lit, f_base = _literal_expansion(pr["must"], pr["cand"], pr["imp"], cost, bins, n_bins)
    assert np.array_equal(lit, pr["trans"])
    assert f_base == pr["f_base"]
    act, must, trans = pr["act"], pr["must"], pr["trans"]
    assert np.all(must <= trans) and np.all(trans <= act)
    assert pr["trans_loads"].max() == pr["f_base"]
    for e in np.flatnonzero(pr["pruned"]):
        b = 0 if bins is None else bins[e]
        assert pr["trans_loads"][b] + cost[e] > pr["f_base"]
    # no expert whose gate weight reaches tau is pruned
    for t in range(ids.shape[0]):
        for e, gv in zip(ids[t], g[t]):
            if gv >= tau:
                assert trans[e]


def test_special_cases():
    rng = np.random.default_rng(7)
    E = 16
    s, keys, ids, g = _random_batch(rng, 10, E, 4, 2, 4)
    cost = rng.uniform(1, 5, E).astype(np.float32)
    bins = (np.arange(E) // 4).astype(np.int32)
    # tau = 0 prunes nothing
    assert not prune_batch(ids, g, E, 0.0, cost, bins, 4)["pruned"].any()
    # all experts resident prunes nothing
    assert not prune_batch(ids, g, E, 0.5, np.zeros(E, np.float32), bins, 4)["pruned"].any()
    # one bin: only zero-cost candidates survive
    c2 = cost.copy()
    c2[::3] = 0
    pr = prune_batch(ids, g, E, 0.3, c2, None, 1)
    assert np.array_equal(pr["promoted"], pr["cand"] & (c2 == 0))
    # uniform cost with one bin is plain threshold pruning
    pr = prune_batch(ids, g, E, 0.3, np.full(E, 3.0, np.float32), None, 1)
    assert np.array_equal(pr["pruned"], pr["cand"])
    # scaling every cost by a power of two changes no decision
    base = prune_batch(ids, g, E, 0.3, cost, bins, 4)
    for j in (-7, 3, 20):
        sc = prune_batch(ids, g, E, 0.3, (cost * np.float32(2.0 ** j)).astype(np.float32), bins, 4)
        assert np.array_equal(sc["trans"], base["trans"])


def test_empty_trans_fallback():
    # tau above any gate weight: A_must is empty; with every cost positive the
    # expansion keeps nothing, so A_trans would be empty and the steps rerun
    # with each token's top expert mandatory
    rng = np.random.default_rng(8)
    E = 16
    s, keys, ids, g = _random_batch(rng, 6, E, 4, 2, 4)
    pr = prune_batch(ids, g, E, 2.0, np.ones(E, np.float32), None, 1)
    assert pr["fallback"]
    for t in range(6):
        assert pr["trans"][ids[t][int(np.argmax(g[t]))]]
    assert np.array_equal(pr["must"], _mask(E, pr["top1"]))
    # one free (zero-cost) activated expert: A_trans = {it}, no fallback
    c = np.ones(E, np.float32)
    free = int(ids[3][2])
    c[free] = 0.0
    pr = prune_batch(ids, g, E, 2.0, c, None, 1)
    assert not pr["fallback"] and not pr["must"].any()
    assert np.flatnonzero(pr["trans"]).tolist() == [free]


def test_step1_literal_vs_keep_top1(golden):
    # Sec. IV-B step 1 as written against the stricter variant that also
    # keeps each token's top expert, on a hand example where they differ
    g_ = golden("mandatory_step1_hand_example.json")
    E = g_["E"]
    ids = np.array(g_["orig_ids"])
    g = np.array(g_["g"])
    bins = np.array(g_["bins"], dtype=np.int32)
    for key, keep in (("literal", False), ("keep_top1", True)):
        want = g_[key]
        pr = prune_batch(ids, g, E, g_["theta"], np.array(g_["cost"], np.float32), bins, g_["n_bins"],
                         rule="sum", keep_top1=keep)
        assert pr["imp"].tolist() == g_["expected_importance"]
        assert np.flatnonzero(pr["must"]).tolist() == want["must"], want["note"]
        assert pr["must_loads"].tolist() == want["must_loads"]
        assert pr["f_base"] == want["f_base"]
        assert pr["cand_order"] == want["cand_order"]
        assert np.flatnonzero(pr["promoted"]).tolist() == want["promoted"]
        assert np.flatnonzero(pr["trans"]).tolist() == want["trans"]
        assert np.flatnonzero(pr["pruned"]).tolist() == want["pruned"]
        assert pr["trans_loads"].tolist() == want["trans_loads"]
        assert pr["fallback"] == want["fallback"]
    for case in g_["empty_cases"]:
        pr = prune_batch(ids, g, E, case["theta"], np.array(case["cost"], np.float32), bins, g_["n_bins"],
                         rule="sum")
        assert np.flatnonzero(pr["must"]).tolist() == case["must"], case["note"]
        assert np.flatnonzero(pr["trans"]).tolist() == case["trans"], case["note"]
        assert np.flatnonzero(pr["pruned"]).tolist() == case["pruned"], case["note"]
        assert pr["fallback"] == case["fallback"], case["note"]


@pytest.mark.parametrize("seed", range(4))
def test_keep_top1_contains_literal(seed):
    # the variant only adds mandatory experts: its A_must holds the literal
    # one and every token's top expert, and it prunes a subset of what the
    # literal set prunes whenever both keep at least one expert
    rng = np.random.default_rng(50 + seed)
    E = 16
    s, keys, ids, g = _random_batch(rng, 8, E, 4, 2, 4)
    cost = rng.uniform(1, 4, E).astype(np.float32)
    bins = (np.arange(E) // 4).astype(np.int32)
    for rule, th in (("max", 0.3), ("sum", 0.6), ("sum", 1.5)):
        lit = prune_batch(ids, g, E, th, cost, bins, 4, rule=rule)
        top = prune_batch(ids, g, E, th, cost, bins, 4, rule=rule, keep_top1=True)
        assert not top["fallback"]
        assert np.all(top["must"] >= _mask(E, top["top1"]))
        if not lit["fallback"]:
            assert np.all(top["must"] >= lit["must"])
        else:
            assert np.array_equal(lit["must"], top["must"]) and np.array_equal(lit["trans"], top["trans"])


def test_loads_exact_under_dynamic_range():
    # fp32 costs whose max/min ratio stays below 2^20 sum exactly in float64,
    # so the fixed-order loads equal the exactly rounded sums.
    rng = np.random.default_rng(9)
    cost = (rng.uniform(0.56, 26.9, 256) * 88080384).astype(np.float32)
    member = rng.random(256) < 0.7
    from oracle import bin_loads
    bins = (np.arange(256) // 32).astype(np.int32)
    loads = bin_loads(member, cost, bins, 8)
    for b in range(8):
        sel = [float(cost[e]) for e in range(256) if member[e] and bins[e] == b]
        assert loads[b] == math.fsum(sel)


def test_threshold_is_inclusive():
    # Sec. IV-B step 1: importance at or above the threshold is mandatory
    act = np.ones(4, dtype=bool)
    imp = np.array([0.25, 0.125, 0.5, 0.0625])
    must, cand = mandatory_split(act, imp, 0.125, [])
    assert must.tolist() == [True, True, True, False]
    assert cand.tolist() == [False, False, False, True]


def test_importance_rules_hand_example(golden):
    from oracle import cir_mandatory, gate_weights, importance_sum
    g_ = golden("importance_rules_hand_example.json")
    E = g_["E"]
    ids = np.array(g_["orig_ids"])
    s = np.array(g_["scores"])
    g = np.array([gate_weights(s[t], ids[t]) for t in range(ids.shape[0])])
    np.testing.assert_array_equal(g, np.array(g_["expected_g"]))
    imp = importance_sum(ids, g, E)
    assert imp.tolist() == g_["expected_sum_importance"]
    pr = prune_batch(ids, g, E, g_["sum_theta"], np.ones(E, np.float32), None, 1, rule="sum")
    assert np.flatnonzero(pr["must"]).tolist() == g_["expected_sum_must"]
    for case in g_["cir_cases"]:
        m = cir_mandatory(ids, s, case["theta_imp"], E)
        assert np.flatnonzero(m).tolist() == case["expected_must"], case["note"]
        pr = prune_batch(ids, g, E, case["theta_imp"], np.ones(E, np.float32), None, 1, rule="cir", s=s)
        assert np.flatnonzero(pr["must"]).tolist() == case["expected_must"]


@pytest.mark.parametrize("seed", range(4))
def test_importance_rule_invariants(seed):
    rng = np.random.default_rng(300 + seed)
    E, T, k = 16, 20, 4
    s, keys, ids, g = route_batch(rng.standard_normal((T, E)).astype(np.float32), None, 4, 2, k)
    from oracle import importance_sum
    imp = importance_sum(ids, g, E)
    np.testing.assert_allclose(imp.sum(), T, rtol=1e-14)       # every token's weights sum to one
    cost = rng.uniform(1, 4, E).astype(np.float32)
    bins = (np.arange(E) // 4).astype(np.int32)
    # CIR with ratio 1 keeps everything; a tiny ratio keeps only each token's top expert
    full = prune_batch(ids, g, E, 1.0, cost, bins, 4, rule="cir", s=s)
    assert np.array_equal(full["must"], full["act"]) and not full["pruned"].any()
    tiny = prune_batch(ids, g, E, 1e-9, cost, bins, 4, rule="cir", s=s)
    assert np.array_equal(tiny["must"], np.isin(np.arange(E), tiny["top1"]))
    # SUM with a threshold above the batch total: A_must empty, every cost
    # positive, so A_trans would be empty and the fallback keeps the top experts
    top = prune_batch(ids, g, E, T + 1.0, cost, bins, 4, rule="sum")
    assert top["fallback"]
    assert np.array_equal(top["must"], np.isin(np.arange(E), top["top1"]))
    # larger thresholds never grow the step-1 set (SUM) and larger ratios
    # never shrink it (CIR), among calls that need no fallback
    for rule in ("sum", "cir"):
        prev = None
        for th in ((0.2, 0.5, 1.0, 2.0) if rule == "sum" else (0.3, 0.6, 0.9)):
            pr = prune_batch(ids, g, E, th, cost, bins, 4, rule=rule, s=s)
            if pr["fallback"]:
                continue
            m = pr["must"]
            if prev is not None:
                assert np.all(m <= prev) if rule == "sum" else np.all(prev <= m)
            prev = m


def test_step1_readings_differ_on_tiny_layers():
    # the GPU parity cases of both readings (tiny layer, Zipf costs on 4 bins)
    # include calls where the two prune different sets and calls that need
    # the fallback
    from oracle import moe_layer_ref
    from synth_inputs import TINY_F32, make_routing_inputs
    sh = TINY_F32
    differ = fallback = 0
    for T in (1, 5, 16, 40, 300):
        for rule, tau in (("sum", 1.2), ("sum", 2.5), ("max", 0.3)):
            inp = make_routing_inputs(sh, seed=60 + T, T=T, zipf_logit_s=1.1, cost_kind="zipf", n_bins=4)
            kw = dict(E=sh.E, n_group=sh.n_group, topk_group=sh.topk_group, k=sh.k, routed_scaling=1.0,
                      tau=tau, n_bins=4, logits=inp.logits, cost=inp.cost, bins=inp.bins, rule=rule)
            a = moe_layer_ref(**kw)
            b = moe_layer_ref(**kw, keep_top1=True)
            differ += int(not np.array_equal(a["trans"], b["trans"]))
            fallback += a["stats"]["fallback"]
    assert differ > 0 and fallback > 0
