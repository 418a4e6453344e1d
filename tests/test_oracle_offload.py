"""Pins of the offload-residency oracle: a hand-worked LRU sequence, the
closed form of an LRU cache that never overflows, and what the Sec. IV-A
cost model implies for pruning with a one-link residency cost table."""
from collections import OrderedDict

import numpy as np
import pytest

import oracle
from oracle import offload as off
from synth_inputs import TINY_F32, make_routing_inputs


def test_lru_hand_example(golden):
    g = golden("lru_hand_example.json")
    cache = OrderedDict()
    for need, want in zip(g["calls"], g["expected"]):
        got = off.lru_call(cache, g["capacity"], need)
        for key in ("hits", "cached", "staged", "evicted"):
            assert got[key] == want[key], (need, key)
        assert sorted(cache) == want["resident_after"]


def _recency_top(history, capacity):
    """Closed form: with no call needing more experts than the capacity, the
    resident set is the `capacity` experts with the latest (last call, index)."""
    last = {}
    for i, need in enumerate(history):
        for e in need:
            last[e] = i
    ranked = sorted(last, key=lambda e: (last[e], e), reverse=True)
    return set(ranked[:capacity])


@pytest.mark.parametrize("seed", range(5))
def test_lru_matches_recency_closed_form(seed):
    rng = np.random.default_rng(seed)
    E, capacity = 24, 7
    cache = OrderedDict()
    history = []
    for _ in range(60):
        need = sorted(rng.choice(E, size=int(rng.integers(0, capacity + 1)), replace=False).tolist())
        history.append(need)
        res = off.lru_call(cache, capacity, need)
        assert res["staged"] == []
        assert set(cache) == _recency_top(history, capacity)
        assert len(res["hits"]) + len(res["cached"]) == len(need)


def test_lru_overflow_stages_highest_indices():
    cache = OrderedDict((e, None) for e in (5, 6))
    res = off.lru_call(cache, 3, [0, 1, 2, 3, 6])
    # 6 hits; 5 is the only victim; 0 takes the free slot, 1 evicts 5; 2, 3 staged.
    assert res == {"hits": [6], "cached": [0, 1], "staged": [2, 3], "evicted": [5]}
    assert list(cache) == [0, 1, 6]


def test_residency_cost_table():
    c = off.residency_cost({1, 3}, 5, 2.5)
    assert c.dtype == np.float32
    assert c.tolist() == [2.5, 0.0, 2.5, 0.0, 2.5]


@pytest.mark.parametrize("tau", [0.0, 0.05, 0.1])
def test_one_link_pruning_keeps_resident_drops_absent(tau):
    """With one bin (the host link) and zero cost for resident experts,
    cost-invariant expansion (Sec. IV-B step 3) promotes exactly the resident
    candidates whenever some mandatory expert is absent or the baseline is 0;
    every candidate that would need a transfer is pruned."""
    shape = TINY_F32
    inp = make_routing_inputs(shape, seed=3, zipf_logit_s=1.2)
    rng = np.random.default_rng(0)
    resident = set(rng.choice(shape.E, size=6, replace=False).tolist())
    cost = off.residency_cost(resident, shape.E, 1.0)
    ref = oracle.moe_layer_ref(E=shape.E, n_group=shape.n_group, topk_group=shape.topk_group, k=shape.k,
                               routed_scaling=1.0, tau=tau, n_bins=1, logits=inp.logits, cost=cost)
    cand = np.flatnonzero(ref["cand"])
    for e in cand:
        assert bool(ref["promoted"][e]) == (e in resident), e
    if tau == 0.0:
        assert not ref["pruned"].any()
    # A_trans = must + resident candidates; nothing absent joins without being mandatory
    for e in np.flatnonzero(ref["trans"]):
        assert ref["must"][e] or e in resident


def test_offload_sequence_costs_follow_residency():
    shape = TINY_F32
    calls = [make_routing_inputs(shape, seed=s, zipf_logit_s=1.2) for s in range(6)]

    def route(i, cost):
        return oracle.moe_layer_ref(E=shape.E, n_group=shape.n_group, topk_group=shape.topk_group, k=shape.k,
                                    routed_scaling=1.0, tau=0.1, n_bins=1, logits=calls[i].logits, cost=cost)

    seen = list(off.offload_sequence(route, shape.E, 4, 3.0, len(calls)))
    assert seen[0]["resident_before"] == set() and np.all(seen[0]["cost"] == 3.0)
    for prev, cur in zip(seen, seen[1:]):
        assert cur["resident_before"] == prev["resident_after"]
        assert set(np.flatnonzero(cur["cost"] == 0)) == cur["resident_before"]
        assert len(cur["resident_after"]) <= 4
