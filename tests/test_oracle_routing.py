"""Pins for the oracle's router (sigmoid scores, group-limited top-k, gate
weights) against hand-computed values, closed forms, library routines and a
counting restatement of the selection rule."""
import itertools

import numpy as np
import pytest
import scipy.special
import torch

from oracle import gate_weights, group_limited_topk, route_batch, sigmoid_scores


def test_hand_example(golden):
    g = golden("routing_hand_example.json")
    s = np.array(g["scores"], dtype=np.float64)
    ids, key = group_limited_topk(s, None, g["n_group"], g["topk_group"], g["k"])
    assert ids == g["expected_ids"]
    ids1, _ = group_limited_topk(s, None, 1, 1, g["k"])
    assert ids1 == g["expected_ids_one_group"]
    # the group scores as the rule defines them (top-2 sums, exact for dyadics)
    gs = [sorted(s[2 * i:2 * i + 2])[::-1] for i in range(4)]
    assert [a + b for a, b in gs] == g["expected_group_scores"]


def test_sigmoid_against_library_and_closed_forms():
    z = np.random.default_rng(1).standard_normal(1000) * 6
    s = sigmoid_scores(z)
    np.testing.assert_allclose(s, scipy.special.expit(z), rtol=1e-15, atol=0)
    np.testing.assert_allclose(s + sigmoid_scores(-z), 1.0, rtol=0, atol=4.5e-16)
    assert sigmoid_scores(np.array([0.0]))[0] == 0.5
    assert sigmoid_scores(np.array([-1000.0]))[0] == 0.0
    assert sigmoid_scores(np.array([1000.0]))[0] == 1.0


def test_one_group_is_plain_topk():
    rng = np.random.default_rng(2)
    for _ in range(50):
        s = rng.random(16)
        bias = rng.standard_normal(16) * 0.1
        ids, key = group_limited_topk(s, bias, 1, 1, 5)
        ref = np.lexsort((np.arange(16), -(s + bias)))[:5].tolist()
        assert ids == ref


def test_singleton_groups_reduce_to_topk():
    rng = np.random.default_rng(3)
    s = rng.random(8)
    ids, _ = group_limited_topk(s, None, 8, 3, 3)
    assert ids == np.argsort(-s, kind="stable")[:3].tolist()


def _counting_rule(s, bias, n_group, topk_group, k):
    """Restatement by counting: a group is kept iff fewer than topk_group
    groups beat it; an expert of a kept group is selected iff fewer than k
    experts of kept groups beat it ("beat" = larger value, or equal value
    and lower index)."""
    E = len(s)
    key = s + (0 if bias is None else bias)
    gsz = E // n_group
    gs = []
    for g in range(n_group):
        m = key[g * gsz:(g + 1) * gsz]
        top2 = np.sort(m)[::-1]
        gs.append(top2[0] + top2[1] if gsz > 1 else top2[0])
    beats = lambda va, ia, vb, ib: va > vb or (va == vb and ia < ib)  # noqa: E731
    kept = [g for g in range(n_group)
            if sum(beats(gs[h], h, gs[g], g) for h in range(n_group)) < topk_group]
    pool = [e for g in kept for e in range(g * gsz, (g + 1) * gsz)]
    sel = [e for e in pool if sum(beats(key[o], o, key[e], e) for o in pool) < k]
    return set(sel)


@pytest.mark.parametrize("E,G,tg,k", [(16, 4, 2, 4), (32, 8, 3, 6), (12, 3, 1, 2), (8, 4, 2, 2)])
def test_counting_restatement(E, G, tg, k):
    rng = np.random.default_rng(E * 100 + k)
    for _ in range(40):
        # coarse values make exact ties frequent
        s = rng.integers(0, 6, E) / 8.0
        bias = None if rng.random() < 0.5 else rng.integers(-2, 3, E) / 16.0
        ids, _ = group_limited_topk(s, bias, G, tg, k)
        assert set(ids) == _counting_rule(s, bias, G, tg, k)
        assert len(ids) == k == len(set(ids))


def test_equal_logits_pick_lowest_indices():
    logits = np.zeros((3, 16), dtype=np.float32)
    s, keys, ids, g = route_batch(logits, None, 4, 2, 4)
    assert ids.tolist() == [[0, 1, 2, 3]] * 3
    np.testing.assert_allclose(g, 0.25, rtol=0, atol=0)


def test_gate_weights_sum_to_one_and_ignore_bias():
    rng = np.random.default_rng(4)
    logits = rng.standard_normal((20, 32)).astype(np.float32)
    bias = (rng.standard_normal(32) * 0.5).astype(np.float32)
    s, keys, ids, g = route_batch(logits, bias, 8, 4, 6)
    np.testing.assert_allclose(g.sum(axis=1), 1.0, rtol=0, atol=4e-16)
    for t in range(20):
        np.testing.assert_allclose(g[t], s[t, ids[t]] / s[t, ids[t]].sum(), rtol=1e-15)
        # rank order: key descending
        kk = keys[t, ids[t]]
        assert np.all(kk[:-1] >= kk[1:])


def test_bias_moves_selection():
    logits = np.zeros((1, 8), dtype=np.float32)
    logits[0, :] = [3, 2, 1, 0, -1, -2, -3, -4]
    bias = np.zeros(8, dtype=np.float32)
    bias[7] = 2.0
    _, _, ids, g = route_batch(logits, bias, 1, 1, 2)
    assert ids[0].tolist() == [7, 0]
    s = scipy.special.expit(logits[0].astype(np.float64))
    np.testing.assert_allclose(g[0], [s[7] / (s[7] + s[0]), s[0] / (s[7] + s[0])], rtol=1e-15)


def test_scores_match_torch_sigmoid():
    z = torch.randn(4, 64, dtype=torch.float64, generator=torch.Generator().manual_seed(5))
    np.testing.assert_allclose(sigmoid_scores(z.numpy()), torch.sigmoid(z).numpy(), rtol=4.5e-16, atol=0)


def test_exhaustive_tiny_selection():
    # all 4-expert, 2-group layouts with values in {0,1,2}: every pattern
    for vals in itertools.product(range(3), repeat=4):
        s = np.array(vals, dtype=np.float64)
        ids, _ = group_limited_topk(s, None, 2, 1, 1)
        assert set(ids) == _counting_rule(s, None, 2, 1, 1)
        ids, _ = group_limited_topk(s, None, 2, 2, 3)
        assert set(ids) == _counting_rule(s, None, 2, 2, 3)


def test_gate_weights_order_fixed():
    s = np.array([0.1, 0.7, 0.2, 0.9])
    g = gate_weights(s, [3, 1])
    assert g.tolist() == [0.9 / 1.6, 0.7 / 1.6]
