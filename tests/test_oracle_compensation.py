"""Pins for the oracle's compensation step (Sec. IV-C): a hand-computed
example and the invariants it must satisfy on random batches."""
import numpy as np
import pytest

import oracle
from oracle import compensate_batch, compensate_token, group_limited_topk, prune_batch, route_batch


def test_hand_example(golden):
    g = golden("compensation_hand_example.json")
    s = np.array(g["scores"])
    ids, key = group_limited_topk(s, None, g["n_group"], g["topk_group"], g["k"])
    assert ids == g["expected_orig_ids"]
    tot = sum(s[e] for e in ids)
    np.testing.assert_allclose([s[e] / tot for e in ids], g["expected_orig_g"], rtol=1e-15)
    trans = np.zeros(8, dtype=bool)
    trans[g["trans"]] = True
    fid, fw, nref = compensate_token(key, s, ids, trans, g["k"], g["routed_scaling"])
    assert fid == g["expected_final_ids"]
    np.testing.assert_allclose(fw, g["expected_final_w"], rtol=1e-15)
    assert nref == 2


@pytest.mark.parametrize("seed", range(5))
@pytest.mark.parametrize("tau", [0.0, 0.2, 0.3])
def test_invariants(seed, tau):
    rng = np.random.default_rng(100 + seed)
    E, k, rs = 16, 4, 2.5
    T = [1, 3, 16, 16, 40][seed]
    logits = rng.standard_normal((T, E)).astype(np.float32)
    bias = (rng.standard_normal(E) * 0.1).astype(np.float32)
    s, keys, ids, g = route_batch(logits, bias, 4, 2, k)
    cost = rng.uniform(1, 3, E).astype(np.float32)
    bins = (np.arange(E) // 4).astype(np.int32)
    pr = prune_batch(ids, g, E, tau, cost, bins, 4)
    fid, fw, nref = compensate_batch(keys, s, ids, pr["trans"], k, rs)
    n_trans = int(pr["trans"].sum())
    for t in range(T):
        row = [e for e in fid[t] if e >= 0]
        assert len(row) == len(set(row)) == min(k, n_trans)
        assert all(pr["trans"][e] for e in row)
        np.testing.assert_allclose(fw[t].sum(), rs, rtol=1e-15)
        assert np.all(fw[t][len(row):] == 0) and np.all(fid[t][len(row):] == -1)
        for e, gv in zip(ids[t], g[t]):
            if gv >= tau:
                assert e in row
        if tau == 0.0:
            assert row == ids[t].tolist()
        if T == 1:
            assert set(row) == {e for e in ids[t] if pr["trans"][e]}
        kk = keys[t, row]
        assert np.all(kk[:-1] >= kk[1:])


def test_refill_ignores_groups():
    # token 0 routes inside group 0; token 1 activates group 1 experts, which
    # become the only survivors token 0 can be refilled with.
    E = 8
    s = np.array([[0.9, 0.8, 0.7, 0.6, 0.1, 0.1, 0.1, 0.1],
                  [0.1, 0.1, 0.1, 0.1, 0.9, 0.8, 0.7, 0.6]])
    keys = s.copy()
    trans = np.zeros(E, dtype=bool)
    trans[[0, 5, 6]] = True
    ids = np.array([[0, 1], [4, 5]])
    fid, fw, nref = compensate_batch(keys, s, ids, trans, 2, 1.0)
    assert fid[0].tolist() == [0, 5]
    assert fid[1].tolist() == [5, 6]
    assert nref == 2


# ---- literal top-k of the masked scores (Sec. IV-C read literally) -----------

def test_literal_hand_example():
    # E=4 in two groups {0,1}, {2,3}; one group per token, k=2.  Scores
    # [0.9, 0.1, 0.8, 0.7] (bias 0, so keys = scores): group sums 1.0 and
    # 1.5 select group 1, K_t = {2, 3}.  With A_trans = {0, 2, 3} (expert 0
    # activated by another token) keep-and-refill keeps {2, 3}; the literal
    # top-2 of the masked scores is {0, 2}, dropping the token's own expert 3.
    sc = np.array([[0.9, 0.1, 0.8, 0.7]])
    logits = np.log(sc / (1.0 - sc))
    _, _, ids, _ = oracle.route_batch(logits, np.zeros(4), 2, 1, 2)
    assert sorted(ids[0].tolist()) == [2, 3]
    trans = np.array([True, False, True, True])
    sid, sw, sn = compensate_batch(sc, sc, ids, trans, 2, 2.5, "score")
    lid, lw, ln = compensate_batch(sc, sc, ids, trans, 2, 2.5, "literal")
    assert sid[0].tolist() == [2, 3] and sn == 0
    assert lid[0].tolist() == [0, 2] and ln == 1
    np.testing.assert_allclose(lw[0], [2.5 * 0.9 / 1.7, 2.5 * 0.8 / 1.7], rtol=0, atol=1e-15)


@pytest.mark.parametrize("seed", range(3))
def test_literal_is_top_k_of_trans(seed):
    # brute force: each token's K_final is the first k of A_trans ordered by
    # (key desc, index asc), whatever its own K_t was
    shape, inp = _ablation_case(seed)
    ref = oracle.moe_layer_ref(E=shape.E, n_group=shape.n_group, topk_group=shape.topk_group, k=shape.k,
                               routed_scaling=1.0, tau=0.8, n_bins=1, logits=inp.logits, cost=inp.cost,
                               rule="cir", refill="literal")
    trans = np.flatnonzero(ref["trans"]).tolist()
    n_out = 0
    for t in range(inp.logits.shape[0]):
        order = sorted(trans, key=lambda e: (-ref["keys"][t, e], e))[:shape.k]
        assert [e for e in ref["topk_ids"][t] if e >= 0] == order
        assert abs(sum(ref["topk_w"][t]) - 1.0) < 1e-12
        n_out += sum(1 for e in order if e not in ref["orig_ids"][t])
    assert ref["stats"]["n_refill"] == n_out


def test_literal_equals_score_for_one_token():
    # T = 1: A_trans lies inside the token's own K_t, so both readings agree
    shape, inp = _ablation_case(5, T=1)
    for tau in (0.0, 0.8):
        kw = dict(E=shape.E, n_group=shape.n_group, topk_group=shape.topk_group, k=shape.k, routed_scaling=1.0,
                  tau=tau, n_bins=1, logits=inp.logits, cost=inp.cost, rule="cir")
        a = oracle.moe_layer_ref(**kw, refill="score")
        b = oracle.moe_layer_ref(**kw, refill="literal")
        assert np.array_equal(a["topk_ids"], b["topk_ids"])
        np.testing.assert_array_equal(a["topk_w"], b["topk_w"])


# ---- refill variants of the compensation ablation ----------------------------

def test_splitmix64_published_outputs(golden):
    from oracle.compensation import splitmix64
    g = golden("splitmix64.json")
    gamma = int(g["gamma"], 16)
    got = [splitmix64(i * gamma) for i in range(3)]
    assert got == [int(v, 16) for v in g["outputs_from_state_0"]]


def _ablation_case(seed=0, T=16):
    from synth_inputs import TINY_F32, make_routing_inputs
    shape = TINY_F32
    inp = make_routing_inputs(shape, seed=seed, T=T, zipf_logit_s=1.2, cost_kind="zipf")
    return shape, inp


@pytest.mark.parametrize("seed", range(3))
def test_refill_none_keeps_only_survivors(seed):
    shape, inp = _ablation_case(seed)
    ref = oracle.moe_layer_ref(E=shape.E, n_group=shape.n_group, topk_group=shape.topk_group, k=shape.k,
                               routed_scaling=1.0, tau=0.8, n_bins=1, logits=inp.logits, cost=inp.cost,
                               rule="cir", refill="none")
    trans = ref["trans"]
    for t in range(inp.logits.shape[0]):
        want = [e for e in ref["orig_ids"][t] if trans[e]]
        got = [e for e in ref["topk_ids"][t] if e >= 0]
        assert sorted(got) == sorted(want)
        assert abs(sum(ref["topk_w"][t]) - 1.0) < 1e-12
    assert ref["stats"]["n_refill"] == 0


@pytest.mark.parametrize("seed", range(3))
def test_refill_random_takes_top_random_keys(seed):
    from oracle.compensation import refill_key
    shape, inp = _ablation_case(seed)
    kw = dict(E=shape.E, n_group=shape.n_group, topk_group=shape.topk_group, k=shape.k, routed_scaling=1.0,
              tau=0.8, n_bins=1, logits=inp.logits, cost=inp.cost, rule="cir")
    score = oracle.moe_layer_ref(**kw, refill="score")
    rnd = oracle.moe_layer_ref(**kw, refill="random", seed=7)
    trans = rnd["trans"]
    assert np.array_equal(trans, score["trans"])   # the refill never changes the pruning
    pool_all = set(np.flatnonzero(trans).tolist())
    for t in range(inp.logits.shape[0]):
        orig = set(rnd["orig_ids"][t].tolist())
        keep = {e for e in orig if trans[e]}
        fin = {e for e in rnd["topk_ids"][t].tolist() if e >= 0}
        assert keep <= fin and fin <= pool_all
        assert len(fin) == min(shape.k, len(pool_all))
        added = fin - keep
        rest = pool_all - orig - added
        # every added expert's key beats every left-out candidate's key
        if added and rest:
            assert min(refill_key(7, t, e, shape.E) for e in added) > max(refill_key(7, t, e, shape.E) for e in rest)
    other = oracle.moe_layer_ref(**kw, refill="random", seed=8)
    if rnd["stats"]["n_refill"] > 0:
        assert not np.array_equal(rnd["topk_ids"], other["topk_ids"])


def test_refill_variants_agree_without_pruning():
    shape, inp = _ablation_case(1)
    kw = dict(E=shape.E, n_group=shape.n_group, topk_group=shape.topk_group, k=shape.k, routed_scaling=1.0,
              tau=0.0, n_bins=1, logits=inp.logits, cost=inp.cost)
    a = oracle.moe_layer_ref(**kw, refill="score")
    for mode in ("none", "random"):
        b = oracle.moe_layer_ref(**kw, refill=mode, seed=3)
        assert np.array_equal(a["topk_ids"], b["topk_ids"])
