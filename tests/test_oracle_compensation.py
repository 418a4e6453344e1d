"""Pins for the oracle's compensation step (Sec. IV-C): a hand-computed
example and the invariants it must satisfy on random batches."""
import numpy as np
import pytest

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
