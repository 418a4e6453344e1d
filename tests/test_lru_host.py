"""The residency plan of caee_offload_layer (caee_lru_step, host code of
the C ABI) against the LRU oracle, on random call sequences.  No GPU."""
from collections import OrderedDict

import numpy as np
import pytest

from oracle import offload as off
from paper_2606_29982_amd import caee


def _state(E, n_cache):
    return (np.full(E, -1, np.int32), np.full(n_cache, -1, np.int32), np.full(n_cache, -1, np.int64))


@pytest.mark.parametrize("seed,E,n_cache,n_stage", [(0, 16, 4, 2), (1, 32, 8, 3), (2, 256, 64, 16),
                                                    (3, 20, 1, 1), (4, 12, 12, 0)])
def test_lru_step_matches_oracle(seed, E, n_cache, n_stage):
    rng = np.random.default_rng(seed)
    slot_of, slot_expert, slot_used = _state(E, n_cache)
    cache = OrderedDict()
    # Zipf-like popularity so that hits, evictions and (when allowed) staging all happen.
    p = 1.0 / np.arange(1, E + 1) ** 1.2
    p = p[rng.permutation(E)]
    p /= p.sum()
    for call in range(80):
        hi = n_cache + n_stage * 3 if n_stage else n_cache
        size = int(rng.integers(0, min(E, hi) + 1))
        need_ids = np.sort(rng.choice(E, size=size, replace=False, p=p))
        need = np.zeros(E, np.uint8)
        need[need_ids] = 1
        before = set(np.flatnonzero(slot_of >= 0).tolist())
        fetch, fetch_slot, (hits, misses, staged, evictions) = caee.lru_step(
            E, n_cache, n_stage, slot_of, slot_expert, slot_used, call, need)
        want = off.lru_call(cache, n_cache, need_ids.tolist())
        assert hits == len(want["hits"]) and misses == len(want["cached"]) + len(want["staged"])
        assert staged == len(want["staged"]) and evictions == len(want["evicted"])
        assert fetch.tolist() == want["cached"] + want["staged"]
        after = set(np.flatnonzero(slot_of >= 0).tolist())
        assert after == set(cache)
        assert before - after == set(want["evicted"])
        # cached misses land in their cache slot, staged ones cycle through the staging slots
        nc = len(want["cached"])
        for i, e in enumerate(fetch.tolist()):
            if i < nc:
                assert fetch_slot[i] == slot_of[e] and slot_expert[fetch_slot[i]] == e
            else:
                assert fetch_slot[i] == n_cache + (i - nc) % n_stage
        assert np.all(slot_used[slot_of[need_ids][slot_of[need_ids] >= 0]] == call)


def test_lru_step_capacity_error_leaves_state():
    E, n_cache = 8, 2
    slot_of, slot_expert, slot_used = _state(E, n_cache)
    need = np.zeros(E, np.uint8)
    need[[1, 2, 3]] = 1
    s0 = (slot_of.copy(), slot_expert.copy(), slot_used.copy())
    with pytest.raises(caee.CaeeError) as ei:
        caee.lru_step(E, n_cache, 0, slot_of, slot_expert, slot_used, 0, need)
    assert ei.value.status == caee.CAEE_ERR_CAPACITY
    for a, b in zip(s0, (slot_of, slot_expert, slot_used)):
        assert np.array_equal(a, b)


def test_lru_step_rejects_inconsistent_state():
    E, n_cache = 8, 2
    slot_of, slot_expert, slot_used = _state(E, n_cache)
    slot_of[3] = 1          # slot 1 does not hold expert 3
    with pytest.raises(caee.CaeeError) as ei:
        caee.lru_step(E, n_cache, 1, slot_of, slot_expert, slot_used, 0, np.zeros(E, np.uint8))
    assert ei.value.status == caee.CAEE_ERR_INVALID_ARG
    slot_of[3] = -1
    slot_expert[0], slot_of[2], slot_used[0] = 2, 0, 5
    with pytest.raises(caee.CaeeError):   # last use not before this call
        caee.lru_step(E, n_cache, 1, slot_of, slot_expert, slot_used, 5, np.zeros(E, np.uint8))
