"""Offload residency (fp64 CAEE oracle) -- TEST INFRASTRUCTURE ONLY.

In the offloading deployment (Sec. V-B) every routed expert lives in host
memory and a bounded set of them in device memory.  The cost model of
Sec. IV-A gives each expert the residency factor R(e, d): 1 when using it
would trigger a host-to-device transfer, 0 when it is already on the device
(a cache hit).  The layer's cost table is therefore R(e) * C(e): zero for
resident experts and the transfer cost for the others, all on one link.

The paper's own system manages its per-device cache with LFU; the workload
here uses a least-recently-used cache, whose plain definition is written out
below.  Readings taken where LRU needs a convention:
  * time advances by layer calls: every expert a call needs (its A_trans)
    counts as used at that call; among experts last used by the same call,
    the lower expert index counts as older;
  * a call's misses are inserted in ascending expert order; each takes a
    free slot if there is one, otherwise evicts the least recently used
    resident expert that this call does not need;
  * when every resident expert is needed by the call, a further miss is
    "staged": brought in for this call only and not cached.
"""
from __future__ import annotations

from collections import OrderedDict

import numpy as np


def residency_cost(resident, E: int, miss_cost: float) -> np.ndarray:
    """Cost table R(e) * C(e) (Sec. IV-A): 0 for resident experts, miss_cost
    for the others.  fp32, as the table the layer takes."""
    cost = np.full(E, np.float32(miss_cost), dtype=np.float32)
    for e in resident:
        cost[int(e)] = 0.0
    return cost


def lru_call(cache: "OrderedDict[int, None]", capacity: int, needed) -> dict:
    """One layer call against an LRU cache of ``capacity`` experts.

    ``cache`` holds the resident experts, least recently used first, and is
    updated in place.  Returns the call's hits, cached misses, staged misses
    and evicted experts (each in the order they happened)."""
    need = sorted(int(e) for e in needed)
    need_set = set(need)
    hits = [e for e in need if e in cache]
    misses = [e for e in need if e not in cache]
    cached, staged, evicted = [], [], []
    for e in misses:
        if len(cache) < capacity:
            cache[e] = None
            cached.append(e)
            continue
        victim = next((v for v in cache if v not in need_set), None)
        if victim is None:
            staged.append(e)
            continue
        del cache[victim]
        evicted.append(victim)
        cache[e] = None
        cached.append(e)
    # Every needed expert that is now resident was used by this call; among
    # them the lower index is the older one.
    for e in sorted(hits + cached):
        cache.move_to_end(e)
    return {"hits": hits, "cached": cached, "staged": staged, "evicted": evicted}


def offload_sequence(route_call, E: int, capacity: int, miss_cost: float, n_calls: int):
    """Runs ``n_calls`` layer calls against one LRU cache, starting empty.

    ``route_call(i, cost)`` must return the oracle layer result (a dict with
    the ``trans`` membership of A_trans) of call ``i`` under cost table
    ``cost``.  Yields, per call, the cost table, the layer result, the LRU
    outcome and the resident set after the call."""
    cache: "OrderedDict[int, None]" = OrderedDict()
    for i in range(n_calls):
        resident_before = set(cache)
        cost = residency_cost(resident_before, E, miss_cost)
        ref = route_call(i, cost)
        needed = np.flatnonzero(ref["trans"])
        lru = lru_call(cache, capacity, needed)
        yield {"cost": cost, "ref": ref, "lru": lru, "resident_before": resident_before,
               "resident_after": set(cache)}
