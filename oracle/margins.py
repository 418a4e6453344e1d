"""Decision margins of a routed, pruned and compensated batch (oracle,
fp64) -- how far each discrete decision of the layer is from flipping.

Test infrastructure only; see the package docstring.

Each routing and pruning step of the layer is a comparison: a group or an
expert is selected when its score beats the next one (Sec. II-A top-k, with
group-limited routing), an expert is mandatory when its importance reaches
the threshold (Sec. IV-B step 1), candidates are visited in importance order
(step 3), and freed slots are refilled by router key (Sec. IV-C).  The
margin of a decision is the gap between the two values it compares; a gap
below the floating-point noise of the two implementations (about 1e-12 for
these float64 decisions) marks a near-tie, where two correct
implementations may legitimately disagree.  Cost comparisons are exact sums
(no margin).
"""
from __future__ import annotations

import numpy as np


def _gap(sorted_desc, n):
    """Gap between the n-th and (n+1)-th of a descending list (inf when
    either is missing)."""
    if n <= 0 or n >= len(sorted_desc):
        return float("inf")
    return float(sorted_desc[n - 1] - sorted_desc[n])


def decision_margins(ref: dict, *, n_group: int, topk_group: int, k: int, tau: float, rule: str) -> dict:
    """Smallest margin of each kind over the batch, from the outputs of
    ``moe_layer_ref``: "group" (last selected vs first dropped group score),
    "topk" (k-th vs (k+1)-th key inside the selected groups), "threshold"
    (|I(e) - tau| over A_act for MAX and SUM; for CIR |CIR(m) - theta| at
    the two prefix lengths around each token's cut), "order" (importance
    gap of consecutive candidates in visiting order), "refill" (last
    refilled vs first unused key of the pool), and "min" over all."""
    keys, s, ids, g = ref["keys"], ref["s"], ref["orig_ids"], ref["g"]
    T, E = keys.shape
    gsz = E // n_group
    m = {"group": float("inf"), "topk": float("inf"), "threshold": float("inf"),
         "order": float("inf"), "refill": float("inf")}
    trans = ref["trans"]
    for t in range(T):
        key = keys[t]
        gs = []
        for grp in range(n_group):
            mem = np.sort(key[grp * gsz:(grp + 1) * gsz])[::-1]
            gs.append(mem[0] + mem[1] if gsz >= 2 else mem[0])
        order = np.argsort(-np.array(gs), kind="stable")
        m["group"] = min(m["group"], _gap(np.array(gs)[order], topk_group))
        allowed = np.concatenate([np.arange(grp * gsz, (grp + 1) * gsz) for grp in order[:topk_group]])
        m["topk"] = min(m["topk"], _gap(np.sort(key[allowed])[::-1], k))
        if rule == "cir":
            sv = np.sort(s[t, ids[t]])[::-1]
            ratio = np.cumsum(sv) / sv.sum()
            cut = int(np.argmax(ratio >= tau)) if np.any(ratio >= tau) else len(sv) - 1
            for j in (cut - 1, cut):
                if 0 <= j < len(sv):
                    m["threshold"] = min(m["threshold"], abs(float(ratio[j]) - tau))
        # refill: the pool is A_trans minus K_t, ranked by key
        kept = [e for e in ids[t] if trans[e]]
        n_fill = k - len(kept)
        pool = np.array([key[e] for e in np.flatnonzero(trans) if e not in set(ids[t].tolist())])
        if n_fill > 0 and len(pool) > n_fill:
            m["refill"] = min(m["refill"], _gap(np.sort(pool)[::-1], n_fill))
    act = ref["act"]
    if rule in ("max", "sum") and act.any():
        m["threshold"] = min(m["threshold"], float(np.min(np.abs(ref["imp"][act] - tau))))
    cand = ref["cand_order"]
    for a, b in zip(cand, cand[1:]):
        m["order"] = min(m["order"], float(ref["imp"][a] - ref["imp"][b]))
    m["min"] = min(m.values())
    return m
