"""Router scoring and group-limited top-k selection (oracle, fp64).

Test infrastructure only; see the package docstring.

Paper: the MoE output equation of Sec. II-A (a router picks a set K_t of k
experts per token and weights them by normalised scores G(t)_e summing to 1).
The paper names DeepSeek's group routing (Sec. V-C discussion) without
defining it; the definition used here is the DeepSeek layer's: sigmoid
scores, a per-expert bias added for selection only, each group scored by the
sum of its two best biased scores, the best ``topk_group`` groups kept, then
the best ``k`` experts inside them.  All ties go to the lower index.
"""
from __future__ import annotations

import numpy as np


def sigmoid_scores(logits: np.ndarray) -> np.ndarray:
    """s = 1 / (1 + exp(-logit)), element-wise, in float64."""
    z = np.asarray(logits, dtype=np.float64)
    with np.errstate(over="ignore"):
        return 1.0 / (1.0 + np.exp(-z))


def _rank_key(val: float, idx: int):
    # Sort key: larger value first, then lower index.
    return (-val, idx)


def group_limited_topk(s: np.ndarray, bias, n_group: int, topk_group: int, k: int):
    """Select K_t for one token from its scores ``s`` (length E, float64).

    key_e = s_e + bias_e.  Group g holds experts [g*E/n_group, (g+1)*E/n_group).
    Group score = sum of its two largest keys (its only key when a group has a
    single expert).  Keep the ``topk_group`` best groups, then the ``k`` best
    experts among them.  Returns expert ids in rank order (key descending,
    index ascending) and the key vector.
    """
    E = s.shape[0]
    key = s + (np.zeros(E) if bias is None else np.asarray(bias, dtype=np.float64))
    gs_size = E // n_group
    group_score = []
    for g in range(n_group):
        members = sorted(key[g * gs_size:(g + 1) * gs_size].tolist(), reverse=True)
        group_score.append(members[0] + members[1] if gs_size >= 2 else members[0])
    groups = sorted(range(n_group), key=lambda g: _rank_key(group_score[g], g))[:topk_group]
    allowed = [e for g in groups for e in range(g * gs_size, (g + 1) * gs_size)]
    ids = sorted(allowed, key=lambda e: _rank_key(float(key[e]), e))[:k]
    return ids, key


def gate_weights(s: np.ndarray, ids) -> np.ndarray:
    """G(t)_e = s_e / sum_{e' in K_t} s_e' (Sec. II-A: the weights of the
    selected experts sum to one).  The sum runs over ``ids`` in the given
    order, one float64 addition at a time."""
    total = 0.0
    for e in ids:
        total += float(s[e])
    return np.array([float(s[e]) / total for e in ids], dtype=np.float64)


def route_batch(logits: np.ndarray, bias, n_group: int, topk_group: int, k: int):
    """Route every token.  Returns (s [T][E], key [T][E], ids [T][k] int,
    g [T][k] float64), ids in rank order."""
    s = sigmoid_scores(logits)
    T, E = s.shape
    ids = np.zeros((T, k), dtype=np.int64)
    g = np.zeros((T, k), dtype=np.float64)
    keys = np.zeros((T, E), dtype=np.float64)
    for t in range(T):
        sel, key = group_limited_topk(s[t], bias, n_group, topk_group, k)
        ids[t] = sel
        g[t] = gate_weights(s[t], sel)
        keys[t] = key
    return s, keys, ids, g
