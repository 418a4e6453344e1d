"""The whole CAEE MoE layer (oracle, fp64): route, prune, compensate, then
the expert FFN and weighted combine.

Test infrastructure only; see the package docstring.
"""
from __future__ import annotations

import numpy as np

from .compensation import compensate_batch
from .ffn import bf16_bits_to_f64, swiglu_expert
from .pruning import prune_batch
from .routing import route_batch


def decode_x(x, x_dtype: str) -> np.ndarray:
    if x_dtype == "f32":
        return np.asarray(x, np.float64)
    if x_dtype == "bf16":
        return bf16_bits_to_f64(x)
    raise ValueError(x_dtype)


def moe_layer_ref(*, E, n_group, topk_group, k, routed_scaling, tau, n_bins,
                  logits, bias=None, cost, bins=None,
                  x=None, x_dtype="f32", w_dtype="f32", n_shared=0,
                  get_expert=None, get_shared=None, tokens=None, rule="max", refill="score",
                  seed=0, keep_top1=False) -> dict:
    """Run the layer.  Routing/pruning/compensation always run on the whole
    batch (pruning is a batch-level decision).  When ``x`` and the weight
    getters are given, the output rows y_t are computed for ``tokens``
    (default: every token).

    ``get_expert(e)`` / ``get_shared(s)`` return float64 (w13 [2f][d],
    w2 [d][f]) for routed expert e / shared expert s.
    """
    logits = np.asarray(logits, np.float32)
    T = logits.shape[0]
    s, keys, orig_ids, g = route_batch(logits, bias, n_group, topk_group, k)
    pr = prune_batch(orig_ids, g, E, tau, cost, bins, n_bins, rule=rule, s=s, keep_top1=keep_top1)
    ids, w, n_refill = compensate_batch(keys, s, orig_ids, pr["trans"], k, routed_scaling, refill, seed)
    out = dict(s=s, keys=keys, orig_ids=orig_ids, g=g, topk_ids=ids, topk_w=w, **pr)
    out["stats"] = dict(
        n_act=int(pr["act"].sum()), n_must=int(pr["must"].sum()),
        n_cand=int(pr["cand"].sum()), n_promoted=int(pr["promoted"].sum()),
        n_pruned=int(pr["pruned"].sum()), n_trans=int(pr["trans"].sum()),
        n_refill=int(n_refill), n_pad=int((ids < 0).sum()), fallback=int(pr["fallback"]))
    if x is None or get_expert is None:
        return out
    tokens = list(range(T)) if tokens is None else list(tokens)
    xs = decode_x(np.asarray(x)[tokens], x_dtype)
    d = xs.shape[1]
    y = np.zeros((len(tokens), d), dtype=np.float64)
    fp8 = w_dtype == "fp8"
    # Group the requested tokens by expert so each expert is widened once.
    users = {}
    for row, t in enumerate(tokens):
        for slot in range(k):
            e = int(ids[t, slot])
            if e >= 0:
                users.setdefault(e, []).append((row, w[t, slot]))
    for e in sorted(users):
        w13, w2 = get_expert(e)
        rows = [r for r, _ in users[e]]
        ye = swiglu_expert(xs[rows], w13, w2, fp8_acts=fp8)
        for j, (r, wt) in enumerate(users[e]):
            y[r] += wt * ye[j]
    for sh in range(n_shared):
        w13, w2 = get_shared(sh)
        y += swiglu_expert(xs, w13, w2, fp8_acts=fp8)
    out["y"] = y
    out["y_tokens"] = tokens
    return out
