"""Shared helpers of the GPU parity tests: run a layer through the C ABI and
through the fp64 oracle on the same seeded inputs, and compare."""
from __future__ import annotations

import numpy as np
import torch

import oracle
from paper_2606_29982_amd import caee


def to_dev(a, dev):
    if a is None:
        return None
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).to(dev).view(torch.bfloat16)
    return torch.from_numpy(a).to(dev)


def w_to_dev(W: dict, dev) -> dict:
    return {k: to_dev(v, dev) for k, v in W.items()}


def dev_to_np_bits(t):
    """Device tensor -> numpy in storage encoding (bf16 as uint16 bits)."""
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    if t.dtype == torch.uint8:
        return t.cpu().numpy()
    return t.cpu().numpy()


def getters_np(W: dict, w_dtype: str):
    def get(e):
        return oracle.expert_weights_f64(W["w13"][e], W["w2"][e], w_dtype,
                                         W.get("w13_scale", [None] * (e + 1))[e],
                                         W.get("w2_scale", [None] * (e + 1))[e])

    def get_sh(s):
        return oracle.expert_weights_f64(W["sh_w13"][s], W["sh_w2"][s], w_dtype,
                                         W.get("sh_w13_scale", [None] * (s + 1))[s],
                                         W.get("sh_w2_scale", [None] * (s + 1))[s])
    return get, get_sh


def getters_dev(Wd: dict, w_dtype: str):
    """Oracle weight getters reading one expert at a time from device tensors."""
    def fetch(prefix, i):
        w13 = dev_to_np_bits(Wd[prefix + "w13"][i])
        w2 = dev_to_np_bits(Wd[prefix + "w2"][i])
        s13 = Wd[prefix + "w13_scale"][i].cpu().numpy() if prefix + "w13_scale" in Wd else None
        s2 = Wd[prefix + "w2_scale"][i].cpu().numpy() if prefix + "w2_scale" in Wd else None
        return oracle.expert_weights_f64(w13, w2, w_dtype, s13, s2)
    return (lambda e: fetch("", e)), (lambda s: fetch("sh_", s))


def oracle_layer(shape, inp, tau, n_bins, get=None, get_sh=None, tokens=None, with_y=True, rule="max",
                 refill="score", seed=0, keep_top1=False):
    T = inp.logits.shape[0]
    # the C ABI carries tau and the routed scaling as fp32
    ref = oracle.moe_layer_ref(
        E=shape.E, n_group=shape.n_group, topk_group=shape.topk_group, k=shape.k,
        routed_scaling=float(np.float32(shape.routed_scaling)), tau=float(np.float32(tau)),
        n_bins=n_bins, logits=inp.logits, rule=rule,
        bias=inp.bias, cost=inp.cost, bins=inp.bins if n_bins > 1 else None,
        x=inp.x if with_y else None, x_dtype=shape.x_dtype, w_dtype=shape.w_dtype,
        n_shared=shape.n_shared, get_expert=get if with_y else None, get_shared=get_sh,
        tokens=tokens if tokens is not None else (list(range(T)) if with_y else None), refill=refill, seed=seed,
        keep_top1=keep_top1)
    if T > 0:
        ref["margins"] = oracle.decision_margins(ref, n_group=shape.n_group, topk_group=shape.topk_group,
                                                 k=shape.k, tau=float(np.float32(tau)), rule=rule)
    return ref


def gpu_layer(shape, inp, tau, n_bins, Wd, dev, route_only=False, rule="max", refill="score", seed=0,
              keep_top1=False):
    """Run caee_moe_layer (or caee_route_prune) and return numpy results."""
    T = inp.logits.shape[0]
    layer = caee.Layer.from_shape(shape, T=T, tau=tau, n_bins=n_bins, importance=rule, refill=refill, seed=seed,
                                  keep_top1=keep_top1)
    ws = caee.alloc_workspace(layer, dev)
    out = caee.alloc_route_out(layer, dev)
    logits = to_dev(inp.logits, dev)
    bias = to_dev(inp.bias, dev)
    cost = to_dev(inp.cost, dev)
    bins = to_dev(inp.bins, dev) if n_bins > 1 else None
    res = {}
    if route_only:
        caee.route_prune(layer, logits, bias, cost, bins, out, ws)
    else:
        ydt = torch.float32 if shape.y_dtype == "f32" else torch.bfloat16
        # guard bands around y catch writes outside it
        yfull = torch.full((T + 2, shape.d), 7.0, dtype=ydt, device=dev)
        y = yfull[1:T + 1]
        caee.moe_layer(layer, to_dev(inp.x, dev), logits, bias, cost, bins, Wd, y, ws, out)
        torch.cuda.synchronize()
        assert torch.all(yfull[0] == 7.0) and torch.all(yfull[T + 1] == 7.0), "write outside y"
        res["y"] = y.float().cpu().numpy().astype(np.float64)
    torch.cuda.synchronize()
    for k_, v in out.items():
        res[k_] = v.cpu().numpy()
    return res


def unpack_masks(words: np.ndarray, E: int):
    w = words.astype(np.int64) & 0xFFFFFFFF
    bits = ((w[:, :, None] >> np.arange(32)) & 1).reshape(4, -1)[:, :E].astype(bool)
    return dict(act=bits[0], must=bits[1], trans=bits[2], pruned=bits[3])


NEAR_TIE = 1e-9   # a float64 decision margin below this is a near-tie (two correct results may differ)


def check_route(got, ref, E):
    mg = ref.get("margins")
    if mg is not None:
        print("  decision margins: " + ", ".join(f"{k_} {v:.2e}" for k_, v in mg.items()), flush=True)
    tie = "" if mg is None or mg["min"] >= NEAR_TIE else f" (near-tie: smallest decision margin {mg['min']:.2e})"
    assert np.array_equal(got["orig_ids"], ref["orig_ids"]), "K_t differs" + tie
    m = unpack_masks(got["masks"], E)
    for name in ("act", "must", "trans", "pruned"):
        assert np.array_equal(m[name], ref[name]), f"{name} set differs" + tie
    assert np.array_equal(got["topk_ids"], ref["topk_ids"]), "K_final differs" + tie
    st = ref["stats"]
    want = [st["n_act"], st["n_must"], st["n_cand"], st["n_promoted"], st["n_pruned"], st["n_trans"],
            st["n_refill"], st["n_pad"], st["fallback"]]
    assert got["stats"].tolist() == want, (got["stats"].tolist(), want)
    loads = got["bin_loads"]
    assert np.array_equal(loads[0], ref["act_loads"])
    assert np.array_equal(loads[1], ref["must_loads"])
    assert np.array_equal(loads[2], ref["trans_loads"])
    np.testing.assert_allclose(got["topk_w"], ref["topk_w"], rtol=1e-6, atol=1e-7)


def check_y(y_got, y_ref, rel_tol):
    err = np.abs(y_got - y_ref).max()
    scale = np.abs(y_ref).max()
    assert err <= rel_tol * scale, f"max|err| {err:.4e} > {rel_tol} * max|ref| {scale:.4e}"
    return err / scale


def run_offload_sequence(shape, calls, Wl, dev, n_cache, n_stage, fetch_batch, tau, rule, miss_cost,
                         get, get_sh, y_tokens=None, y_tol=None):
    """Runs ``calls`` through one caee_offload handle (weights ``Wl`` on the
    device, in their layout, copied to pinned host memory for it) and checks
    every call against the oracle's LRU sequence and against caee_moe_layer
    given the same residency cost table.  ``y_tokens(i)`` names the tokens
    whose output the oracle evaluates at call i (None: none)."""
    import dataclasses

    from oracle import offload as off

    T = calls[0].logits.shape[0]
    layer = caee.Layer.from_shape(shape, T=T, tau=tau, n_bins=1, importance=rule)
    host = caee.pin_host_weights(Wl)
    slot13, slot2 = caee.alloc_slots(layer, n_cache + n_stage, dev)
    h = caee.Offload(layer, host["w13"], host["w2"], slot13, slot2, Wl.get("sh_w13"), Wl.get("sh_w2"),
                     n_cache, n_stage, miss_cost, fetch_batch, Wl.get("layout", caee.LAYOUT_ROWMAJOR))
    ws = caee.alloc_workspace(layer, dev)
    ws2 = caee.alloc_workspace(layer, dev)
    out = caee.alloc_route_out(layer, dev)
    out2 = caee.alloc_route_out(layer, dev)
    ydt = torch.float32 if shape.y_dtype == "f32" else torch.bfloat16
    want = {"hits": 0, "misses": 0, "staged": 0, "evictions": 0, "needed": 0}

    def route(i, cost):
        toks = y_tokens(i) if y_tokens else None
        inp = dataclasses.replace(calls[i], cost=cost)
        return oracle_layer(shape, inp, tau, 1, get, get_sh, tokens=toks, with_y=bool(toks), rule=rule)

    try:
        for i, step in enumerate(off.offload_sequence(route, shape.E, n_cache, miss_cost, len(calls))):
            inp = calls[i]
            print(f"offload call {i}: T={T} tau={tau} rule={rule} n_cache={n_cache} n_stage={n_stage} "
                  f"batch={fetch_batch}", flush=True)
            x, logits, bias = to_dev(inp.x, dev), to_dev(inp.logits, dev), to_dev(inp.bias, dev)
            yfull = torch.full((T + 2, shape.d), 7.0, dtype=ydt, device=dev)
            h(layer, x, logits, bias, yfull[1:T + 1], ws, out)
            # the same call through caee_moe_layer with the same cost table
            y2 = torch.empty((T, shape.d), dtype=ydt, device=dev)
            caee.moe_layer(layer, x, logits, bias, to_dev(step["cost"], dev), None, Wl, y2, ws2, out2)
            torch.cuda.synchronize()
            assert torch.all(yfull[0] == 7.0) and torch.all(yfull[T + 1] == 7.0), "write outside y"
            got = {k: v.cpu().numpy() for k, v in out.items()}
            check_route(got, step["ref"], shape.E)
            assert torch.equal(yfull[1:T + 1], y2), "offloaded layer differs from caee_moe_layer"
            for k_ in out:
                assert torch.equal(out[k_], out2[k_]), k_
            assert set(np.flatnonzero(h.residency() >= 0).tolist()) == step["resident_after"]
            lru = step["lru"]
            want["hits"] += len(lru["hits"])
            want["misses"] += len(lru["cached"]) + len(lru["staged"])
            want["staged"] += len(lru["staged"])
            want["evictions"] += len(lru["evicted"])
            want["needed"] += len(lru["hits"]) + len(lru["cached"]) + len(lru["staged"])
            if y_tokens and y_tokens(i):
                toks = y_tokens(i)
                y_got = yfull[1:T + 1].float().cpu().numpy().astype(np.float64)[toks]
                rel = check_y(y_got, step["ref"]["y"], y_tol)
                print(f"  y of {len(toks)} tokens: max|err|/max|ref| = {rel:.3e}", flush=True)
        st = h.stats()
        for k_, v in want.items():
            assert st[k_] == v, (k_, st[k_], v)
        assert st["calls"] == len(calls)
        wbytes = 3 * shape.f * shape.d * (4 if shape.w_dtype == "f32" else 2)
        assert st["bytes_h2d"] == want["misses"] * wbytes
        return st
    finally:
        h.close()
