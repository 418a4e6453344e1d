"""Benchmark of the CAEE MoE-layer hot path on one MI355X.

One step = one full layer call (caee_moe_layer: routing, cost-aware
pruning, compensation, grouped SwiGLU expert FFN, combine) on a resident
batch of synthetic DeepSeek-R1-shaped inputs: d=7168, f=2048, 256 routed
experts in 8 groups (top-4 groups, top-8 experts), 1 shared expert, bf16
weights drawn N(0, 0.02), sigmoid router with bias, routed scaling 2.5.
The headline workload is a decode batch of T=32 tokens with pruning off
(the dense-routing baseline).  Prints one JSON line.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-sweep] [--no-cpu] [--copy-bytes N]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E, published
FP8_PEAK_TFLOPS = 5000.0        # MI355X dense fp8 MFMA, published
W_EXPERT_BYTES = 3 * 7168 * 2048 * 2
W_EXPERT_BYTES_FP8 = 3 * 7168 * 2048 + 4 * (2 * 2048 // 128) * (7168 // 128) + 4 * (7168 // 128) * (2048 // 128)
PAIR_FLOPS = 6 * 7168 * 2048    # one (token, expert) pair through gate, up and down
METRIC = "MoE-layer tokens/s + achieved HBM GB/s (% of peak) at T=1..128, with vs without pruning"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gate_up_deepseek_r1_t32_traffic.json")
# The gate/up kernel's source and the header holding its tuning constants:
# a traffic figure holds only for the build they describe.
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2606_29982_amd", "csrc", n)
                  for n in ("ffn.hip", "ffn_tile.h", "caee_internal.h")]


# MFMA counters of the 8-bit prefill launches at T=4096, for the build of
# these sources.
MFMA_FILE = os.path.join(ROOT, "profiles", "prefill8_deepseek_r1_t4096_mfma.json")
PREFILL_SOURCES = [os.path.join(ROOT, "paper_2606_29982_amd", "csrc", n)
                   for n in ("ffn_prefill8.hip", "fp8_codec.h", "caee_internal.h")]


def kernel_sources_sha256(paths=None):
    h = hashlib.sha256()
    for path in paths or KERNEL_SOURCES:
        with open(path, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def mfma_counter_entry():
    """MFMA busy share of the prefill launches (matrix-pipe busy cycles over
    SIMD cycles) from a committed rocprofv3 counter run, or None when missing
    or taken on a different kernel source."""
    try:
        with open(MFMA_FILE) as fh:
            rec = json.load(fh)
        if rec.get("sources_sha256") != kernel_sources_sha256(PREFILL_SOURCES):
            return None
        return {k: rec[k] for k in ("gate_up", "down")}
    except (OSError, ValueError, KeyError):
        return None


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--T", type=int, default=32)
    ap.add_argument("--no-sweep", action="store_true")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-offload", action="store_true")
    ap.add_argument("--no-calibrate", action="store_true")
    ap.add_argument("--offload-calls", type=int, default=256,
                    help="decode calls of the offloading sequence (T=16 each)")
    ap.add_argument("--case", default=None,
                    help="time one configuration only, DTYPE:T[:skewed] (e.g. bf16:128:skewed, fp8:4096), "
                         "and print its line instead of the headline")
    ap.add_argument("--graph", action="store_true",
                    help="with --case: also time single graph replays after a cache flush, and print them")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="finish with one device-to-device copy of this many bytes (a known-size "
                         "reference for HBM traffic counters)")
    return ap.parse_args()


def log(msg):
    print(msg, file=sys.stderr, flush=True)


class Case:
    """Device-resident inputs and buffers of one layer call."""

    def __init__(self, shape, T, tau, n_bins, W, dev, seed, skewed, rule="max", cost_kind=None):
        import torch
        from paper_2606_29982_amd import caee
        from synth_inputs import make_routing_inputs
        if cost_kind is None:
            cost_kind = "zipf" if skewed else "flat"
        self.inp = make_routing_inputs(shape, seed=seed, T=T, zipf_logit_s=1.1 if skewed else None,
                                       cost_kind=cost_kind, n_bins=n_bins)
        self.layer = caee.Layer.from_shape(shape, T=T, tau=tau, n_bins=n_bins, importance=rule)
        to = lambda a: None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(dev)  # noqa: E731
        self.x = torch.from_numpy(self.inp.x.view(np.int16)).to(dev).view(torch.bfloat16)
        self.logits = to(self.inp.logits)
        self.bias = to(self.inp.bias)
        self.cost = to(self.inp.cost)
        self.bins = to(self.inp.bins) if n_bins > 1 else None
        self.W = W
        self.y = torch.empty((T, shape.d), dtype=torch.bfloat16, device=dev)
        self.T = T
        self.ws = caee.alloc_workspace(self.layer, dev)
        self.out = caee.alloc_route_out(self.layer, dev)
        self.caee = caee

    def step(self):
        self.caee.moe_layer(self.layer, self.x, self.logits, self.bias, self.cost, self.bins, self.W,
                            self.y, self.ws, self.out)

    def stats(self):
        return self.out["stats"].cpu().numpy().tolist()

    def routed_pairs(self):
        return int((self.out["topk_ids"] >= 0).sum().item())


def time_steps(case, steps, warmup):
    import torch
    for _ in range(warmup):
        case.step()
    torch.cuda.synchronize()
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(steps):
        case.step()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / steps


def graph_protocol(case, warmup=10, iters=50, flush_mb=512):
    """The layer call captured once in a HIP graph and replayed: `warmup`
    replays, then `iters` replays each timed on its own with events, with the
    caches flushed before each one (outside the timed region) in two ways:
      * "write": a `flush_mb` MB buffer is written, so that the 256 MB
        memory-side cache holds nothing of the previous call -- but it then
        holds the flush's own dirty lines, which the timed call has to write
        back to HBM as it streams its weights;
      * "clean": the same write, then a second `flush_mb` MB buffer is read,
        which evicts those dirty lines (written back before the timed call):
        the call starts from caches that hold neither its data nor dirty
        lines.
    A third series runs the same flushed single calls eagerly (the layer's
    launches issued one by one, no graph), the clean flush before each.
    Returns the median and the 10th / 90th percentiles of all three, in us."""
    import torch
    case.step()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        case.step()
    for _ in range(warmup):
        g.replay()
    flush = torch.empty(flush_mb << 20, dtype=torch.uint8, device=case.y.device)
    rd = torch.ones(flush_mb << 17, dtype=torch.int64, device=case.y.device)
    res = {"iters": iters, "warmup": warmup, "flush_mb": flush_mb}
    for mode in ("write", "clean"):
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(iters)]
        for a, b in ev:
            flush.fill_(1)
            if mode == "clean":
                rd.sum()
            a.record()
            g.replay()
            b.record()
        torch.cuda.synchronize()
        us = np.array([a.elapsed_time(b) * 1e3 for a, b in ev])
        key = "" if mode == "clean" else "_write_flush"
        res["us_p50" + key] = round(float(np.median(us)), 1)
        res["us_p10" + key] = round(float(np.percentile(us, 10)), 1)
        res["us_p90" + key] = round(float(np.percentile(us, 90)), 1)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(iters)]
    for a, b in ev:
        flush.fill_(1)
        rd.sum()
        a.record()
        case.step()
        b.record()
    torch.cuda.synchronize()
    us = np.array([a.elapsed_time(b) * 1e3 for a, b in ev])
    res["us_p50_eager"] = round(float(np.median(us)), 1)
    res["us_p10_eager"] = round(float(np.percentile(us, 10)), 1)
    res["us_p90_eager"] = round(float(np.percentile(us, 90)), 1)
    del g, flush, rd
    return res


def layer_bytes(shape, T, n_trans):
    """Algorithmic HBM bytes of one layer call: weights of every executed
    expert (A_trans plus the shared one), x read, y written, router logits,
    bias/cost/bin tables."""
    return ((n_trans + shape.n_shared) * W_EXPERT_BYTES + T * shape.d * 2 * 2
            + T * shape.E * 4 + 12 * shape.E)


def gate_up_bytes(shape, T, n_experts, rows):
    """Algorithmic bytes of one gate/up launch: the gate and up matrices of
    the experts it runs, x read once, the bf16 SwiGLU rows written."""
    return n_experts * 2 * shape.f * shape.d * 2 + T * shape.d * 2 + rows * shape.f * 2


def traffic_entry():
    """HBM traffic of the gate/up kernel from committed rocprofv3 counter
    runs, or None when missing or taken on a different kernel source."""
    try:
        with open(TRAFFIC_FILE) as fh:
            rec = json.load(fh)
        if rec.get("sources_sha256") != kernel_sources_sha256():
            return None
        return rec.get("bytes_per_launch")
    except (OSError, ValueError):
        return None


def cpu_baseline(shape, case, W, sample_tokens):
    """The fp64 oracle on the host cores: routing + pruning + compensation of
    the whole batch and the expert FFN of ``sample_tokens`` tokens."""
    import torch
    import oracle
    try:
        from threadpoolctl import threadpool_info
        blas = threadpool_info()
        cores = max([int(i.get("num_threads", 1)) for i in blas] or [1])
        vendor = ",".join(sorted({i.get("internal_api", "?") for i in blas}))
    except Exception:
        cores, vendor = len(os.sched_getaffinity(0)), "unknown"
    inp = case.inp
    ref = oracle.moe_layer_ref(E=shape.E, n_group=shape.n_group, topk_group=shape.topk_group, k=shape.k,
                               routed_scaling=shape.routed_scaling, tau=case.layer.tau,
                               n_bins=case.layer.n_bins, logits=inp.logits, bias=inp.bias, cost=inp.cost,
                               bins=inp.bins)
    tokens = list(range(sample_tokens))
    need = sorted({int(e) for t in tokens for e in ref["topk_ids"][t] if e >= 0})
    host = {}
    for e in need:   # stage the stored bf16 weights in host memory (not timed)
        host[e] = (W["w13"][e].view(torch.int16).cpu().numpy().view(np.uint16),
                   W["w2"][e].view(torch.int16).cpu().numpy().view(np.uint16))
    sh = (W["sh_w13"][0].view(torch.int16).cpu().numpy().view(np.uint16),
          W["sh_w2"][0].view(torch.int16).cpu().numpy().view(np.uint16))
    t0 = time.perf_counter()
    oracle.moe_layer_ref(
        E=shape.E, n_group=shape.n_group, topk_group=shape.topk_group, k=shape.k,
        routed_scaling=shape.routed_scaling, tau=case.layer.tau, n_bins=case.layer.n_bins,
        logits=inp.logits, bias=inp.bias, cost=inp.cost, bins=inp.bins, x=inp.x, x_dtype="bf16",
        w_dtype="bf16", n_shared=shape.n_shared,
        get_expert=lambda e: oracle.expert_weights_f64(host[e][0], host[e][1], "bf16"),
        get_shared=lambda s: oracle.expert_weights_f64(sh[0], sh[1], "bf16"), tokens=tokens)
    dt = time.perf_counter() - t0
    return {"value": round(sample_tokens / dt, 4), "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "sample": (f"fp64 numpy oracle ({vendor} BLAS): routing, pruning and compensation of all "
                       f"{case.layer.T} tokens plus the expert FFN of {sample_tokens} of them "
                       f"({len(need)} routed experts + 1 shared), {dt:.1f} s"),
            "seconds": round(dt, 2)}


def pinned_h2d_gbps(dev, nbytes, reps=8, n_streams=3):
    """Peak host-to-device bandwidth of page-locked memory: one expert-sized
    copy repeated on a stream, timed with events, best of `n_streams`
    streams (the copy runtime can put one stream's copies of a given size on
    a half-rate path)."""
    import torch
    src = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
    src.fill_(1)
    dst = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    best = 0.0
    for _ in range(n_streams):
        s = torch.cuda.Stream(device=dev)
        with torch.cuda.stream(s):
            dst.copy_(src, non_blocking=True)
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(s)
            for _ in range(reps):
                dst.copy_(src, non_blocking=True)
            b.record(s)
        b.synchronize()
        best = max(best, reps * nbytes / (a.elapsed_time(b) * 1e-3) / 1e9)
    del src, dst
    return best


def offload_rows(args, shape, Wt, dev, link_model=None):
    """The offloading deployment: all 256 bf16 experts in page-locked host
    memory, a 64-expert LRU device cache plus a 16-slot staging ring, misses
    copied on a side stream while resident experts compute.  A sequence of
    T=16 decode calls with Zipf(1.2) expert popularity, cache cold at the
    start, for several pruning thresholds."""
    import torch
    from paper_2606_29982_amd import caee
    from synth_inputs import make_call_sequence

    T, n_cache, n_stage, batch = 16, 64, 16, 4
    t0 = time.time()
    host = caee.pin_host_weights(Wt)
    torch.cuda.synchronize()
    log(f"offload: experts copied to page-locked host memory in {time.time() - t0:.1f}s")
    b_pcie = pinned_h2d_gbps(dev, W_EXPERT_BYTES)
    if link_model is not None:      # calibrated alpha * S / B + beta
        miss_us = float(link_model.cost_us(W_EXPERT_BYTES))
    else:                           # alpha = 1, beta = 0 at the measured peak
        miss_us = W_EXPERT_BYTES / (b_pcie * 1e9) * 1e6
    log(f"offload: pinned H2D peak {b_pcie:.1f} GB/s, miss cost {miss_us:.0f} us per expert")
    calls = make_call_sequence(shape, seed=args.seed + 5, n_calls=args.offload_calls, T=T, zipf_logit_s=1.2)
    dev_calls = [(torch.from_numpy(c.x.view(np.int16)).to(dev).view(torch.bfloat16),
                  torch.from_numpy(c.logits).to(dev), torch.from_numpy(c.bias).to(dev)) for c in calls]
    rows = []
    # MAX rule at the workload's thresholds, then the offloading rule of the
    # paper (cumulative importance ratio) at its three retention thresholds.
    for rule, tau in (("max", 0.0), ("max", 0.05), ("max", 0.1), ("cir", 0.9), ("cir", 0.8), ("cir", 0.7)):
        layer = caee.Layer.from_shape(shape, T=T, tau=tau, n_bins=1, importance=rule)
        s13, s2 = caee.alloc_slots(layer, n_cache + n_stage, dev)
        h = caee.Offload(layer, host["w13"], host["w2"], s13, s2, Wt["sh_w13"], Wt["sh_w2"], n_cache, n_stage,
                         miss_us, batch, caee.LAYOUT_TILED)
        ws = caee.alloc_workspace(layer, dev)
        out = caee.alloc_route_out(layer, dev)
        y = torch.empty((T, shape.d), dtype=torch.bfloat16, device=dev)
        acc = torch.zeros(caee.STATS, dtype=torch.int64, device=dev)
        for x, logits, bias in dev_calls[:4]:        # warm-up, then a cold cache
            h(layer, x, logits, bias, y, ws, out)
        torch.cuda.synchronize()
        h.reset()
        t1 = time.perf_counter()
        for x, logits, bias in dev_calls:
            h(layer, x, logits, bias, y, ws, out)
            acc += out["stats"]
        torch.cuda.synchronize()
        wall = time.perf_counter() - t1
        st = h.stats()
        a = acc.cpu().tolist()
        n = len(dev_calls)
        gbps = st["bytes_h2d"] / wall / 1e9
        rows.append({"T": T, "calls": n, "tau": tau, "rule": rule, "n_bins": 1, "cache_slots": n_cache,
                     "staging_slots": n_stage, "fetch_batch": batch,
                     "tokens_per_s": round(T * n / wall, 1), "ms_per_call": round(wall / n * 1e3, 3),
                     "h2d_gbps": round(gbps, 2), "h2d_peak_gbps": round(b_pcie, 2),
                     "h2d_frac": round(gbps / b_pcie, 4),
                     "hit_rate": round(st["hits"] / max(st["needed"], 1), 4),
                     "fetched_per_call": round(st["misses"] / n, 2), "staged_per_call": round(st["staged"] / n, 2),
                     "act_per_call": round(a[0] / n, 2), "pruned_per_call": round(a[4] / n, 2),
                     "executed_per_call": round(st["needed"] / n + shape.n_shared, 2)})
        log(f"offload {rows[-1]}")
        h.close()
        del s13, s2, ws
        torch.cuda.empty_cache()
    del host
    return {"b_pcie_gbps": round(b_pcie, 2), "miss_cost_us": round(miss_us, 1),
            "miss_cost_source": "calibrated" if link_model is not None else "measured peak", "rows": rows}


def known_copy(args, dev):
    """One device-to-device copy of --copy-bytes bytes: a kernel of known
    traffic that calibrates the profiler's HBM byte counters."""
    import torch
    if args.copy_bytes > 0:
        src = torch.empty(args.copy_bytes, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst


def run_case(args, dev):
    """One configuration (e.g. for a profiler run): the sweep's inputs for
    bf16 (Zipf-skewed when asked, 8 bins, no pruning) or the 8-bit rows'
    inputs (tau 0.05, 8 bins), timed over --steps calls."""
    import torch
    from paper_2606_29982_amd import caee
    from synth_inputs import R1_BF16, R1_FP8, make_expert_weights_torch
    parts = args.case.split(":")
    dtype, T = parts[0], int(parts[1])
    skewed = len(parts) > 2 and parts[2] == "skewed"
    shape = {"bf16": R1_BF16, "fp8": R1_FP8}[dtype]
    W = caee.pack_weights(make_expert_weights_torch(shape, seed=args.seed, device=dev), dtype)
    torch.cuda.synchronize()
    tau = 0.0 if dtype == "bf16" else 0.05
    c = Case(shape, T, tau, 8, W, dev, args.seed, skewed=skewed, cost_kind="zipf")
    ms = time_steps(c, args.steps, args.warmup)
    s = c.stats()
    b = (s[5] + shape.n_shared) * (W_EXPERT_BYTES if dtype == "bf16" else W_EXPERT_BYTES_FP8)
    line = {"case": args.case, "us_per_step": round(ms * 1e3, 1), "tokens_per_s": round(T / (ms * 1e-3), 1),
            "weight_gbps": round(b / (ms * 1e-3) / 1e9, 1), "executed": s[5] + shape.n_shared,
            "steps": args.steps, "warmup": args.warmup}
    if args.graph:
        gp = graph_protocol(c)
        line["graph_protocol"] = gp
        line["weight_frac_flushed"] = round(b / (gp["us_p50"] * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4)
        line["weight_frac_flushed_eager"] = round(b / (gp["us_p50_eager"] * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4)
    print(json.dumps(line), flush=True)


def ablation_rows(args, shape, Wt, dev):
    """Compensation ablation, a synthetic stand-in for the paper's comparison
    of random selection with its compensation: an offloading-style layer
    (the 32 most popular experts resident at cost 0, the others at cost 1,
    one bin, the CIR rule) pruned at theta_imp 0.9 / 0.8 / 0.7, and the
    relative output error ||y - y_dense|| / ||y_dense|| against the same
    layer without pruning, for the paper's score-based refill, a random
    refill (mean of 4 seeds), no refill (renormalise only) and the literal
    top-k of the masked router keys (which can also replace a token's own
    surviving experts; its row also reports its error at tau = 0).  With random
    expert weights a refilled expert's output is uncorrelated with the one it
    replaces, so this measures how far each variant moves the output, not
    the task accuracy the paper reports."""
    import torch
    from paper_2606_29982_amd import caee
    from synth_inputs import make_call_sequence, popularity_ranks
    ranks = popularity_ranks(shape, args.seed + 9)
    cost = torch.from_numpy(np.where(ranks < 32, 0.0, 1.0).astype(np.float32)).to(dev)
    rows = []
    for T in (8, 32, 128):
        c = make_call_sequence(shape, seed=args.seed + 9, n_calls=1, T=T, zipf_logit_s=1.2)[0]
        x = torch.from_numpy(c.x.view(np.int16)).to(dev).view(torch.bfloat16)
        logits = torch.from_numpy(c.logits).to(dev)
        bias = torch.from_numpy(c.bias).to(dev)

        def run(tau, refill="score", seed=0, rule="cir"):
            layer = caee.Layer.from_shape(shape, T=T, tau=tau, n_bins=1, importance=rule, refill=refill, seed=seed)
            ws = caee.alloc_workspace(layer, dev)
            out = caee.alloc_route_out(layer, dev)
            y = torch.empty((T, shape.d), dtype=torch.bfloat16, device=dev)
            caee.moe_layer(layer, x, logits, bias, cost, None, Wt, y, ws, out)
            return y.float(), out["stats"].cpu().tolist()

        y0, _ = run(0.0, rule="max")      # tau = 0: nothing pruned
        n0 = float(torch.linalg.norm(y0))
        lit0 = float(torch.linalg.norm(run(0.0, "literal", rule="max")[0] - y0)) / n0
        for theta in (0.9, 0.8, 0.7):
            errs = {}
            st = None
            for mode in ("score", "none", "literal"):
                y, st_m = run(theta, mode)
                errs[mode] = float(torch.linalg.norm(y - y0)) / n0
                st = st if st is not None else st_m
            rnd = [float(torch.linalg.norm(run(theta, "random", sd)[0] - y0)) / n0 for sd in range(4)]
            errs["random"] = float(np.mean(rnd))
            rows.append({"T": T, "theta_imp": theta, "pruned": st[4], "refilled_slots": st[6],
                         "rel_err_score": round(errs["score"], 5), "rel_err_random": round(errs["random"], 5),
                         "rel_err_none": round(errs["none"], 5), "rel_err_literal": round(errs["literal"], 5),
                         "rel_err_literal_tau0": round(lit0, 5)})
            log(f"ablation {rows[-1]}")
    return rows


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU; --gpus {args.gpus} is not supported "
              "(the layer is measured on one MI355X; multi-GPU sharding is not built)", file=sys.stderr)
        sys.exit(2)
    if args.case:
        import torch
        run_case(args, torch.device("cuda:0"))
        known_copy(args, torch.device("cuda:0"))
        return
    import torch
    from paper_2606_29982_amd import caee
    from synth_inputs import R1_BF16, make_expert_weights_torch

    dev = torch.device("cuda:0")
    shape = R1_BF16
    t0 = time.time()
    log("drawing R1-shaped bf16 expert weights on the device")
    W = make_expert_weights_torch(shape, seed=args.seed, device=dev)
    # the kernels stream the tiled layout; the row-major copy feeds the oracle
    Wt = caee.pack_weights(W, "bf16")
    torch.cuda.synchronize()
    log(f"weights ready in {time.time() - t0:.1f}s")

    # Headline: T=32 decode batch, pruning off.
    head = Case(shape, args.T, 0.0, 1, Wt, dev, args.seed, skewed=False)
    ms = time_steps(head, args.steps, args.warmup)
    st = head.stats()
    n_trans = st[5]
    rows = args.T * shape.k + args.T * shape.n_shared
    # Per-kernel durations over a second timed region with library events on.
    caee.timing_reset()
    caee.timing_enable(True)
    ms_ev = time_steps(head, args.steps, 0)
    # Per step: summed duration and number of launches of each kernel kind.
    kern, launches = {}, {}
    for kind in caee.KERNEL_KINDS:
        tot, n = caee.timing_query(kind)
        kern[kind] = tot / args.steps
        launches[kind] = n / args.steps
    caee.timing_enable(False)
    caee.timing_reset()
    log(f"T={args.T}: {ms * 1e3:.1f} us/step ({ms_ev * 1e3:.1f} with kernel events); kernels (us per step): "
        + ", ".join(f"{k} {v * 1e3:.1f} ({launches[k]:.0f} launches)" for k, v in kern.items()))

    b_layer = layer_bytes(shape, args.T, n_trans)
    # The gate/up launch of the routed and shared experts.
    n_gu = max(int(round(launches["gate_up"])), 1)
    gu_rows = args.T * (shape.k + shape.n_shared)
    gu_bytes = gate_up_bytes(shape, args.T, n_trans + shape.n_shared, gu_rows)
    gu_bytes += (n_gu - 1) * args.T * shape.d * 2   # every launch reads x once
    gu_gbps = gu_bytes / (kern["gate_up"] * 1e-3) / 1e9
    traffic = traffic_entry()
    roofline = {"kernel": "k_gate_up (expert gate/up + SwiGLU)", "bound": "hbm",
                "achieved": round(gu_gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": round(gu_gbps / HBM_PEAK_GBPS, 4), "traffic": traffic,
                "launches_per_step": n_gu, "bytes_per_launch": round(gu_bytes / n_gu),
                "avg_launch_us": round(kern["gate_up"] / n_gu * 1e3, 2)}
    result = {
        "metric": METRIC, "value": round(args.T / (ms * 1e-3), 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "deepseek-r1-moe-layer-bf16-decode", "T": args.T, "d": shape.d, "f": shape.f,
                   "E": shape.E, "n_group": shape.n_group, "topk_group": shape.topk_group, "k": shape.k,
                   "n_shared": shape.n_shared, "tau": 0.0, "pruning": "off", "weight_layout": "tiled",
                   "parallelism": "single-gpu"},
        "hbm_gbps": round(b_layer / (ms * 1e-3) / 1e9, 1),
        "hbm_frac": round(b_layer / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
        "experts_executed": n_trans + shape.n_shared,
        "kernel_us_per_step": {k: round(v * 1e3, 2) for k, v in kern.items()},
        "roofline": roofline,
    }
    # The same call captured in a HIP graph, memory-side cache flushed before
    # every timed replay (median and spread of single calls).
    result["graph_protocol"] = graph_protocol(head)
    gp = result["graph_protocol"]
    result["hbm_frac_flushed"] = round(b_layer / (gp["us_p50"] * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4)
    result["hbm_frac_flushed_write"] = round(b_layer / (gp["us_p50_write_flush"] * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4)
    result["hbm_frac_flushed_eager"] = round(b_layer / (gp["us_p50_eager"] * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4)
    log(f"graph protocol {result['graph_protocol']}")

    link_model = None
    if not args.no_calibrate:
        # Offline cost calibration (alpha, beta of both data paths), before the
        # sweeps: run after them (and the 8-bit rows and the ablation), this
        # process's 42 MB host copies took twice their time.
        from paper_2606_29982_amd import calibrate as cal
        cres = cal.calibrate(dev)
        link_model = cres["link"]
        result["calibration"] = {
            "hbm": {**cres["hbm"].as_dict(), "expert_cost_us": round(float(cres["hbm"].cost_us(W_EXPERT_BYTES)), 2)},
            "h2d": {**cres["link"].as_dict(), "expert_cost_us": round(float(cres["link"].cost_us(W_EXPERT_BYTES)), 1)},
            "samples": cres["samples"]}
        log(f"calibration {result['calibration']}")

    if not args.no_sweep:
        # Zipf-skewed popularity and cost table, experts placed on 8 bins
        # (EP8-style), with and without pruning under each importance rule.
        sweep = []
        for T in (1, 8, 32, 128):
            for rule, tau, n_bins in (("max", 0.0, 8), ("max", 0.1, 8), ("sum", 0.6, 8), ("cir", 0.8, 8)):
                c = Case(shape, T, tau, n_bins, Wt, dev, args.seed, skewed=True, rule=rule)
                m = time_steps(c, max(10, args.steps // 2), 3)
                gp = graph_protocol(c, warmup=5, iters=20)
                s = c.stats()
                b = layer_bytes(shape, T, s[5])
                loads = c.out["bin_loads"].cpu().numpy() / 1e9   # cost units (weight bytes x multiplier), in G
                sweep.append({"T": T, "rule": rule, "tau": tau, "n_bins": n_bins, "inputs": "zipf-skewed",
                              "pruning": "off" if tau == 0.0 else "on",
                              "us_per_step": round(m * 1e3, 1), "tokens_per_s": round(T / (m * 1e-3), 1),
                              "hbm_gbps": round(b / (m * 1e-3) / 1e9, 1),
                              "hbm_frac": round(b / (m * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
                              "act": s[0], "must": s[1], "pruned": s[4], "executed": s[5] + shape.n_shared,
                              "fallback": s[8],
                              "graph_flushed_us_p50": gp["us_p50"], "graph_flushed_us_p10": gp["us_p10"],
                              "graph_flushed_us_p90": gp["us_p90"],
                              "hbm_frac_flushed": round(b / (gp["us_p50"] * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
                              "graph_write_flush_us_p50": gp["us_p50_write_flush"],
                              "hbm_frac_flushed_write": round(b / (gp["us_p50_write_flush"] * 1e-6) / 1e9
                                                              / HBM_PEAK_GBPS, 4),
                              "eager_flushed_us_p50": gp["us_p50_eager"],
                              "hbm_frac_flushed_eager": round(b / (gp["us_p50_eager"] * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
                              "bin_loads_g": {"act": [round(v, 3) for v in loads[0]],
                                              "must": [round(v, 3) for v in loads[1]],
                                              "trans": [round(v, 3) for v in loads[2]]},
                              "f_base_g": round(float(loads[1].max()), 3)})
                log(f"sweep {sweep[-1]}")
                del c
        result["sweep"] = sweep

    if not args.no_sweep:
        # 8-bit expert weights (e4m3, 128x128 block scales), activations
        # quantised per token per 128 channels: decode and prefill, tau=0.05.
        from synth_inputs import R1_FP8
        W8 = caee.pack_weights(make_expert_weights_torch(R1_FP8, seed=args.seed, device=dev), "fp8")
        fp8_rows = []
        for T, steps in ((64, max(10, args.steps // 2)), (4096, 5)):
            c = Case(R1_FP8, T, 0.05, 8, W8, dev, args.seed, skewed=False, cost_kind="zipf")
            m = time_steps(c, steps, 2)
            s = c.stats()
            pairs = c.routed_pairs() + T * R1_FP8.n_shared
            b = (s[5] + R1_FP8.n_shared) * W_EXPERT_BYTES_FP8 + T * R1_FP8.d * 4 + T * R1_FP8.E * 4
            tflops = pairs * PAIR_FLOPS / (m * 1e-3) / 1e12
            fp8_rows.append({"T": T, "tau": 0.05, "n_bins": 8, "rule": "max", "weights": "e4m3 + fp32 128x128 scales",
                             "us_per_step": round(m * 1e3, 1), "tokens_per_s": round(T / (m * 1e-3), 1),
                             "hbm_gbps": round(b / (m * 1e-3) / 1e9, 1),
                             "hbm_frac": round(b / (m * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
                             "mfma_tflops": round(tflops, 1), "mfma_frac": round(tflops / FP8_PEAK_TFLOPS, 4),
                             "executed": s[5] + R1_FP8.n_shared, "pruned": s[4]})
            if T == 4096:
                # matrix-pipe busy share of the two prefill launches, from counters
                fp8_rows[-1]["mfma_busy_counters"] = mfma_counter_entry()
            log(f"fp8 {fp8_rows[-1]}")
            del c
        result["fp8"] = fp8_rows
        del W8
        torch.cuda.empty_cache()

    if not args.no_sweep:
        result["compensation_ablation"] = ablation_rows(args, shape, Wt, dev)

    if link_model is not None and not args.no_sweep:
        # The host link measured again after the sweeps, the 8-bit rows and the
        # ablation: the same copies, to compare with the samples above.
        from paper_2606_29982_amd import calibrate as cal
        ls, lt = cal.measure_link(dev)
        again = cal.fit_link(ls, lt, cal.LINK_GBPS)
        result["calibration"]["h2d_after_sweeps"] = {**again.as_dict(),
                                                     "samples": [(n, round(t, 2)) for n, t in zip(ls, lt)]}
        log(f"host link after the sweeps {result['calibration']['h2d_after_sweeps']}")

    if not args.no_offload:
        result["offload"] = offload_rows(args, shape, Wt, dev, link_model)

    known_copy(args, dev)
    if not args.no_cpu:
        log("timing the fp64 oracle on the host")
        result["cpu_baseline"] = cpu_baseline(shape, head, W, sample_tokens=args.T)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
