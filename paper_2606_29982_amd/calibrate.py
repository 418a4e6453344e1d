"""Offline cost calibration on the device (Sec. IV-A).

The pruning step takes a per-expert cost table C~(e, d) = alpha_d * S_e / B_d
+ beta_d: the time to bring expert e's S_e bytes through the data path of
device d, whose nominal bandwidth is B_d, with alpha_d the measured
degradation and beta_d a fixed per-expert overhead.  This module measures
both data paths of one MI355X and fits the two constants by least squares:

  * HBM: the expert FFN itself (caee_expert_ffn), one token per expert, for
    several expert sizes (the DeepSeek-R1 hidden size with three
    intermediate sizes) and several expert counts per call; each call is
    modelled as c0 + m * C~(S) (c0: the call's fixed launch and routing-free
    overhead, m experts of S bytes);
  * host link: page-locked host-to-device copies of several sizes.

The fit is numpy least squares on a handful of timings; the timings are of
the library's own kernels and of hipMemcpyAsync.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

HBM_GBPS = 8000.0        # MI355X HBM3E, nominal
LINK_GBPS = 64.0         # PCIe 5.0 x16, nominal per direction


@dataclass
class CostModel:
    """C~(S) = alpha * S / B + beta (microseconds), for one data path."""

    alpha: float
    beta: float
    bandwidth_gbps: float
    r2: float
    c0_us: float = 0.0

    def cost_us(self, nbytes) -> np.ndarray:
        return self.alpha * np.asarray(nbytes, dtype=np.float64) / (self.bandwidth_gbps * 1e3) + self.beta

    def as_dict(self) -> dict:
        return {"alpha": round(self.alpha, 4), "beta_us": round(self.beta, 3),
                "nominal_gbps": self.bandwidth_gbps, "r2": round(self.r2, 5), "c0_us": round(self.c0_us, 2)}


def _lstsq(A: np.ndarray, t: np.ndarray):
    theta, *_ = np.linalg.lstsq(A, t, rcond=None)
    resid = t - A @ theta
    ss = float(np.sum((t - t.mean()) ** 2))
    r2 = 1.0 - float(np.sum(resid ** 2)) / ss if ss > 0 else 1.0
    return theta, r2


def fit_link(sizes_bytes, times_us, bandwidth_gbps: float) -> CostModel:
    """alpha, beta of t = alpha * S / B + beta from (size, time) samples."""
    x = np.asarray(sizes_bytes, dtype=np.float64) / (bandwidth_gbps * 1e3)   # nominal microseconds
    t = np.asarray(times_us, dtype=np.float64)
    if x.size < 2 or np.ptp(x) == 0:
        raise ValueError("at least two distinct sizes are needed")
    theta, r2 = _lstsq(np.stack([x, np.ones_like(x)], axis=1), t)
    return CostModel(float(theta[0]), float(theta[1]), bandwidth_gbps, r2)


def fit_grouped(counts, sizes_bytes, times_us, bandwidth_gbps: float) -> CostModel:
    """alpha, beta (and the per-call c0) of t = c0 + m * (alpha * S / B + beta)."""
    m = np.asarray(counts, dtype=np.float64)
    x = np.asarray(sizes_bytes, dtype=np.float64) / (bandwidth_gbps * 1e3)
    t = np.asarray(times_us, dtype=np.float64)
    theta, r2 = _lstsq(np.stack([m * x, m, np.ones_like(m)], axis=1), t)
    return CostModel(float(theta[0]), float(theta[1]), bandwidth_gbps, r2, float(theta[2]))


def _time_us(fn, reps: int, stream) -> float:
    """Median over `reps` individually timed calls (after one untimed call):
    a one-off stall (first use of a path, an interrupt) does not move it."""
    import torch
    fn()
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    for a, b in ev:
        a.record(stream)
        fn()
        b.record(stream)
    ev[-1][1].synchronize()
    return float(np.median([a.elapsed_time(b) * 1e3 for a, b in ev]))


def measure_link(device, sizes_bytes=(1 << 20, 4 << 20, 16 << 20, 44040192, 88080384), reps: int = 7,
                 n_streams: int = 3):
    """Times (us) of page-locked host-to-device copies of each size: the
    fastest, over `n_streams` streams, of the median of `reps` copies on one
    stream.  The copy runtime picks the copy path per stream and size: on
    one stream a given size can run at half the link rate (about 30 against
    56 GB/s) on every repetition while other sizes run at full rate, and a
    different stream slows a different set of sizes; the calibration wants
    the link, not that choice."""
    import torch
    top = max(sizes_bytes)
    src = torch.empty(top, dtype=torch.uint8, pin_memory=True)
    src.fill_(1)
    dst = torch.empty(top, dtype=torch.uint8, device=device)
    best = [float("inf")] * len(sizes_bytes)
    for _ in range(n_streams):
        s = torch.cuda.Stream(device=device)
        with torch.cuda.stream(s):
            for n in sizes_bytes:                 # warm every size once
                dst[:n].copy_(src[:n], non_blocking=True)
            s.synchronize()
            for i, n in enumerate(sizes_bytes):
                best[i] = min(best[i], _time_us(lambda: dst[:n].copy_(src[:n], non_blocking=True), reps, s))
    return list(sizes_bytes), best


def measure_hbm(device, d: int = 7168, fs=(512, 1024, 2048), counts=(8, 16, 32, 64), reps: int = 7, seed: int = 0):
    """Times (us) of caee_expert_ffn calls running m bf16 experts of size
    3*d*f*2 bytes with one token each, for each f in `fs` and m in `counts`."""
    import torch
    from . import caee
    E = max(counts)
    samples = []
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    for f in fs:
        layer = caee.Layer(T=max(counts) // 8, d=d, f=f, E=E, n_group=8, topk_group=8, k=8, n_shared=0,
                           routed_scaling=1.0, w_dtype="bf16", x_dtype="bf16", y_dtype="bf16")
        W = {"w13": (torch.randn((E, 2 * f, d), generator=gen, device=device) * 0.02).to(torch.bfloat16),
             "w2": (torch.randn((E, d, f), generator=gen, device=device) * 0.02).to(torch.bfloat16)}
        Wt = caee.pack_weights(W, "bf16")
        del W
        nbytes = 3 * d * f * 2
        for m in counts:
            T = m // 8
            lay = caee.Layer(**{**layer.__dict__, "T": T})
            x = torch.randn((T, d), generator=gen, device=device).to(torch.bfloat16)
            ids = torch.arange(m, dtype=torch.int32, device=device).reshape(T, 8)
            w = torch.full((T, 8), 1.0 / 8, dtype=torch.float32, device=device)
            y = torch.empty((T, d), dtype=torch.bfloat16, device=device)
            ws = caee.alloc_workspace(lay, device)
            st = torch.cuda.current_stream(device)
            t = _time_us(lambda: caee.expert_ffn(lay, x, ids, w, Wt, y, ws), reps, st)
            samples.append((m, nbytes, t))
        del Wt
        torch.cuda.empty_cache()
    return samples


def calibrate(device) -> dict:
    """Both data paths of the device: {'hbm': CostModel, 'link': CostModel,
    'samples': ...}."""
    measure_link(device, reps=3)                  # one full untimed pass over the copy path
    ls, lt = measure_link(device)
    link = fit_link(ls, lt, LINK_GBPS)
    hs = measure_hbm(device)
    hbm = fit_grouped([s[0] for s in hs], [s[1] for s in hs], [s[2] for s in hs], HBM_GBPS)
    return {"hbm": hbm, "link": link,
            "samples": {"hbm": [(m, n, round(t, 2)) for m, n, t in hs],
                        "link": [(n, round(t, 2)) for n, t in zip(ls, lt)]},
            "raw": {"hbm": hs, "link": list(zip(ls, lt))}}


def cost_table(model: CostModel, expert_bytes, E: int, resident=None) -> np.ndarray:
    """Per-expert fp32 cost table (us).  With `resident` (a boolean mask) the
    residency factor of Sec. IV-A applies: resident experts cost 0."""
    c = np.full(E, float(model.cost_us(expert_bytes)), dtype=np.float32)
    if resident is not None:
        c[np.asarray(resident, dtype=bool)] = 0.0
    return c
