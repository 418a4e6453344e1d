"""Seeded generators for MoE-layer inputs: hidden states, router logits,
router bias, per-expert cost table, expert-to-bin placement and expert
weights.

Random-number streams: every tensor draws from its own stream so a single
expert can be regenerated without drawing the rest of the layer.
``numpy.random.default_rng(SeedSequence([seed, stream]))`` with streams

  0 hidden states x        1 router logits        2 router bias
  3 cost multipliers       4 popularity permutation   5 cost permutation
  (99, s) shared expert s  100 + e routed expert e (w13 drawn before w2)

Normal draws are fp32 ``standard_normal * std`` and are then encoded to the
storage dtype with round-to-nearest-even.  DeepSeek-R1-sized expert weights
(256 experts of 3 x 7168 x 2048) are drawn on the GPU with torch's device
generator, one expert at a time, seeded from the same (seed, stream) pairs;
those values differ from the numpy draws but are just as reproducible.
"""
from __future__ import annotations

from dataclasses import dataclass, replace
from typing import Optional

import numpy as np


@dataclass(frozen=True)
class LayerShape:
    """One MoE layer: sizes, routing hyper-parameters and storage dtypes."""

    name: str
    T: int            # tokens in the batch
    d: int            # hidden size
    f: int            # expert intermediate size
    E: int            # routed experts
    n_group: int      # expert groups for group-limited routing
    topk_group: int   # groups kept per token
    k: int            # experts kept per token
    n_shared: int     # always-active shared experts
    routed_scaling: float
    w_dtype: str      # 'f32' | 'bf16' | 'fp8'
    x_dtype: str      # 'f32' | 'bf16'
    y_dtype: str      # 'f32' | 'bf16'
    w_std: float
    bias_std: float   # 0 => no router bias
    tau: float = 0.0
    n_bins: int = 1

    def with_(self, **kw) -> "LayerShape":
        return replace(self, **kw)


# Tiny fp32 layer: 16 experts in 4 groups, top-2 groups then top-4 experts.
TINY_F32 = LayerShape(
    name="tiny-fp32", T=16, d=256, f=128, E=16, n_group=4, topk_group=2, k=4,
    n_shared=1, routed_scaling=1.0, w_dtype="f32", x_dtype="f32", y_dtype="f32",
    w_std=0.05, bias_std=0.0, tau=0.1, n_bins=4)

# DeepSeek-R1-shaped MoE layer in bf16: 256 experts in 8 groups, top-4
# groups then top-8 experts, sigmoid scores + bias, routed scaling 2.5.
R1_BF16 = LayerShape(
    name="deepseek-r1-bf16", T=32, d=7168, f=2048, E=256, n_group=8,
    topk_group=4, k=8, n_shared=1, routed_scaling=2.5, w_dtype="bf16",
    x_dtype="bf16", y_dtype="bf16", w_std=0.02, bias_std=0.01, tau=0.0,
    n_bins=1)

# Same layer with OCP e4m3 expert weights and fp32 128x128 block scales.
R1_FP8 = R1_BF16.with_(name="deepseek-r1-fp8", w_dtype="fp8", T=64, tau=0.05,
                       n_bins=8)

WORKLOADS = {s.name: s for s in (TINY_F32, R1_BF16, R1_FP8)}

_W_ITEMSIZE = {"f32": 4, "bf16": 2, "fp8": 1}


def weight_bytes_per_expert(shape: LayerShape) -> int:
    """Bytes of one expert's gate, up and down matrices (plus fp8 scales)."""
    n = 3 * shape.d * shape.f * _W_ITEMSIZE[shape.w_dtype]
    if shape.w_dtype == "fp8":
        n += 4 * (2 * shape.f // 128) * (shape.d // 128)
        n += 4 * (shape.d // 128) * (shape.f // 128)
    return n


def _rng(seed: int, *stream: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([int(seed), *map(int, stream)]))


def _torch_seed(seed: int, *stream: int) -> int:
    st = np.random.SeedSequence([int(seed), *map(int, stream)]).generate_state(2, np.uint32)
    return int(st[0]) | (int(st[1] & 0x7FFFFFFF) << 32)


def bf16_bits_from_f32(a: np.ndarray) -> np.ndarray:
    """Encode fp32 values as bf16 bit patterns, rounding to nearest even."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    rounded = u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return (rounded >> np.uint32(16)).astype(np.uint16)


def _encode(a: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return np.ascontiguousarray(a, dtype=np.float32)
    if dtype == "bf16":
        return bf16_bits_from_f32(a)
    raise ValueError(dtype)


def _zipf_probs(n: int, s: float) -> np.ndarray:
    r = np.arange(1, n + 1, dtype=np.float64)
    p = r ** (-s)
    return p / p.sum()


@dataclass
class RoutingInputs:
    """Host arrays for one layer call (storage dtypes)."""

    x: np.ndarray                 # [T][d] fp32 or bf16 bits (uint16)
    logits: np.ndarray            # [T][E] fp32
    bias: Optional[np.ndarray]    # [E] fp32 or None
    cost: np.ndarray              # [E] fp32, >= 0
    bins: Optional[np.ndarray]    # [E] int32 or None (one bin)


def make_routing_inputs(shape: LayerShape, seed: int = 0, T: Optional[int] = None,
                        zipf_logit_s: Optional[float] = None,
                        cost_kind: str = "uniform",
                        n_bins: Optional[int] = None) -> RoutingInputs:
    """Hidden states ~N(0,1), router logits ~N(0,1) (+ a Zipf-skewed
    per-expert offset when ``zipf_logit_s`` is given), bias ~N(0, bias_std),
    cost table of kind ``cost_kind`` and a contiguous expert-to-bin map."""
    T = shape.T if T is None else int(T)
    x = _rng(seed, 0).standard_normal((T, shape.d), dtype=np.float32)
    logits = _rng(seed, 1).standard_normal((T, shape.E), dtype=np.float32)
    if zipf_logit_s is not None:
        # Popularity skew: expert e gets offset ln(E * p_rank(e)), with p a
        # Zipf(s) law over a random rank permutation.
        perm = _rng(seed, 4).permutation(shape.E)
        p = _zipf_probs(shape.E, zipf_logit_s)
        mu = np.log(shape.E * p[perm]).astype(np.float32)
        logits = (logits + mu[None, :]).astype(np.float32)
    bias = None
    if shape.bias_std > 0:
        bias = (_rng(seed, 2).standard_normal(shape.E, dtype=np.float32)
                * np.float32(shape.bias_std)).astype(np.float32)
    nb = shape.n_bins if n_bins is None else int(n_bins)
    return RoutingInputs(
        x=_encode(x, shape.x_dtype),
        logits=np.ascontiguousarray(logits, dtype=np.float32),
        bias=bias,
        cost=make_cost_table(shape, seed, cost_kind),
        bins=make_bins(shape, nb),
    )


def popularity_ranks(shape: LayerShape, seed: int) -> np.ndarray:
    """Popularity rank of every expert (0 = most popular) under the Zipf
    offset of make_routing_inputs / make_call_sequence (stream 4)."""
    return _rng(seed, 4).permutation(shape.E)


def make_call_sequence(shape: LayerShape, seed: int, n_calls: int, T: Optional[int] = None,
                       zipf_logit_s: float = 1.2) -> list:
    """Inputs of ``n_calls`` consecutive layer calls (decode steps) that share
    one expert-popularity law: call i draws fresh hidden states ~N(0,1)
    (stream (0, i)) and logits ~N(0,1) (stream (1, i)), plus the fixed offset
    ln(E * p_rank(e)) of a Zipf(``zipf_logit_s``) law over a rank permutation
    drawn once (stream 4).  The bias is fixed across calls; the cost table is
    left at zero (an offloading caller derives it from residency)."""
    T = shape.T if T is None else int(T)
    perm = _rng(seed, 4).permutation(shape.E)
    mu = np.log(shape.E * _zipf_probs(shape.E, zipf_logit_s)[perm]).astype(np.float32)
    bias = None
    if shape.bias_std > 0:
        bias = (_rng(seed, 2).standard_normal(shape.E, dtype=np.float32)
                * np.float32(shape.bias_std)).astype(np.float32)
    calls = []
    for i in range(int(n_calls)):
        x = _rng(seed, 0, i).standard_normal((T, shape.d), dtype=np.float32)
        logits = _rng(seed, 1, i).standard_normal((T, shape.E), dtype=np.float32) + mu[None, :]
        calls.append(RoutingInputs(x=_encode(x, shape.x_dtype),
                                   logits=np.ascontiguousarray(logits, dtype=np.float32), bias=bias,
                                   cost=np.zeros(shape.E, np.float32), bins=None))
    return calls


def make_cost_table(shape: LayerShape, seed: int = 0, kind: str = "uniform") -> np.ndarray:
    """Per-expert data-movement cost in bytes-equivalent units.

    ``uniform``: weight bytes x U(0.5, 2).
    ``zipf``:    weight bytes x (1/2 + E/2 * q_rank(e)), q a Zipf(1.1) law over
                 an independent random permutation (hot/cold skew, mean 1).
    ``flat``:    weight bytes for every expert.
    ``zero``:    every expert resident (cost 0).
    """
    wb = float(weight_bytes_per_expert(shape))
    if kind == "uniform":
        m = _rng(seed, 3).uniform(0.5, 2.0, shape.E)
    elif kind == "zipf":
        perm = _rng(seed, 5).permutation(shape.E)
        q = _zipf_probs(shape.E, 1.1)
        m = 0.5 + 0.5 * shape.E * q[perm]
    elif kind == "flat":
        m = np.ones(shape.E)
    elif kind == "zero":
        m = np.zeros(shape.E)
    else:
        raise ValueError(kind)
    return (m * wb).astype(np.float32)


def make_bins(shape: LayerShape, n_bins: int) -> Optional[np.ndarray]:
    """Contiguous placement of experts on ``n_bins`` devices (EP-style);
    None for a single bin."""
    if n_bins <= 1:
        return None
    if shape.E % n_bins:
        raise ValueError("E must be a multiple of n_bins")
    return (np.arange(shape.E, dtype=np.int32) // (shape.E // n_bins)).astype(np.int32)


def _fp8_blocks_torch(w_f32, block: int = 128):
    """Encode a [R][C] fp32 torch tensor as e4m3 codes with fp32 per
    block x block scales (scale = block amax / 448, 1 for an all-zero block)."""
    import torch
    R, C = w_f32.shape
    wb = w_f32.reshape(R // block, block, C // block, block)
    amax = wb.abs().amax(dim=(1, 3))
    scale = torch.where(amax > 0, amax / 448.0, torch.ones_like(amax)).to(torch.float32)
    q = (wb / scale[:, None, :, None]).clamp_(-448.0, 448.0)
    codes = q.reshape(R, C).to(torch.float8_e4m3fn).view(torch.uint8)
    return codes, scale


def make_expert_weights_np(shape: LayerShape, seed: int = 0, experts=None):
    """Expert weights on the host, one expert per (seed, stream).

    Returns a dict with ``w13`` [n][2f][d], ``w2`` [n][d][f] for the routed
    experts listed in ``experts`` (default: all) and ``sh_w13``/``sh_w2`` for
    the shared experts, in storage dtype; fp8 adds ``*_scale`` arrays.
    Intended for small layers (the tiny workload and unit tests).
    """
    experts = range(shape.E) if experts is None else list(experts)

    def one(*stream):
        g = _rng(seed, *stream)
        w13 = g.standard_normal((2 * shape.f, shape.d), dtype=np.float32) * np.float32(shape.w_std)
        w2 = g.standard_normal((shape.d, shape.f), dtype=np.float32) * np.float32(shape.w_std)
        return w13.astype(np.float32), w2.astype(np.float32)

    out = {}
    for key, streams in (("", [(100 + e,) for e in experts]),
                         ("sh_", [(99, s) for s in range(shape.n_shared)])):
        w13s, w2s = [], []
        for st in streams:
            a, b = one(*st)
            w13s.append(a)
            w2s.append(b)
        w13 = np.stack(w13s) if w13s else np.zeros((0, 2 * shape.f, shape.d), np.float32)
        w2 = np.stack(w2s) if w2s else np.zeros((0, shape.d, shape.f), np.float32)
        if shape.w_dtype == "fp8":
            import torch
            w13 = bf16_bits_from_f32(w13).astype(np.uint32) << np.uint32(16)
            w2 = bf16_bits_from_f32(w2).astype(np.uint32) << np.uint32(16)
            w13 = w13.view(np.float32)
            w2 = w2.view(np.float32)
            c13, s13, c2, s2 = [], [], [], []
            for i in range(w13.shape[0]):
                c, s = _fp8_blocks_torch(torch.from_numpy(w13[i].copy()))
                c13.append(c.numpy()); s13.append(s.numpy())
                c, s = _fp8_blocks_torch(torch.from_numpy(w2[i].copy()))
                c2.append(c.numpy()); s2.append(s.numpy())
            n = w13.shape[0]
            out[key + "w13"] = np.stack(c13) if n else np.zeros((0, 2 * shape.f, shape.d), np.uint8)
            out[key + "w2"] = np.stack(c2) if n else np.zeros((0, shape.d, shape.f), np.uint8)
            out[key + "w13_scale"] = (np.stack(s13) if n else
                                      np.zeros((0, 2 * shape.f // 128, shape.d // 128), np.float32))
            out[key + "w2_scale"] = (np.stack(s2) if n else
                                     np.zeros((0, shape.d // 128, shape.f // 128), np.float32))
        else:
            out[key + "w13"] = _encode(w13, shape.w_dtype)
            out[key + "w2"] = _encode(w2, shape.w_dtype)
    return out


def make_expert_weights_torch(shape: LayerShape, seed: int, device):
    """All expert weights drawn directly in device memory (torch tensors).

    bf16/f32: ``w13`` [E][2f][d], ``w2`` [E][d][f] (+ ``sh_w13``/``sh_w2``).
    fp8: uint8 e4m3 codes plus fp32 ``*_scale`` block scales of the same
    bf16 draws.  Each expert draws from its own seeded torch generator.
    """
    import torch
    tdt = {"f32": torch.float32, "bf16": torch.bfloat16, "fp8": torch.uint8}[shape.w_dtype]
    E, S, d, f = shape.E, shape.n_shared, shape.d, shape.f
    out = {
        "w13": torch.empty((E, 2 * f, d), dtype=tdt, device=device),
        "w2": torch.empty((E, d, f), dtype=tdt, device=device),
        "sh_w13": torch.empty((S, 2 * f, d), dtype=tdt, device=device),
        "sh_w2": torch.empty((S, d, f), dtype=tdt, device=device),
    }
    if shape.w_dtype == "fp8":
        out["w13_scale"] = torch.empty((E, 2 * f // 128, d // 128), dtype=torch.float32, device=device)
        out["w2_scale"] = torch.empty((E, d // 128, f // 128), dtype=torch.float32, device=device)
        out["sh_w13_scale"] = torch.empty((S, 2 * f // 128, d // 128), dtype=torch.float32, device=device)
        out["sh_w2_scale"] = torch.empty((S, d // 128, f // 128), dtype=torch.float32, device=device)
    gen = torch.Generator(device=device)

    def fill(prefix, i, stream):
        gen.manual_seed(_torch_seed(seed, *stream))
        for name, rows, cols in (("w13", 2 * f, d), ("w2", d, f)):
            w = torch.randn((rows, cols), generator=gen, device=device, dtype=torch.float32)
            w.mul_(shape.w_std)
            if shape.w_dtype == "f32":
                out[prefix + name][i].copy_(w)
            elif shape.w_dtype == "bf16":
                out[prefix + name][i].copy_(w.to(torch.bfloat16))
            else:
                codes, sc = _fp8_blocks_torch(w.to(torch.bfloat16).to(torch.float32))
                out[prefix + name][i].copy_(codes)
                out[prefix + name + "_scale"][i].copy_(sc)
            del w

    for e in range(E):
        fill("", e, (100 + e,))
    for s in range(S):
        fill("sh_", s, (99, s))
    return out
