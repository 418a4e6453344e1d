"""Expert FFN and combine (oracle, fp64) -- the MoE output equation of
Sec. II-A: y_t = sum over e in K_t of G(t)_e * E_e(t).

Test infrastructure only; see the package docstring.

Each expert E_e is a SwiGLU feed-forward block with gate, up and down
matrices of d x f (3 x 7168 x 2048 for DeepSeek-R1, Sec. V-B):
    E(x) = W2 (silu(W1 x) * (W3 x)),   silu(z) = z / (1 + exp(-z)),
with w13 = [W1; W3] stored [2f][d] and W2 stored [d][f].  Shared experts are
added for every token with weight 1.  Stored bf16/fp32 values are widened
exactly to float64 and no intermediate rounding happens, except on the 8-bit
path: there the weights are e4m3 codes times fp32 128x128 block scales, and
the activations entering each matrix product (x, then the SwiGLU output) are
quantised per token per 128 channels, as the kernel does, with the
quantisation decisions taken in fp32 like the kernel takes them.
"""
from __future__ import annotations

import numpy as np

E4M3_MAX = 448.0


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> float64 (exact)."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def _e4m3_table() -> np.ndarray:
    """Values of the OCP FP8 E4M3 (fn) codes 0..126: 1 sign, 4 exponent bits
    (bias 7), 3 mantissa bits; exponent field 0 is subnormal (m/8 * 2^-6);
    code 127 (S.1111.111) is NaN and there are no infinities."""
    vals = []
    for c in range(127):
        ex, man = c >> 3, c & 7
        if ex == 0:
            vals.append((man / 8.0) * 2.0 ** -6)
        else:
            vals.append((1.0 + man / 8.0) * 2.0 ** (ex - 7))
    return np.array(vals, dtype=np.float64)


_E4M3_POS = _e4m3_table()
# Every byte: codes 0..127 are the positive half (127 = NaN), bit 7 the sign.
_E4M3_ALL = np.concatenate([_E4M3_POS, [np.nan], -_E4M3_POS, [np.nan]])


def e4m3_decode(codes: np.ndarray) -> np.ndarray:
    """e4m3 codes (uint8) -> float64.  NaN codes decode to NaN."""
    c = np.ascontiguousarray(codes, dtype=np.uint8)
    return _E4M3_ALL[c.ravel()].reshape(c.shape)


def e4m3_encode_rne(v: np.ndarray) -> np.ndarray:
    """Round float values to the nearest e4m3 code, ties to the even code,
    saturating at +-448.  Returns uint8 codes."""
    x = np.asarray(v, dtype=np.float64)
    a = np.minimum(np.abs(x), E4M3_MAX)
    hi = np.searchsorted(_E4M3_POS, a, side="left")     # first value >= a
    hi = np.minimum(hi, 126)
    lo = np.maximum(hi - 1, 0)
    d_lo = a - _E4M3_POS[lo]
    d_hi = _E4M3_POS[hi] - a
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (hi % 2 == 0))
    code = np.where(pick_hi, hi, lo).astype(np.uint8)
    return np.where(x < 0, code | np.uint8(0x80), code).astype(np.uint8)


def quantize_e4m3_blocks(a: np.ndarray, block: int = 128):
    """Per-row, per-``block``-column quantisation of a [n][c] array.

    In fp32 (the kernel's precision): amax of the block, scale = amax / 448
    (1 when amax is 0), code = e4m3 rounding of value / scale.  Returns
    (codes [n][c] uint8, scales [n][c/block] fp32, dequantised float64)."""
    a32 = np.asarray(a, dtype=np.float32)
    n, c = a32.shape
    blocks = a32.reshape(n, c // block, block)
    amax = np.abs(blocks).max(axis=2)
    scale = np.where(amax > 0, amax / np.float32(E4M3_MAX), np.float32(1.0)).astype(np.float32)
    ratio = (blocks / scale[:, :, None]).astype(np.float32)
    codes = e4m3_encode_rne(ratio).reshape(n, c)
    deq = (e4m3_decode(codes).reshape(n, c // block, block)
           * scale[:, :, None].astype(np.float64)).reshape(n, c)
    return codes, scale, deq


def expert_weights_f64(w13, w2, dtype: str, w13_scale=None, w2_scale=None, block: int = 128):
    """Widen one expert's stored matrices to float64 ([2f][d], [d][f])."""
    if dtype == "f32":
        return np.asarray(w13, np.float64), np.asarray(w2, np.float64)
    if dtype == "bf16":
        return bf16_bits_to_f64(w13), bf16_bits_to_f64(w2)
    if dtype == "fp8":
        out = []
        for codes, sc in ((w13, w13_scale), (w2, w2_scale)):
            v = e4m3_decode(codes)
            r, c = v.shape
            # element (i, j) times the scale of block (i // block, j // block)
            sc = np.asarray(sc, np.float64)
            blocks = v.reshape(r // block, block, c // block, block)
            out.append((blocks * sc[:, None, :, None]).reshape(r, c))
        return out[0], out[1]
    raise ValueError(dtype)


def silu(z: np.ndarray) -> np.ndarray:
    with np.errstate(over="ignore"):
        return z / (1.0 + np.exp(-z))


def swiglu_expert(x: np.ndarray, w13: np.ndarray, w2: np.ndarray, fp8_acts: bool = False) -> np.ndarray:
    """E(x) for the rows of x [n][d]: W2 (silu(W1 x) * (W3 x)), float64.
    With ``fp8_acts`` the activations entering each product are quantised
    per token per 128 channels first."""
    f = w13.shape[0] // 2
    xin = quantize_e4m3_blocks(x)[2] if fp8_acts else x
    gate = xin @ w13[:f].T
    up = xin @ w13[f:].T
    h = silu(gate) * up
    if fp8_acts:
        h = quantize_e4m3_blocks(h)[2]
    return h @ w2.T
