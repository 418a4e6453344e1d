"""Pins for the oracle's expert FFN, combine and number codecs: OCP e4m3
table values, torch's converters, a closed-form SwiGLU case and brute-force
dense evaluation of all experts."""
import numpy as np
import pytest
import torch

from oracle import (bf16_bits_to_f64, e4m3_decode, e4m3_encode_rne, expert_weights_f64,
                    moe_layer_ref, quantize_e4m3_blocks, swiglu_expert)
from synth_inputs import (TINY_F32, bf16_bits_from_f32, make_expert_weights_np,
                          make_routing_inputs)


def test_e4m3_table(golden):
    g = golden("e4m3_ocp.json")
    for code, val in g["decode"]:
        got = e4m3_decode(np.array([code], np.uint8))[0]
        assert got == val and np.signbit(got) == np.signbit(val)
    for val, code in g["encode"]:
        assert int(e4m3_encode_rne(np.array([val]))[0]) == code, val
    assert np.isnan(e4m3_decode(np.array([127, 255], np.uint8))).all()


def test_e4m3_against_torch():
    codes = np.array([c for c in range(256) if c & 0x7F != 0x7F], np.uint8)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    np.testing.assert_array_equal(e4m3_decode(codes), ref)
    # every representable value, every midpoint and random values inside range
    pos = np.sort(e4m3_decode(codes[codes < 127]))
    mids = (pos[1:] + pos[:-1]) / 2
    rnd = np.random.default_rng(0).standard_normal(20000) * 50
    v = np.concatenate([pos, mids, -mids, rnd.clip(-448, 448)]).astype(np.float32)
    ours = e4m3_decode(e4m3_encode_rne(v))
    theirs = torch.from_numpy(v).to(torch.float8_e4m3fn).to(torch.float64).numpy()
    np.testing.assert_array_equal(np.abs(ours), np.abs(theirs))


def test_bf16_decode_against_torch():
    a = np.random.default_rng(1).standard_normal(5000).astype(np.float32) * 3
    bits = bf16_bits_from_f32(a)
    ref = torch.from_numpy(a).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(bf16_bits_to_f64(bits), ref)


def test_quantize_blocks():
    rng = np.random.default_rng(2)
    a = rng.standard_normal((3, 256)).astype(np.float32)
    a[1, :128] = 0
    codes, scale, deq = quantize_e4m3_blocks(a)
    assert scale[1, 0] == 1.0 and np.all(deq[1, :128] == 0)
    np.testing.assert_allclose(scale[0], np.abs(a[0].reshape(2, 128)).max(axis=1) / 448, rtol=1e-7)
    # e4m3 keeps 3 mantissa bits: relative error <= 2^-4 for normal values
    big = np.abs(a) > 0.05
    assert np.all(np.abs(deq - a)[big] <= np.abs(a)[big] * 2.0 ** -4 + 1e-12)
    # the block max maps to 448 exactly
    assert np.all(np.abs(e4m3_decode(codes)).reshape(3, 2, 128).max(axis=2)[[0, 2]] == 448)


def test_swiglu_closed_form():
    d = f = 8
    rng = np.random.default_rng(3)
    x = rng.standard_normal((5, d))
    w13 = np.zeros((2 * f, d))
    w13[:f] = np.eye(d)           # gate = x
    w13[f:] = 2 * np.eye(d)       # up = 2x
    perm = rng.permutation(d)
    w2 = np.eye(d)[perm]          # y = P h
    y = swiglu_expert(x, w13, w2)
    h = (x / (1 + np.exp(-x))) * (2 * x)
    np.testing.assert_allclose(y, h[:, perm], rtol=1e-15)


def test_swiglu_against_torch():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((4, 32))
    w13 = rng.standard_normal((48, 32)) * 0.2
    w2 = rng.standard_normal((32, 24)) * 0.2
    tx, t13, t2 = map(torch.from_numpy, (x, w13, w2))
    ref = torch.nn.functional.linear(
        torch.nn.functional.silu(torch.nn.functional.linear(tx, t13[:24]))
        * torch.nn.functional.linear(tx, t13[24:]), t2)
    np.testing.assert_allclose(swiglu_expert(x, w13, w2), ref.numpy(), rtol=1e-13, atol=1e-15)


@pytest.mark.parametrize("tau", [0.0, 0.1, 0.3])
def test_brute_force_dense(tau):
    shape = TINY_F32
    inp = make_routing_inputs(shape, seed=0)
    W = make_expert_weights_np(shape, seed=0)
    get = lambda e: expert_weights_f64(W["w13"][e], W["w2"][e], "f32")  # noqa: E731
    get_sh = lambda s: expert_weights_f64(W["sh_w13"][s], W["sh_w2"][s], "f32")  # noqa: E731
    ref = moe_layer_ref(E=shape.E, n_group=shape.n_group, topk_group=shape.topk_group, k=shape.k,
                        routed_scaling=shape.routed_scaling, tau=tau, n_bins=4, logits=inp.logits,
                        bias=inp.bias, cost=inp.cost, bins=inp.bins, x=inp.x, x_dtype="f32",
                        w_dtype="f32", n_shared=1, get_expert=get, get_shared=get_sh)
    # evaluate every expert on every token, then weight by the dense matrix
    x = inp.x.astype(np.float64)
    dense = np.zeros((shape.T, shape.E))
    for t in range(shape.T):
        for slot in range(shape.k):
            if ref["topk_ids"][t, slot] >= 0:
                dense[t, ref["topk_ids"][t, slot]] += ref["topk_w"][t, slot]
    y = np.zeros((shape.T, shape.d))
    for e in range(shape.E):
        w13, w2 = get(e)
        y += dense[:, e:e + 1] * swiglu_expert(x, w13, w2)
    w13, w2 = get_sh(0)
    y += swiglu_expert(x, w13, w2)
    np.testing.assert_allclose(ref["y"], y, rtol=1e-12, atol=1e-14)
    if tau == 0.0:
        assert np.array_equal(ref["topk_ids"], ref["orig_ids"])


def test_fp8_weights_decode():
    shape = TINY_F32.with_(w_dtype="fp8")
    W = make_expert_weights_np(shape, seed=0, experts=[0])
    Wb = make_expert_weights_np(TINY_F32.with_(w_dtype="bf16"), seed=0, experts=[0])
    w13, w2 = expert_weights_f64(W["w13"][0], W["w2"][0], "fp8", W["w13_scale"][0], W["w2_scale"][0])
    ref13 = bf16_bits_to_f64(Wb["w13"][0])
    # block-scaled e4m3 keeps each weight within 2^-4 of its bf16 value,
    # or within half the smallest step of its block near zero
    step = np.repeat(np.repeat(W["w13_scale"][0], 128, 0), 128, 1) * 2.0 ** -9
    assert np.all(np.abs(w13 - ref13) <= np.abs(ref13) * 2.0 ** -4 + step)
