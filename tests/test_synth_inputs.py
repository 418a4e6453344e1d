"""The shared input generator: encodings and recipe shapes."""
import numpy as np
import torch

from synth_inputs import (R1_BF16, TINY_F32, bf16_bits_from_f32, make_bins, make_cost_table,
                          make_expert_weights_np, make_routing_inputs, weight_bytes_per_expert)


def test_bf16_encoding_matches_torch_rne():
    a = np.random.default_rng(0).standard_normal(10000).astype(np.float32)
    a[:4] = [1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -8), 65504.0]   # ties
    ref = torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(bf16_bits_from_f32(a), ref)


def test_recipe_shapes_and_ranges():
    inp = make_routing_inputs(TINY_F32, seed=0)
    assert inp.x.shape == (16, 256) and inp.x.dtype == np.float32
    assert inp.logits.shape == (16, 16) and inp.bias is None
    assert inp.bins.tolist() == [0] * 4 + [1] * 4 + [2] * 4 + [3] * 4
    wb = weight_bytes_per_expert(TINY_F32)
    assert wb == 3 * 256 * 128 * 4
    assert np.all(inp.cost >= 0.5 * wb) and np.all(inp.cost <= 2 * wb)
    r1 = make_routing_inputs(R1_BF16, seed=0, T=8, zipf_logit_s=1.1, cost_kind="zipf", n_bins=8)
    assert r1.x.dtype == np.uint16 and r1.bias.shape == (256,)
    assert weight_bytes_per_expert(R1_BF16) == 88080384
    m = r1.cost / 88080384.0
    assert abs(m.mean() - 1.0) < 1e-3 and m.min() > 0.5 and m.max() < 27.0


def test_streams_are_independent():
    a = make_expert_weights_np(TINY_F32, seed=3, experts=[5])
    b = make_expert_weights_np(TINY_F32, seed=3)
    np.testing.assert_array_equal(a["w13"][0], b["w13"][5])
    np.testing.assert_array_equal(a["sh_w2"], b["sh_w2"])
    c = make_cost_table(TINY_F32, 0, "zero")
    assert not c.any()
    assert make_bins(TINY_F32, 1) is None
