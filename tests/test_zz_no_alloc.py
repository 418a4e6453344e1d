"""caee_moe_layer_noalloc (the whole layer in the library's own scratch
array, for callers that cannot allocate) against caee_moe_layer with a
caller workspace: two calls in a row, the second with a smaller batch, on a
tiny layer and at the DeepSeek-R1 shape.  The two share their kernels, so
every output must match bit for bit; outputs are also held to the oracle's
tolerance on the tiny layer."""
import numpy as np
import pytest
import torch

from caee_cases import check_route, check_y, getters_np, oracle_layer, to_dev, w_to_dev
from paper_2606_29982_amd import caee
from synth_inputs import R1_BF16, TINY_F32, make_expert_weights_np, make_expert_weights_torch, make_routing_inputs

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def _both(shape, inp, Wd, tau, n_bins, rule="max"):
    T = inp.logits.shape[0]
    layer = caee.Layer.from_shape(shape, T=T, tau=tau, n_bins=n_bins, importance=rule)
    ydt = torch.float32 if shape.y_dtype == "f32" else torch.bfloat16
    x, logits, bias = to_dev(inp.x, DEV), to_dev(inp.logits, DEV), to_dev(inp.bias, DEV)
    cost = to_dev(inp.cost, DEV)
    bins = to_dev(inp.bins, DEV) if n_bins > 1 else None
    out_a = caee.alloc_route_out(layer, DEV)
    out_b = caee.alloc_route_out(layer, DEV)
    ya = torch.full((T + 2, shape.d), 7.0, dtype=ydt, device=DEV)
    yb = torch.full((T + 2, shape.d), 7.0, dtype=ydt, device=DEV)
    ws = caee.alloc_workspace(layer, DEV)
    caee.moe_layer(layer, x, logits, bias, cost, bins, Wd, ya[1:T + 1], ws, out_a)
    caee.moe_layer_noalloc(layer, x, logits, bias, cost, bins, Wd, yb[1:T + 1], out_b)
    torch.cuda.synchronize()
    assert torch.all(yb[0] == 7.0) and torch.all(yb[T + 1] == 7.0), "write outside y"
    assert torch.equal(ya, yb), "outputs differ from caee_moe_layer"
    for k in out_a:
        assert torch.equal(out_a[k], out_b[k]), k
    res = {k: v.cpu().numpy() for k, v in out_b.items()}
    res["y"] = yb[1:T + 1].float().cpu().numpy().astype(np.float64)
    return res


@pytest.mark.parametrize("T1,T2", [(40, 7), (300, 16)])
def test_noalloc_matches_workspace_entry_tiny(T1, T2):
    shape = TINY_F32
    W = make_expert_weights_np(shape, seed=3)
    Wd = w_to_dev(W, DEV)
    get, get_sh = getters_np(W, "f32")
    for T in (T1, T2):
        inp = make_routing_inputs(shape, seed=T, T=T, n_bins=4)
        print(f"noalloc tiny T={T}", flush=True)
        got = _both(shape, inp, Wd, 0.2, 4)
        ref = oracle_layer(shape, inp, 0.2, 4, get, get_sh)
        check_route(got, ref, shape.E)
        check_y(got["y"], ref["y"], 1e-5)


def test_noalloc_matches_workspace_entry_r1():
    print("drawing R1-shaped bf16 expert weights on the device", flush=True)
    W = caee.pack_weights(make_expert_weights_torch(R1_BF16, seed=0, device=DEV), "bf16")
    torch.cuda.synchronize()
    try:
        # 128 skewed tokens (big chunks, run on the one stream here) then 8
        for T in (128, 8):
            inp = make_routing_inputs(R1_BF16, seed=T, T=T, zipf_logit_s=1.1, cost_kind="zipf", n_bins=8)
            print(f"noalloc R1 T={T}", flush=True)
            _both(R1_BF16, inp, W, 0.1, 8)
        # a batch whose workspace exceeds the array is refused before any launch
        layer = caee.Layer.from_shape(R1_BF16, T=256, tau=0.0, n_bins=1)
        assert caee.workspace_size(layer) > caee.SCRATCH_BYTES
        inp = make_routing_inputs(R1_BF16, seed=1, T=256)
        y = torch.full((256, R1_BF16.d), 5.0, dtype=torch.bfloat16, device=DEV)
        with pytest.raises(caee.CaeeError) as ei:
            caee.moe_layer_noalloc(layer, to_dev(inp.x, DEV), to_dev(inp.logits, DEV), to_dev(inp.bias, DEV),
                                   to_dev(inp.cost, DEV), None, W, y)
        assert ei.value.status == caee.CAEE_ERR_UNSUPPORTED
        torch.cuda.synchronize()
        assert torch.all(y == 5.0)
    finally:
        del W
        torch.cuda.empty_cache()
