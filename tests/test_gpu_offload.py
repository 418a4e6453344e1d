"""Offload residency on the GPU (caee_offload_layer): a sequence of layer
calls against the oracle's LRU cache.  Every call's routing decisions are
bit-exact, outputs within tolerance, the device cache holds exactly the
oracle's resident set, and the result is bit-identical to caee_moe_layer
given the same residency cost table."""
import numpy as np
import pytest
import torch

from caee_cases import getters_np, run_offload_sequence, to_dev, w_to_dev
from paper_2606_29982_amd import caee
from synth_inputs import TINY_F32, make_call_sequence, make_expert_weights_np

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


@pytest.fixture(scope="module")
def tiny_w():
    W = make_expert_weights_np(TINY_F32, seed=0)
    return W, w_to_dev(W, DEV)


@pytest.mark.parametrize("n_cache,n_stage,batch,tau,rule,tiled", [
    (4, 2, 1, 0.1, "max", False),
    (4, 2, 3, 0.0, "max", True),
    (4, 4, 4, 0.1, "max", True),
    (6, 2, 2, 0.8, "cir", True),
    (16, 0, 2, 0.0, "max", False),
    (0, 3, 2, 0.05, "max", True),
])
def test_tiny_offload_sequence(tiny_w, n_cache, n_stage, batch, tau, rule, tiled):
    W, Wd = tiny_w
    Wl = caee.pack_weights(Wd, "f32") if tiled else dict(Wd, layout=caee.LAYOUT_ROWMAJOR)
    calls = make_call_sequence(TINY_F32, seed=7, n_calls=12, zipf_logit_s=1.2)
    get, get_sh = getters_np(W, "f32")
    st = run_offload_sequence(TINY_F32, calls, Wl, DEV, n_cache, n_stage, batch, tau, rule, miss_cost=3.0,
                              get=get, get_sh=get_sh, y_tokens=lambda i: list(range(16)), y_tol=1e-5)
    if n_cache < TINY_F32.E:
        assert st["misses"] > 0


def test_tiny_offload_capacity_error(tiny_w):
    _, Wd = tiny_w
    calls = make_call_sequence(TINY_F32, seed=7, n_calls=1)
    layer = caee.Layer.from_shape(TINY_F32, T=16, tau=0.0, n_bins=1)
    host = caee.pin_host_weights(dict(Wd, layout=0))
    s13, s2 = caee.alloc_slots(layer, 2, DEV)
    h = caee.Offload(layer, host["w13"], host["w2"], s13, s2, Wd["sh_w13"], Wd["sh_w2"], 2, 0, 1.0, 2, 0)
    try:
        ws = caee.alloc_workspace(layer, DEV)
        y = torch.full((16, TINY_F32.d), 7.0, device=DEV)
        inp = calls[0]
        with pytest.raises(caee.CaeeError) as ei:
            h(layer, to_dev(inp.x, DEV), to_dev(inp.logits, DEV), None, y, ws)
        assert ei.value.status == caee.CAEE_ERR_CAPACITY
        torch.cuda.synchronize()
        assert torch.all(y == 7.0)
        assert np.all(h.residency() == -1)
        assert h.stats()["calls"] == 0
    finally:
        h.close()


def test_tiny_offload_reset_and_rejects(tiny_w):
    _, Wd = tiny_w
    calls = make_call_sequence(TINY_F32, seed=3, n_calls=2)
    layer = caee.Layer.from_shape(TINY_F32, T=16, tau=0.1, n_bins=1)
    host = caee.pin_host_weights(dict(Wd, layout=0))
    s13, s2 = caee.alloc_slots(layer, 6, DEV)
    # pageable host memory is refused
    pageable = [torch.empty_like(host["w13"][0], device="cpu") for _ in range(TINY_F32.E)]
    with pytest.raises(caee.CaeeError):
        caee.Offload(layer, pageable, host["w2"], s13, s2, Wd["sh_w13"], Wd["sh_w2"], 4, 2, 1.0, 2, 0)
    h = caee.Offload(layer, host["w13"], host["w2"], s13, s2, Wd["sh_w13"], Wd["sh_w2"], 4, 2, 1.0, 2, 0)
    try:
        ws = caee.alloc_workspace(layer, DEV)
        y = torch.empty((16, TINY_F32.d), device=DEV)
        inp = calls[0]
        h(layer, to_dev(inp.x, DEV), to_dev(inp.logits, DEV), None, y, ws)
        torch.cuda.synchronize()
        assert h.stats()["calls"] == 1 and np.any(h.residency() >= 0)
        # n_bins other than 1 and a layer of another shape are refused
        with pytest.raises(caee.CaeeError):
            bad = caee.Layer.from_shape(TINY_F32, T=16, tau=0.1, n_bins=4)
            h(bad, to_dev(inp.x, DEV), to_dev(inp.logits, DEV), None, y, caee.alloc_workspace(bad, DEV))
        with pytest.raises(caee.CaeeError):
            bad = caee.Layer.from_shape(TINY_F32, T=16, tau=0.1, n_bins=1, n_shared=0)
            h(bad, to_dev(inp.x, DEV), to_dev(inp.logits, DEV), None, y, caee.alloc_workspace(bad, DEV))
        h.reset()
        assert np.all(h.residency() == -1) and h.stats()["calls"] == 0
        # T = 0 does nothing
        z = caee.Layer.from_shape(TINY_F32, T=0, tau=0.1, n_bins=1)
        h(z, to_dev(inp.x, DEV), to_dev(inp.logits, DEV), None, y, caee.alloc_workspace(z, DEV))
        assert h.stats()["calls"] == 0
    finally:
        h.close()
