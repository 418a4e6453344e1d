"""Run as its own process by tests/test_gpu_graph.py: the first layer call of
the process happens under HIP-graph capture, so the library creates its
second stream (and the events that fork work onto it and join it back)
while the caller's stream is capturing.  The replays are then checked bit
for bit against eager calls.  Prints "first call under capture ok"."""
import os
import sys

import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))

from caee_cases import to_dev, w_to_dev  # noqa: E402
from paper_2606_29982_amd import caee  # noqa: E402
from synth_inputs import TINY_F32, make_expert_weights_np, make_routing_inputs  # noqa: E402

DEV = torch.device("cuda:0")
shape = TINY_F32.with_(name="tiny-bf16", w_dtype="bf16", x_dtype="bf16", y_dtype="bf16")
T = 40     # experts with more than 32 rows: big chunks on the library's second stream
layer = caee.Layer.from_shape(shape, T=T, tau=0.2, n_bins=4)
W = caee.pack_weights(w_to_dev(make_expert_weights_np(shape, seed=1), DEV), "bf16")
inp = make_routing_inputs(shape, seed=2, T=T, n_bins=4, zipf_logit_s=1.1)
x, logits = to_dev(inp.x, DEV), to_dev(inp.logits, DEV)
bias, cost, bins = to_dev(inp.bias, DEV), to_dev(inp.cost, DEV), to_dev(inp.bins, DEV)
bufs = []
for _ in range(2):
    bufs.append((torch.empty((T, shape.d), dtype=torch.bfloat16, device=DEV), caee.alloc_workspace(layer, DEV),
                 caee.alloc_route_out(layer, DEV)))
torch.cuda.synchronize()
g = torch.cuda.CUDAGraph()
with torch.cuda.graph(g):
    y, ws, out = bufs[0]
    caee.moe_layer(layer, x, logits, bias, cost, bins, W, y, ws, out)
torch.cuda.synchronize()
for rep in range(3):
    ye, wse, oute = bufs[1]
    caee.moe_layer(layer, x, logits, bias, cost, bins, W, ye, wse, oute)
    torch.cuda.synchronize()
    bufs[0][0].fill_(float("nan"))
    g.replay()
    torch.cuda.synchronize()
    assert torch.equal(bufs[0][0], ye), f"replay {rep}: y differs from the eager call"
    for name in ("topk_ids", "topk_w", "stats", "masks"):
        assert torch.equal(bufs[0][2][name], oute[name]), name
big = int((torch.bincount(oute["topk_ids"].flatten().clamp(min=0).long()) > 32).sum())
assert big > 0, "no expert with more than 32 rows: the second stream was not used"
print("first call under capture ok", flush=True)
