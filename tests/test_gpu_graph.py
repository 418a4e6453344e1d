"""HIP-graph capture of the layer call.

The layer launches a fixed sequence of kernels whose work lists are built on
the device, so one captured call can be replayed for new inputs in the same
buffers.  Each replay is checked bit for bit against an eager call on the
same inputs, with eager calls and synchronisation between the replays:
routing through the fused single-workgroup kernel (5 tokens) and through
the token-parallel kernels with big chunks on the second stream (40 tokens),
bf16 weights, and the 8-bit path with the prefill GEMM (600 tokens)."""
import numpy as np
import pytest
import torch

from caee_cases import to_dev, w_to_dev
from paper_2606_29982_amd import caee
from synth_inputs import TINY_F32, make_expert_weights_np, make_routing_inputs

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")

TINY_BF16 = TINY_F32.with_(name="tiny-bf16", w_dtype="bf16", x_dtype="bf16", y_dtype="bf16")
TINY_FP8 = TINY_F32.with_(name="tiny-fp8", w_dtype="fp8", x_dtype="bf16", y_dtype="bf16")


class Buffers:
    def __init__(self, shape, layer, T):
        ydt = torch.float32 if shape.y_dtype == "f32" else torch.bfloat16
        self.y = torch.empty((T, shape.d), dtype=ydt, device=DEV)
        self.ws = caee.alloc_workspace(layer, DEV)
        self.out = caee.alloc_route_out(layer, DEV)


@pytest.mark.parametrize("shape,T,tiled", [(TINY_F32, 5, False), (TINY_F32, 40, False), (TINY_BF16, 40, True),
                                           (TINY_FP8, 600, True)])
def test_graph_replays_match_eager(shape, T, tiled):
    print(f"graph {shape.name} T={T} tiled={tiled}", flush=True)
    n_bins = 4
    layer = caee.Layer.from_shape(shape, T=T, tau=0.2, n_bins=n_bins)
    W = w_to_dev(make_expert_weights_np(shape, seed=1), DEV)
    if tiled:
        W = caee.pack_weights(W, shape.w_dtype)
    inps = [make_routing_inputs(shape, seed=s, T=T, n_bins=n_bins, zipf_logit_s=1.1) for s in (2, 3)]
    x = to_dev(inps[0].x, DEV).clone()
    logits = to_dev(inps[0].logits, DEV).clone()
    bias = to_dev(inps[0].bias, DEV)
    cost = to_dev(inps[0].cost, DEV)
    bins = to_dev(inps[0].bins, DEV)
    eager, graph = Buffers(shape, layer, T), Buffers(shape, layer, T)

    def call(b):
        caee.moe_layer(layer, x, logits, bias, cost, bins, W, b.y, b.ws, b.out)

    call(eager)                       # first use creates the library's second stream
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call(graph)
    torch.cuda.synchronize()
    for rnd, src in enumerate((0, 1, 0, 1)):
        x.copy_(to_dev(inps[src].x, DEV))
        logits.copy_(to_dev(inps[src].logits, DEV))
        call(eager)
        torch.cuda.synchronize()
        graph.y.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        print(f"  replay {rnd} on inputs {src}", flush=True)
        assert torch.equal(graph.y, eager.y), "y of the replay differs from the eager call"
        for name in ("topk_ids", "topk_w", "stats", "masks"):
            assert torch.equal(graph.out[name], eager.out[name]), name
    # the two input sets route differently, so the replays did not reuse a result
    assert not torch.equal(to_dev(inps[0].logits, DEV), to_dev(inps[1].logits, DEV))


def test_first_call_of_a_process_under_capture():
    # A fresh process whose first layer call is captured: the library's
    # second stream and its fork/join events are created during capture.
    import subprocess
    import sys
    script = __file__.replace("test_gpu_graph.py", "graph_first_call.py")
    print("running the first call of a new process under graph capture", flush=True)
    r = subprocess.run([sys.executable, "-u", script], capture_output=True, text=True, timeout=240)
    print(r.stdout[-2000:], r.stderr[-2000:], flush=True)
    assert r.returncode == 0 and "first call under capture ok" in r.stdout
