"""GPU parity at the DeepSeek-R1 layer shape (d=7168, f=2048, 256 experts in
8 groups, top-4 groups, top-8 experts, 1 shared expert, bf16 weights), in
the launch configuration the benchmark times.  Routing, pruning and
compensation are compared on every token; the layer output on sampled
tokens, which the oracle evaluates one by one in fp64."""
import numpy as np
import pytest
import torch

from caee_cases import check_route, check_y, getters_dev, gpu_layer, oracle_layer
from paper_2606_29982_amd import caee
from synth_inputs import R1_BF16, make_expert_weights_torch, make_routing_inputs

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


@pytest.fixture(scope="module")
def r1_weights():
    print("drawing R1-shaped bf16 expert weights on the device", flush=True)
    W = make_expert_weights_torch(R1_BF16, seed=0, device=DEV)
    torch.cuda.synchronize()
    yield W
    del W
    torch.cuda.empty_cache()


@pytest.fixture(scope="module")
def r1_tiled(r1_weights):
    Wt = caee.pack_weights(r1_weights, "bf16")
    torch.cuda.synchronize()
    yield Wt
    del Wt
    torch.cuda.empty_cache()


def _inputs(T, skewed, n_bins, seed=0):
    return make_routing_inputs(R1_BF16, seed=seed, T=T, zipf_logit_s=1.1 if skewed else None,
                               cost_kind="zipf" if skewed else "flat", n_bins=n_bins)


RULE_TAUS = {"max": (0.0, 0.02, 0.05, 0.1), "sum": (0.3, 0.6, 1.2), "cir": (0.7, 0.8, 0.9)}


@pytest.mark.parametrize("T", [1, 8, 32, 128])
@pytest.mark.parametrize("skewed", [False, True])
@pytest.mark.parametrize("rule", ["max", "sum", "cir"])
def test_r1_routing_sweep(T, skewed, rule, r1_weights):
    for tau in RULE_TAUS[rule]:
        for n_bins in (1, 8):
            inp = _inputs(T, skewed, n_bins, seed=T)
            print(f"route T={T} skewed={skewed} rule={rule} tau={tau} n_bins={n_bins}", flush=True)
            got = gpu_layer(R1_BF16, inp, tau, n_bins, r1_weights, DEV, route_only=True, rule=rule)
            ref = oracle_layer(R1_BF16, inp, tau, n_bins, with_y=False, rule=rule)
            check_route(got, ref, R1_BF16.E)
            # gate mass conserved on every token
            np.testing.assert_allclose(got["topk_w"].sum(axis=1), R1_BF16.routed_scaling, rtol=2e-6)


def _layer_case(W, T, skewed, tau, n_bins, tokens, rule="max", Wrun=None):
    """Layer parity; ``Wrun`` (default ``W``) is what the GPU runs, ``W``
    the row-major copy the oracle reads."""
    inp = _inputs(T, skewed, n_bins)
    print(f"layer T={T} skewed={skewed} rule={rule} tau={tau} n_bins={n_bins} tokens={tokens}", flush=True)
    got = gpu_layer(R1_BF16, inp, tau, n_bins, W if Wrun is None else Wrun, DEV, rule=rule)
    get, get_sh = getters_dev(W, "bf16")
    ref = oracle_layer(R1_BF16, inp, tau, n_bins, get, get_sh, tokens=tokens, rule=rule)
    check_route(got, ref, R1_BF16.E)
    rel = check_y(got["y"][tokens], ref["y"], 2e-2)
    print(f"  max|err|/max|ref| = {rel:.3e}", flush=True)
    return got, ref


def test_r1_dense_layer_t32(r1_weights):
    # the dense-routing baseline: no pruning
    got, ref = _layer_case(r1_weights, 32, False, 0.0, 1, [0, 17, 31])
    assert ref["stats"]["n_pruned"] == 0


@pytest.mark.parametrize("T,tokens", [(1, [0]), (8, [3, 7]), (128, [0, 64, 127])])
def test_r1_skewed_layer(T, tokens, r1_weights):
    # Zipf-skewed popularity and cost table, 8 bins (EP8-style placement)
    _layer_case(r1_weights, T, True, 0.1, 8, tokens)


@pytest.mark.parametrize("rule,tau,T,tokens", [("sum", 0.6, 64, [0, 33, 63]), ("cir", 0.8, 16, [0, 15]),
                                               ("sum", 1.2, 128, [5, 100])])
def test_r1_pruned_layer(rule, tau, T, tokens, r1_weights):
    # the paper's own importance rules prune at these thresholds
    got, ref = _layer_case(r1_weights, T, True, tau, 8, tokens, rule=rule)
    assert ref["stats"]["n_pruned"] > 0


@pytest.mark.parametrize("T,tokens,rule,tau", [(1, [0], "max", 0.0), (32, [0, 31], "max", 0.0),
                                               (128, [1, 77], "sum", 0.6)])
def test_r1_tiled_weights(T, tokens, rule, tau, r1_weights, r1_tiled):
    _layer_case(r1_weights, T, T == 128, tau, 8, tokens, rule=rule, Wrun=r1_tiled)


@pytest.mark.parametrize("rule,tau", [("max", 0.05), ("cir", 0.8)])
def test_r1_offload_sequence(r1_weights, r1_tiled, rule, tau):
    """The offloading layer at the R1 shape: 256 bf16 experts in pinned host
    memory, a 16-slot device cache and an 8-slot staging ring, T=16 decode
    calls with Zipf(1.2) popularity."""
    from caee_cases import run_offload_sequence
    from synth_inputs import make_call_sequence
    calls = make_call_sequence(R1_BF16, seed=11, n_calls=4, T=16, zipf_logit_s=1.2)
    get, get_sh = getters_dev(r1_weights, "bf16")
    st = run_offload_sequence(R1_BF16, calls, r1_tiled, DEV, n_cache=16, n_stage=8, fetch_batch=4, tau=tau,
                              rule=rule, miss_cost=1760.0, get=get, get_sh=get_sh,
                              y_tokens=lambda i: [0, 15] if i in (0, 3) else None, y_tol=2e-2)
    assert st["misses"] > 0 and st["hits"] > 0


@pytest.mark.parametrize("T", [1, 8, 32, 128])
@pytest.mark.parametrize("refill", ["none", "random", "literal"])
def test_r1_refill_variants(T, refill, r1_weights):
    """Compensation ablation variants at the R1 shape: the offloading rule
    (CIR) with one bin, where every non-mandatory candidate with a cost is
    pruned and many slots are refilled."""
    inp = make_routing_inputs(R1_BF16, seed=T, T=T, zipf_logit_s=1.1, cost_kind="zipf", n_bins=1)
    for tau in (0.9, 0.7):
        print(f"refill={refill} T={T} tau={tau}", flush=True)
        got = gpu_layer(R1_BF16, inp, tau, 1, r1_weights, DEV, route_only=True, rule="cir", refill=refill, seed=5)
        ref = oracle_layer(R1_BF16, inp, tau, 1, with_y=False, rule="cir", refill=refill, seed=5)
        check_route(got, ref, R1_BF16.E)
