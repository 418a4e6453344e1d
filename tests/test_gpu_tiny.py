"""GPU parity on small layers: the HIP path through the C ABI against the
fp64 oracle, element by element.  Indices, masks, counters and bin loads
must match exactly; weights to 1e-6; outputs to 1e-5 * max|ref| (fp32) or
2e-2 * max|ref| (bf16)."""
import numpy as np
import pytest
import torch

from caee_cases import (check_route, check_y, getters_np, gpu_layer, oracle_layer, to_dev,
                        w_to_dev)
from paper_2606_29982_amd import caee
from synth_inputs import TINY_F32, make_expert_weights_np, make_routing_inputs

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
TINY_BF16 = TINY_F32.with_(name="tiny-bf16", w_dtype="bf16", x_dtype="bf16", y_dtype="bf16")
TOL = {"f32": 1e-5, "bf16": 2e-2}


def _run(shape, seed=0, tau=0.1, n_bins=4, T=None, zipf=None, cost_kind="uniform", mutate=None, rule="max",
         tiled=False, refill="score", rseed=0, keep_top1=False):
    inp = make_routing_inputs(shape, seed=seed, T=T, zipf_logit_s=zipf, cost_kind=cost_kind,
                              n_bins=n_bins)
    if mutate:
        mutate(inp)
    W = make_expert_weights_np(shape, seed=seed)
    print(f"case {shape.name} seed={seed} tau={tau} n_bins={n_bins} T={inp.logits.shape[0]} rule={rule} "
          f"refill={refill} keep_top1={keep_top1}", flush=True)
    Wd = w_to_dev(W, DEV)
    if tiled:
        Wd = caee.pack_weights(Wd, shape.w_dtype)
    got = gpu_layer(shape, inp, tau, n_bins, Wd, DEV, rule=rule, refill=refill, seed=rseed, keep_top1=keep_top1)
    get, get_sh = getters_np(W, shape.w_dtype)
    ref = oracle_layer(shape, inp, tau, n_bins, get, get_sh, rule=rule, refill=refill, seed=rseed,
                       keep_top1=keep_top1)
    check_route(got, ref, shape.E)
    check_y(got["y"], ref["y"], TOL[shape.w_dtype])
    return got, ref


@pytest.mark.parametrize("seed", range(5))
@pytest.mark.parametrize("tau,n_bins", [(0.0, 1), (0.1, 4), (0.1, 1), (0.3, 4), (0.3, 2)])
def test_tiny_fp32(seed, tau, n_bins):
    _run(TINY_F32, seed, tau, n_bins)


@pytest.mark.parametrize("seed", range(3))
@pytest.mark.parametrize("tau,n_bins", [(0.0, 1), (0.2, 4)])
def test_tiny_bf16(seed, tau, n_bins):
    _run(TINY_BF16, seed, tau, n_bins)


@pytest.mark.parametrize("T", [1, 2, 7, 33, 100, 128])
def test_ragged_batches(T):
    _run(TINY_F32, seed=11, tau=0.2, n_bins=4, T=T)


def test_skewed_popularity_fills_token_blocks():
    # Zipf-skewed logits send most of 128 tokens to a few experts, so experts
    # get several 16-token MFMA column blocks.
    got, ref = _run(TINY_BF16, seed=3, tau=0.05, n_bins=4, T=128, zipf=1.1)
    counts = np.bincount(ref["topk_ids"][ref["topk_ids"] >= 0], minlength=16)
    assert counts.max() > 48


def test_equal_logits_and_resident_experts():
    def flat(inp):
        inp.logits[:] = 0.0
    got, ref = _run(TINY_F32, seed=1, tau=0.3, n_bins=4, mutate=flat)
    # every token routes to experts 0..3 with weight 1/4 < tau; expert 0 is
    # every token's top expert (lowest index), 1..3 share its bin and are pruned
    assert ref["orig_ids"][0].tolist() == [0, 1, 2, 3]
    assert ref["topk_ids"][0].tolist() == [0, -1, -1, -1]
    # (no weight reaches tau and every cost is positive: A_trans would be
    # empty, so expert 0, every token's top expert, was made mandatory)
    assert ref["stats"]["fallback"] == 1 and got["stats"][8] == 1
    got, ref = _run(TINY_F32, seed=1, tau=0.3, n_bins=4, cost_kind="zero")
    assert not ref["pruned"].any()


def test_threshold_above_every_weight():
    # no expert is mandatory and every cost is positive: A_trans would be
    # empty, so each token's top expert is made mandatory; freed slots refill
    # from A_trans
    got, ref = _run(TINY_F32, seed=2, tau=0.9, n_bins=1, T=3)
    assert ref["stats"]["n_pad"] > 0 and ref["stats"]["fallback"] == 1


@pytest.mark.parametrize("keep_top1", [False, True])
@pytest.mark.parametrize("T", [1, 5, 16, 40, 300])
@pytest.mark.parametrize("rule,tau", [("sum", 1.2), ("sum", 2.5), ("max", 0.3)])
def test_step1_literal_and_keep_top1(keep_top1, T, rule, tau):
    # Sec. IV-B step 1 as written (default) and the variant that also keeps
    # every token's top expert, through the single-workgroup (T <= 16) and
    # the multi-kernel routing paths; Zipf costs on 4 bins
    _run(TINY_F32, seed=60 + T, tau=tau, n_bins=4, T=T, zipf=1.1, cost_kind="zipf", rule=rule,
         keep_top1=keep_top1)


def test_expert_ffn_with_given_ids_and_empty_slots():
    shape = TINY_F32
    inp = make_routing_inputs(shape, seed=4)
    W = make_expert_weights_np(shape, seed=4)
    rng = np.random.default_rng(0)
    ids = -np.ones((shape.T, shape.k), np.int32)
    w = np.zeros((shape.T, shape.k), np.float32)
    for t in range(shape.T):
        n = int(rng.integers(0, shape.k + 1))
        ids[t, :n] = rng.choice(shape.E, n, replace=False)
        w[t, :n] = rng.random(n)
    layer = caee.Layer.from_shape(shape)
    ws = caee.alloc_workspace(layer, DEV)
    y = torch.empty((shape.T, shape.d), dtype=torch.float32, device=DEV)
    caee.expert_ffn(layer, to_dev(inp.x, DEV), to_dev(ids, DEV), to_dev(w, DEV), w_to_dev(W, DEV), y, ws)
    torch.cuda.synchronize()
    get, get_sh = getters_np(W, "f32")
    from oracle import swiglu_expert
    x = inp.x.astype(np.float64)
    ref = np.zeros((shape.T, shape.d))
    for t in range(shape.T):
        for j in range(shape.k):
            if ids[t, j] >= 0:
                w13, w2 = get(int(ids[t, j]))
                ref[t] += float(w[t, j]) * swiglu_expert(x[t:t + 1], w13, w2)[0]
    w13, w2 = get_sh(0)
    ref += swiglu_expert(x, w13, w2)
    check_y(y.cpu().numpy().astype(np.float64), ref, 1e-5)


@pytest.mark.parametrize("T", [40, 1100])
def test_expert_ffn_repeated_ids(T):
    # caller-given ids may name one expert twice in a token's list: each
    # occurrence adds its own weight.  40 tokens take the single-workgroup
    # permutation, 1100 the per-1024-token-block one.
    shape = TINY_F32.with_(T=T)
    inp = make_routing_inputs(shape, seed=12)
    W = make_expert_weights_np(shape, seed=12)
    rng = np.random.default_rng(12)
    ids = np.stack([rng.choice(shape.E, shape.k, replace=False) for _ in range(T)]).astype(np.int32)
    rep = rng.random(T) < 0.3
    ids[rep, 1] = ids[rep, 0]                     # a repeated expert
    ids[rng.random(T) < 0.1, 2] = -1              # some empty slots
    w = rng.random((T, shape.k)).astype(np.float32)
    layer = caee.Layer.from_shape(shape)
    ws = caee.alloc_workspace(layer, DEV)
    yfull = torch.full((T + 2, shape.d), 7.0, dtype=torch.float32, device=DEV)
    print(f"expert_ffn repeated ids T={T}", flush=True)
    caee.expert_ffn(layer, to_dev(inp.x, DEV), to_dev(ids, DEV), to_dev(w, DEV), w_to_dev(W, DEV),
                    yfull[1:T + 1], ws)
    torch.cuda.synchronize()
    assert torch.all(yfull[0] == 7.0) and torch.all(yfull[T + 1] == 7.0), "write outside y"
    get, get_sh = getters_np(W, "f32")
    from oracle import swiglu_expert
    x = inp.x.astype(np.float64)
    ref = np.zeros((T, shape.d))
    for e in range(shape.E):
        rows, cols = np.nonzero(ids == e)
        if rows.size:
            w13, w2 = get(e)
            ye = swiglu_expert(x[rows], w13, w2)
            for r, c, v in zip(rows, cols, ye):
                ref[r] += float(w[r, c]) * v
    w13, w2 = get_sh(0)
    ref += swiglu_expert(x, w13, w2)
    check_y(yfull[1:T + 1].cpu().numpy().astype(np.float64), ref, 1e-5)


def test_expert_ffn_without_rows_writes_zeros():
    # every slot empty and no shared expert: no expert rows, y = 0
    shape = TINY_F32.with_(n_shared=0, T=5)
    layer = caee.Layer.from_shape(shape)
    ws = caee.alloc_workspace(layer, DEV)
    W = w_to_dev(make_expert_weights_np(shape, seed=0), DEV)
    x = torch.randn((shape.T, shape.d), device=DEV)
    ids = torch.full((shape.T, shape.k), -1, dtype=torch.int32, device=DEV)
    w = torch.zeros((shape.T, shape.k), device=DEV)
    y = torch.full((shape.T, shape.d), 7.0, device=DEV)
    caee.expert_ffn(layer, x, ids, w, W, y, ws)
    torch.cuda.synchronize()
    assert torch.all(y == 0.0)


def test_empty_batch_leaves_output_untouched():
    shape = TINY_F32.with_(T=0, n_bins=1)
    layer = caee.Layer.from_shape(shape)
    ws = caee.alloc_workspace(layer, DEV)
    W = w_to_dev(make_expert_weights_np(TINY_F32, seed=0), DEV)
    y = torch.full((1, shape.d), 3.0, device=DEV)
    z = torch.zeros((1, 16), device=DEV)
    caee.moe_layer(layer, y, z, None, z[0], None, W, y, ws)
    torch.cuda.synchronize()
    assert torch.all(y == 3.0)


def test_deterministic_repeat():
    shape = TINY_BF16.with_(T=64)
    inp = make_routing_inputs(shape, seed=9, zipf_logit_s=1.1)
    Wd = w_to_dev(make_expert_weights_np(shape, seed=9), DEV)
    a = gpu_layer(shape, inp, 0.1, 4, Wd, DEV)
    b = gpu_layer(shape, inp, 0.1, 4, Wd, DEV)
    assert np.array_equal(a["y"], b["y"]) and np.array_equal(a["topk_w"], b["topk_w"])


@pytest.mark.parametrize("T", [300, 1100, 1101])
def test_large_batches(T):
    # the shared expert has T > 128 rows, so it spans several FFN chunks;
    # 1100 tokens also takes the permutation path used above 1024 tokens,
    # and an odd count leaves the combine's last pair of tokens with one
    _run(TINY_F32, seed=21, tau=0.1, n_bins=4, T=T)


@pytest.mark.parametrize("seed", range(3))
@pytest.mark.parametrize("rule,tau,n_bins", [("sum", 0.5, 4), ("sum", 1.5, 1), ("sum", 0.0, 4),
                                             ("cir", 0.7, 4), ("cir", 0.9, 2), ("cir", 1.0, 4),
                                             ("cir", 0.3, 1)])
def test_importance_rules(seed, rule, tau, n_bins):
    got, ref = _run(TINY_F32, seed=40 + seed, tau=tau, n_bins=n_bins, rule=rule)
    if rule == "cir" and tau == 1.0:
        assert not ref["pruned"].any()


def test_sum_rule_with_equal_weights():
    # equal logits: every token gives 1/4 to experts 0..3, so I(e) = T/4 exactly
    def flat(inp):
        inp.logits[:] = 0.0
    _run(TINY_F32, seed=2, tau=4.0, n_bins=4, mutate=flat, rule="sum")
    _run(TINY_F32, seed=2, tau=4.5, n_bins=4, mutate=flat, rule="sum")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_tiled_layout_order(dtype):
    # the documented tiled order, restated with numpy: block (t, s) holds 64
    # 16-byte pieces, piece r + 16q = bytes [64s + 16q, +16) of row 16t + r
    rows, cols, count = 48, 128 if dtype == "bf16" else 64, 3
    rng = np.random.default_rng(0)
    src = rng.integers(0, 2**31, (count, rows, cols * (2 if dtype == "bf16" else 4) // 4), dtype=np.int64)
    src = src.astype(np.uint32)
    row_bytes = src.shape[2] * 4
    pieces = src.reshape(count, rows, row_bytes // 16, 4)          # 16-byte pieces of each row
    S = row_bytes // 64
    want = np.empty((count, rows // 16, S, 64, 4), np.uint32)
    for t in range(rows // 16):
        for s_ in range(S):
            for j in range(64):
                want[:, t, s_, j] = pieces[:, 16 * t + (j % 16), 4 * s_ + j // 16]
    dsrc = torch.from_numpy(src.view(np.int32)).to(DEV)
    ddst = torch.empty_like(dsrc)
    caee.pack_matrix(dtype, dsrc, ddst, rows, cols, count)
    torch.cuda.synchronize()
    assert np.array_equal(ddst.cpu().numpy().view(np.uint32).reshape(want.shape), want)


# 1, 3 and 16 tokens: the routing launch runs the shared expert's gate/up;
# 40, 70 and 130 tokens: big chunks (the bf16 GEMM); the down contraction
# (f = 128) is 4 or 8 steps.
@pytest.mark.parametrize("shape", [TINY_F32, TINY_BF16], ids=["f32", "bf16"])
@pytest.mark.parametrize("T", [1, 3, 16, 40, 70, 130])
def test_tiled_weights(shape, T):
    _run(shape, seed=T, tau=0.2, n_bins=4, T=T, tiled=True)


@pytest.mark.parametrize("refill", ["none", "random", "literal"])
@pytest.mark.parametrize("T", [5, 16, 40])
@pytest.mark.parametrize("seed", [0, 3])
def test_tiny_refill_variants(refill, T, seed):
    """Compensation variants (no refill; random refill by SplitMix64 keys;
    the literal top-k of the masked keys) against the oracle, through both
    routing paths."""
    got, ref = _run(TINY_F32, seed=seed, tau=0.7, n_bins=1, T=T, zipf=1.2, cost_kind="zipf", rule="cir",
                    refill=refill, rseed=11 + seed)
    if refill == "none":
        assert got["stats"][6] == 0
