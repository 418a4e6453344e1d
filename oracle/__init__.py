"""CAEE reference oracle (fp64, CPU) -- TEST INFRASTRUCTURE ONLY.

This package is the independent checker of the HIP implementation.  Only the
test-suite, the smoke check and the benchmark's CPU-baseline leg may import
it; the product path (the C-ABI library and its Python binding) never does,
and the oracle never imports the product package.  The two share no code:
the only common dependency is ``synth_inputs``, which draws seeded random
inputs and holds none of the method's arithmetic.

Everything is plain numpy in float64, written step by step in the order of
the paper (Cost-Aware Expert Execution, arxiv 2606.29982):

  routing.py       sigmoid router scores, group-limited top-k, gate weights
                   (the MoE output equation of Sec. II-A; group routing as
                   the DeepSeek layer defines it)
  pruning.py       importance, mandatory/candidate split, baseline cost,
                   cost-invariant expansion, final pruning (Sec. IV-B,
                   steps 1-4, with the cost model of Sec. IV-A)
  compensation.py  masking and final top-k re-selection (Sec. IV-C)
  ffn.py           SwiGLU expert FFN and weighted combine (Sec. II-A), and
                   the OCP e4m3 codec used for 8-bit weights/activations
  layer.py         the whole layer, chaining the above
  offload.py       residency cost table and the LRU device cache (Sec. IV-A, V-B)
  calibration.py   the least-squares fit of the cost model's alpha and beta
                   (Sec. IV-A, offline calibration)
  margins.py       the gap of every routing / pruning decision to its flip
                   (near-ties between two correct implementations)

Where the paper is silent or ambiguous the reading taken is stated in the
docstring of the function that takes it.  Routing and pruning decisions are
taken in float64 here; the kernel takes them in float64 too, so selected and
pruned expert indices are expected to match bit for bit.
"""
from .routing import sigmoid_scores, group_limited_topk, gate_weights, route_batch  # noqa: F401
from .pruning import (importance_max, importance_sum, cir_mandatory, mandatory_split,  # noqa: F401
                      bin_loads, cost_aware_greedy, prune_batch)
from .compensation import compensate_token, compensate_batch  # noqa: F401
from .ffn import (bf16_bits_to_f64, e4m3_decode, e4m3_encode_rne,  # noqa: F401
                  quantize_e4m3_blocks, swiglu_expert, expert_weights_f64)
from .layer import moe_layer_ref  # noqa: F401
from .calibration import fit_alpha_beta, fit_grouped, cost_of  # noqa: F401
from .margins import decision_margins  # noqa: F401
