"""CPU oracle for one Clover speculate-and-verify step (test infrastructure).

A plain, slow, float64 NumPy implementation of what the GPU path computes,
written from the paper (Clover: Regressive Lightweight Speculative Decoding
with Sequential Knowledge, arXiv 2405.00263).  Only the tests, the smoke entry
and the benchmark's CPU-baseline leg may import it; the product path never
does, and it shares no code with the HIP library.

Precision model: arithmetic is float64.  For bf16 workloads the values that the
GPU path stores in bf16 (weights, GEMM inputs, rotated queries and the KV
cache) are rounded to bf16 at the same points (``Precision.store``), so the
two sides differ only by accumulation order and fp32-vs-fp64 rounding.

Parity status per function (see each docstring): every function is pinned by an
invariant test.  The composition of the Clover draft (Augmenting Block -> Attention
Decoder -> head MLP -> shared LM head) is pinned by closed forms (single-key decoder,
identity heads, the path sum of W_O W_V e along each root path); its wiring itself
comes from readings of Sec. 3, because the architecture figure is not available.
"""
from .model import (Precision, rmsnorm, rope, attention, silu, logsumexp,  # noqa: F401
                    LayerWeights, layer_forward, BaseModel)
from .clover import (CloverOracle, SeqState, Tree, Candidates, build_tree, tree_mask,  # noqa: F401
                     accept, rc_embed, attention_decoder, topk_ids)
from .medusa import MedusaOracle  # noqa: F401


def make_oracle(cfg, weights):
    """The oracle of the workload's speculator (Clover heads or the Medusa baseline)."""
    return MedusaOracle(cfg, weights) if getattr(cfg, "draft", "clover") == "medusa" else CloverOracle(cfg, weights)
