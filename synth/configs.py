"""Workload shapes.

The model shapes stand in for the paper's Baichuan-Small (7B) and
Baichuan-Large (>100B) settings (Sec. 4.1, "Models and baselines"); the trained
weights and the internal evaluation dialogues are not available, so weights are
random-init and prompts are uniform-random tokens.  The Clover speculator uses
3 heads as in Sec. 4.1 (4 on the large shape).
"""
from dataclasses import dataclass, field, replace
from typing import Tuple


@dataclass(frozen=True)
class CloverConfig:
    name: str
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    dtype: str                 # "f32" or "bf16": storage type of weights, GEMM inputs, KV
    topk: Tuple[int, ...]      # per-depth branching of the candidate tree; len == number of heads
    tree_tokens: int           # verify tokens per sequence, root included
    batch: int = 1
    prompt_len: Tuple[int, int] = (128, 128)   # inclusive range of prompt lengths
    steps: int = 16
    max_context: int = 4096
    rms_eps: float = 1e-6
    rope_theta: float = 10000.0
    kv_block: int = 16
    draft: str = "clover"      # speculator: "clover" heads or the "medusa" baseline
    # Augmenting Block: "full" layer, "attn" or "mlp" half only, "none"; "default" is
    # "full" for the Clover draft and "none" for the Medusa draft
    ab: str = "default"
    # key set of the Attention Decoder: "single" {e}, "two" {RMSNorm(h), e}, "path" {e_0..}
    ad_keys: str = "single"
    ad_per_head: bool = False  # one Attention Decoder per head instead of one shared
    # regressive block of the Clover draft: the "attention" decoder (Eq. 1-2) or the "mlp"
    # over [RMSNorm(h); e] of the ablation (Sec. 3.2 last paragraph, Sec. 4.3)
    regressive: str = "attention"
    # Medusa draft: the heads "shared" the target's LM head, or each has its own ("per_head",
    # the original Medusa, Sec. 3.4)
    medusa_lm: str = "shared"
    temperature: float = 0.0   # 0: greedy; > 0: the target samples (speculative sampling)
    sample_seed: int = 0

    @property
    def ab_kind(self) -> str:
        if self.ab != "default":
            return self.ab
        return "none" if self.draft == "medusa" else "full"

    @property
    def n_spec_heads(self) -> int:
        return len(self.topk)

    @property
    def q_dim(self) -> int:
        return self.n_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    def n_candidates(self) -> int:
        """Nodes of the fully expanded per-depth top-k tree, root excluded."""
        total, width = 0, 1
        for k in self.topk:
            width *= k
            total += width
        return total

    def with_(self, **kw) -> "CloverConfig":
        return replace(self, **kw)


CONFIGS = {
    # tiny fp32 correctness workload: 2 layers, d=256, 4x64 heads, FFN 688, vocab 1024
    "tiny_fp32": CloverConfig(
        name="tiny_fp32", n_layers=2, d_model=256, n_heads=4, n_kv_heads=4, head_dim=64,
        ffn_dim=688, vocab=1024, dtype="f32", topk=(4, 3, 2), tree_tokens=41,
        batch=1, prompt_len=(128, 128), steps=16, max_context=512),
    # 7B-shape bf16, batch 1, 1024-token prompt, 64-token tree from top-k (8,4,2)
    "llama7b_b1": CloverConfig(
        name="llama7b_b1", n_layers=32, d_model=4096, n_heads=32, n_kv_heads=32, head_dim=128,
        ffn_dim=11008, vocab=125696, dtype="bf16", topk=(8, 4, 2), tree_tokens=64,
        batch=1, prompt_len=(1024, 1024), steps=128, max_context=1024 + 128 * 4 + 128),
    # 7B-shape bf16, batch 8, prompts of 2048..4096 tokens, paged KV
    "llama7b_b8": CloverConfig(
        name="llama7b_b8", n_layers=32, d_model=4096, n_heads=32, n_kv_heads=32, head_dim=128,
        ffn_dim=11008, vocab=125696, dtype="bf16", topk=(8, 4, 2), tree_tokens=64,
        batch=8, prompt_len=(2048, 4096), steps=64, max_context=4096 + 64 * 4 + 128),
    # large dense GQA bf16 shape that fits one 288 GB device, 4 heads
    "large_gqa_b1": CloverConfig(
        name="large_gqa_b1", n_layers=80, d_model=8192, n_heads=64, n_kv_heads=8, head_dim=128,
        ffn_dim=28672, vocab=125696, dtype="bf16", topk=(8, 4, 2, 2), tree_tokens=64,
        batch=1, prompt_len=(2048, 2048), steps=64, max_context=2048 + 64 * 5 + 128),
}
# the same shapes with the Medusa baseline as speculator (no Augmenting Block or Attention
# Decoder; heads on the last hidden state, Cartesian-product tree)
for _n in ("tiny_fp32", "llama7b_b1", "llama7b_b8", "large_gqa_b1"):
    CONFIGS[_n + "_medusa"] = CONFIGS[_n].with_(name=_n + "_medusa", draft="medusa")

# tree-size sweep on the 7B shape: (tree tokens incl. root, per-depth top-k)
SWEEP_TREES = ((16, (4, 2, 2)), (32, (4, 3, 2)), (64, (8, 4, 2)), (128, (16, 4, 2)))
SWEEP_CONTEXTS = (512, 4096, 16384, 32768)


def get_config(name: str) -> CloverConfig:
    return CONFIGS[name]


def tiny_test_config(**kw) -> CloverConfig:
    """A reduced variant of the tiny workload for fast brute-force checks."""
    base = CONFIGS["tiny_fp32"].with_(name="tiny_test", n_layers=2, d_model=64, n_heads=2,
                                      n_kv_heads=2, head_dim=32, ffn_dim=96, vocab=97,
                                      prompt_len=(12, 12), steps=6, max_context=128)
    return base.with_(**kw)
