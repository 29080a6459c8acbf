"""Canonical weight list and seeded random-init weights.

Every tensor is drawn from N(0, 0.02^2) with its own seeded generator; norm
gains are 1 and biases 0 unless ``perturb`` is set (tests use that so gains and
biases are exercised).  bf16 workloads round the drawn fp32 values to bf16
(round to nearest even, done by torch's dtype conversion).
"""
from typing import Dict, List, Tuple

import torch

from .configs import CloverConfig

_LAYER = ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "w_gate", "w_up", "w_down")


def _layer_specs(prefix: str, c: CloverConfig, attn: bool = True,
                 mlp: bool = True) -> List[Tuple[str, Tuple[int, ...]]]:
    d, F = c.d_model, c.ffn_dim
    shapes = {
        "attn_norm": (d,), "wq": (c.q_dim, d), "wk": (c.kv_dim, d), "wv": (c.kv_dim, d),
        "wo": (d, c.q_dim), "mlp_norm": (d,), "w_gate": (F, d), "w_up": (F, d), "w_down": (d, F),
    }
    return [(f"{prefix}.{n}", shapes[n]) for i, n in enumerate(_LAYER) if (attn if i < 5 else mlp)]


def weight_specs(c: CloverConfig) -> List[Tuple[str, Tuple[int, ...]]]:
    """Canonical (name, shape) order; the C library exports the same list."""
    d, V = c.d_model, c.vocab
    specs: List[Tuple[str, Tuple[int, ...]]] = [("emb", (V, d))]
    for l in range(c.n_layers):
        specs += _layer_specs(f"layer{l}", c)
    specs += [("final_norm", (d,)), ("lm_head", (V, d))]
    if c.ab_kind != "none":  # the Augmenting Block's halves
        specs += _layer_specs("ab", c, attn=c.ab_kind in ("full", "attn"), mlp=c.ab_kind in ("full", "mlp"))
    if c.draft != "medusa" and c.regressive == "mlp":  # MLP regressive block over [RMSNorm(h); e]
        specs += [("rb.norm", (d,)), ("rb.w", (d, 2 * d)), ("rb.b", (d,))]
    elif c.draft != "medusa":  # Attention Decoder: Clover heads only; shared, or one per head
        qd = c.n_heads * c.head_dim
        for pre in ([f"ad{j}" for j in range(c.n_spec_heads)] if c.ad_per_head else ["ad"]):
            specs += [(f"{pre}.norm", (d,)), (f"{pre}.wq", (qd, d)), (f"{pre}.wk", (qd, d)),
                      (f"{pre}.wv", (qd, d)), (f"{pre}.wo", (d, qd))]
    for j in range(c.n_spec_heads):
        specs += [(f"head{j}.w1", (d, d)), (f"head{j}.b1", (d,))]
        if c.draft == "medusa" and c.medusa_lm == "per_head":
            specs += [(f"head{j}.lm", (V, d))]
    return specs


def is_bias(name: str) -> bool:
    return name.endswith(".b1") or name == "rb.b"


def is_matrix(name: str) -> bool:
    return not (name.endswith("norm") or is_bias(name))


def _gen(seed: int, idx: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed((seed * 1_000_003 + idx * 7_919 + 12_345) & 0x7FFF_FFFF_FFFF_FFFF)
    return g


def make_weights(c: CloverConfig, seed: int = 0, device="cpu", perturb: bool = False,
                 names=None) -> Dict[str, torch.Tensor]:
    """Return {name: tensor} in the storage dtype on ``device``.

    Values depend on the device whose generator draws them; a test that needs the
    same weights on both sides draws them once and copies them.
    """
    dt = torch.bfloat16 if c.dtype == "bf16" else torch.float32
    out: Dict[str, torch.Tensor] = {}
    for i, (name, shape) in enumerate(weight_specs(c)):
        if names is not None and name not in names:
            continue
        g = _gen(seed, i, device)
        if name.endswith("norm"):
            t = torch.ones(shape, device=device)
            if perturb:
                t = t + 0.1 * torch.randn(shape, generator=g, device=device)
        elif is_bias(name):
            t = torch.zeros(shape, device=device)
            if perturb:
                t = 0.02 * torch.randn(shape, generator=g, device=device)
        else:
            t = torch.randn(shape, generator=g, device=device, dtype=torch.float32) * 0.02
        out[name] = t.to(dt)
    return out
