"""Base transformer of the oracle (Llama-style pre-norm decoder).

Test infrastructure only.  The paper fixes no architecture for the target
model beyond "a transformer LLM"; the workloads are Llama-style (RMSNorm,
rotary embedding with rotate-half pairing, SwiGLU MLP, optional grouped KV
heads), eps 1e-6 and rotary base 10000.

Tree attention (Sec. 2.2): a query attends to every committed key plus the
keys of tree nodes its mask row admits; the mask is the tree's ancestor
matrix.  ``layer_forward`` takes that visibility as an explicit boolean matrix.
"""
from dataclasses import dataclass
from typing import Callable, Dict, List, Optional, Tuple

import numpy as np


def _round_bf16(x) -> np.ndarray:
    """Round to fp32 (nearest even), then to bf16 (nearest even); return float64."""
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000).astype(np.uint32)
    return r.view(np.float32).astype(np.float64)


class Precision:
    """Where a value is stored in the workload's storage type.

    f32 workloads: identity (float64 throughout).  bf16 workloads: the value is
    rounded to bf16, as the GPU stores it.
    """

    def __init__(self, dtype: str):
        assert dtype in ("f32", "bf16")
        self.dtype = dtype

    def store(self, x) -> np.ndarray:
        if self.dtype == "bf16":
            return _round_bf16(x)
        return np.asarray(x, dtype=np.float64)


def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """RMSNorm over the last axis: x / sqrt(mean(x^2) + eps) * g."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def rope(x: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotary embedding, rotate-half pairing (i, i + hd/2).

    x: [n, heads, hd]; pos: [n] integer positions.
    """
    hd = x.shape[-1]
    half = hd // 2
    inv = theta ** (-np.arange(half, dtype=np.float64) * 2.0 / hd)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv[None, :]       # [n, half]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def logsumexp(z: np.ndarray, axis=-1) -> np.ndarray:
    m = np.max(z, axis=axis, keepdims=True)
    return (m + np.log(np.sum(np.exp(z - m), axis=axis, keepdims=True))).squeeze(axis)


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, visible: np.ndarray) -> np.ndarray:
    """Masked softmax attention with grouped KV heads.

    q: [nq, Hq, hd]; k, v: [nk, Hkv, hd]; visible: [nq, nk] bool.  Query head h
    reads KV head h // (Hq // Hkv); scores are scaled by 1/sqrt(hd).
    """
    nq, Hq, hd = q.shape
    Hkv = k.shape[1]
    grp = Hq // Hkv
    out = np.zeros_like(q)
    for h in range(Hq):
        kh, vh = k[:, h // grp, :], v[:, h // grp, :]
        s = (q[:, h, :] @ kh.T) / np.sqrt(hd)                         # [nq, nk]
        s = np.where(visible, s, -np.inf)
        s = s - np.max(s, axis=1, keepdims=True)
        p = np.exp(s)
        p = p / np.sum(p, axis=1, keepdims=True)
        out[:, h, :] = p @ vh
    return out


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


@dataclass
class LayerWeights:
    attn_norm: np.ndarray
    wq: np.ndarray
    wk: np.ndarray
    wv: np.ndarray
    wo: np.ndarray
    mlp_norm: np.ndarray
    w_gate: np.ndarray
    w_up: np.ndarray
    w_down: np.ndarray

    @staticmethod
    def from_dict(w: Dict[str, np.ndarray], prefix: str, partial: bool = False) -> "LayerWeights":
        """partial: tensors of a half the layer does not have (Augmenting Block variants) are None."""
        return LayerWeights(**{f: (w.get(f"{prefix}.{f}") if partial else w[f"{prefix}.{f}"])
                               for f in LayerWeights.__dataclass_fields__})


def layer_forward(x: np.ndarray, pos: np.ndarray, lw: LayerWeights, k_prefix: np.ndarray,
                  v_prefix: np.ndarray, tail_visible: np.ndarray, n_heads: int, n_kv: int,
                  head_dim: int, eps: float, theta: float, prec: Precision, attn: bool = True,
                  mlp: bool = True):
    """One pre-norm decoder layer over new rows ``x`` at positions ``pos``.

    The new rows see all ``k_prefix``/``v_prefix`` keys and the new rows' own keys
    where ``tail_visible`` is set.  Returns (x_out, k_new, v_new) with k_new after
    rotary, both in storage precision (what a KV cache holds).  ``attn`` / ``mlp``
    keep the attention / MLP half (the Augmenting Block variants of Sec. 4.3); without
    the attention half k_new and v_new are None.
    """
    k = v = None
    if attn:
        x, k, v = _attention_half(x, pos, lw, k_prefix, v_prefix, tail_visible, n_heads, n_kv,
                                  head_dim, eps, theta, prec)
    if mlp:
        m = prec.store(rmsnorm(x, lw.mlp_norm, eps))
        act = prec.store(silu(m @ lw.w_gate.T) * (m @ lw.w_up.T))
        x = x + act @ lw.w_down.T
    return x, k, v


def _attention_half(x, pos, lw, k_prefix, v_prefix, tail_visible, n_heads, n_kv, head_dim, eps,
                    theta, prec):
    n = x.shape[0]
    a = prec.store(rmsnorm(x, lw.attn_norm, eps))
    q = rope((a @ lw.wq.T).reshape(n, n_heads, head_dim), pos, theta)
    k = rope((a @ lw.wk.T).reshape(n, n_kv, head_dim), pos, theta)
    v = (a @ lw.wv.T).reshape(n, n_kv, head_dim)
    q, k, v = prec.store(q), prec.store(k), prec.store(v)
    keys = np.concatenate([k_prefix, k], axis=0)
    vals = np.concatenate([v_prefix, v], axis=0)
    visible = np.concatenate([np.ones((n, k_prefix.shape[0]), dtype=bool), tail_visible], axis=1)
    o = attention(q, keys, vals, visible).reshape(n, n_heads * head_dim)
    return x + prec.store(o) @ lw.wo.T, k, v


class BaseModel:
    """The frozen target model: embedding, N decoder layers, final norm, LM head."""

    def __init__(self, cfg, weights: Dict[str, np.ndarray]):
        self.cfg = cfg
        self.w = weights
        self.prec = Precision(cfg.dtype)
        self.layers = [LayerWeights.from_dict(weights, f"layer{l}") for l in range(cfg.n_layers)]

    def run_layer(self, lw: LayerWeights, x, pos, kp, vp, tail_visible):
        c = self.cfg
        return layer_forward(x, pos, lw, kp, vp, tail_visible, c.n_heads, c.n_kv_heads,
                             c.head_dim, c.rms_eps, c.rope_theta, self.prec)

    def empty_kv(self) -> Tuple[np.ndarray, np.ndarray]:
        c = self.cfg
        z = np.zeros((0, c.n_kv_heads, c.head_dim))
        return z, z.copy()

    def logits(self, x_last: np.ndarray) -> np.ndarray:
        """Final RMSNorm and LM head; x_last is the residual after the last layer."""
        c = self.cfg
        return self.prec.store(rmsnorm(x_last, self.w["final_norm"], c.rms_eps)) @ self.w["lm_head"].T

    def forward_rows(self, tokens, pos, kv: Optional[List[Tuple[np.ndarray, np.ndarray]]],
                     tail_visible: np.ndarray):
        """Run new tokens through all layers against per-layer KV prefixes.

        Returns (x_N [n, d], per-layer (k_new, v_new)).
        """
        x = self.w["emb"][np.asarray(tokens)]
        pos = np.asarray(pos)
        new_kv = []
        for l, lw in enumerate(self.layers):
            kp, vp = kv[l] if kv is not None else self.empty_kv()
            x, k, v = self.run_layer(lw, x, pos, kp, vp, tail_visible)
            new_kv.append((k, v))
        return x, new_kv

    def forward_full(self, tokens) -> np.ndarray:
        """Causal forward over a whole token sequence without a cache; returns logits [n, V]."""
        n = len(tokens)
        x, _ = self.forward_rows(tokens, np.arange(n), None, np.tril(np.ones((n, n), dtype=bool)))
        return self.logits(x)

    def greedy_generate(self, prompt, n_new: int) -> List[int]:
        """Plain greedy autoregressive decoding by full recompute (no KV cache).

        The speculative path must reproduce these tokens exactly (Sec. 1 and 2.1:
        speculative decoding keeps the target model's outputs).
        """
        seq = list(prompt)
        out = []
        for _ in range(n_new):
            t = int(np.argmax(self.forward_full(seq)[-1]))
            out.append(t)
            seq.append(t)
        return out
