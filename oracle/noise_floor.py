"""Noise floor of the bf16 precision model through depth (test infrastructure).

The oracle computes in float64 and rounds to bf16 at the points where the GPU stores bf16
(``Precision.store``).  Any implementation that keeps those storage points but sums its
dot products in another order (the GPU sums in fp32, in its own order) rounds a few
elements to the neighbouring bf16 value; the following layers carry these one-step
differences along and add their own.  This script measures how far two such valid
orders drift apart: the oracle's layer (float64 sums) against the same layer written with
float32 matrix products, both from the same embedding rows, layer after layer, at a
workload's shape with random-init weights.  It prints the residual stream's relative
difference after each layer and the logits' max-abs and mean-abs difference at the end.

    python -m oracle.noise_floor llama7b_b1 [layers] [rows]

Measured at the 7B shape (32 layers, 64 causal rows of a uniform-random prompt, weights
drawn on the CPU): the residual streams differ by 2.0e-2 of their rms after the last
layer, and the logits by 0.152 max-abs and 0.021 mean-abs (logit std 1.28); the argmax of
every row agrees.
"""
import sys
import time

import numpy as np

from .model import LayerWeights, Precision, attention, layer_forward, rmsnorm, rope, silu


def _mm32(a, w):
    """a @ w.T with float32 operands and float32 accumulation (both hold bf16 values)."""
    return (np.asarray(a, np.float32) @ np.asarray(w, np.float32).T).astype(np.float64)


def layer_f32_sums(x, pos, lw: LayerWeights, causal, cfg, prec: Precision):
    """The oracle's pre-norm layer on rows that see each other causally (no cache), with
    every matrix product summed in float32 instead of float64."""
    n, H, Hk, hd = x.shape[0], cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    st = prec.store
    a = st(rmsnorm(x, lw.attn_norm, cfg.rms_eps))
    q = st(rope(_mm32(a, lw.wq).reshape(n, H, hd), pos, cfg.rope_theta))
    k = st(rope(_mm32(a, lw.wk).reshape(n, Hk, hd), pos, cfg.rope_theta))
    v = st(_mm32(a, lw.wv).reshape(n, Hk, hd))
    o = attention(q, k, v, causal).reshape(n, H * hd)
    x = x + _mm32(st(o), lw.wo)
    m = st(rmsnorm(x, lw.mlp_norm, cfg.rms_eps))
    act = st(silu(_mm32(m, lw.w_gate)) * _mm32(m, lw.w_up))
    return x + _mm32(act, lw.w_down)


def measure(cfg, n_layers=None, rows=64, seed=0, log=print):
    """Returns (per-layer rms(dx)/rms(x), logits max-abs, logits mean-abs)."""
    import torch
    import synth
    prec = Precision(cfg.dtype)
    fields = list(LayerWeights.__dataclass_fields__)

    def fetch(names):
        w = synth.make_weights(cfg, seed=seed, device="cpu", names=set(names))
        return {k: v.double().numpy() for k, v in w.items()}

    toks = synth.make_prompt(cfg, n=rows)
    xa = synth.make_weights(cfg, seed=seed, device="cpu", names={"emb"})["emb"][torch.tensor(toks)].double().numpy()
    xb = xa.copy()
    pos = np.arange(rows)
    causal = np.tril(np.ones((rows, rows), dtype=bool))
    z = np.zeros((0, cfg.n_kv_heads, cfg.head_dim))
    rel = []
    t0 = time.time()
    for l in range(cfg.n_layers if n_layers is None else n_layers):
        lw = LayerWeights.from_dict(fetch([f"layer{l}.{f}" for f in fields]), f"layer{l}")
        xa, _, _ = layer_forward(xa, pos, lw, z, z, causal, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim,
                                 cfg.rms_eps, cfg.rope_theta, prec)
        xb = layer_f32_sums(xb, pos, lw, causal, cfg, prec)
        rms = float(np.sqrt(np.mean(xa * xa)))
        rel.append(float(np.sqrt(np.mean((xa - xb) ** 2))) / rms)
        log(f"layer {l}: rms(x) {rms:.3f}  rms(dx)/rms(x) {rel[-1]:.3e}  ({time.time() - t0:.0f} s)")
    w = fetch(["final_norm", "lm_head"])
    la = prec.store(rmsnorm(xa, w["final_norm"], cfg.rms_eps)) @ w["lm_head"].T
    lb = prec.store(rmsnorm(xb, w["final_norm"], cfg.rms_eps)) @ w["lm_head"].T
    d = np.abs(la - lb)
    log(f"logits: max |d| {d.max():.3e}  mean |d| {d.mean():.3e}  logit std {la.std():.3f}  "
        f"argmax agreement {np.mean(np.argmax(la, 1) == np.argmax(lb, 1)):.3f}")
    return rel, float(d.max()), float(d.mean())


if __name__ == "__main__":
    import synth
    cfg = synth.get_config(sys.argv[1] if len(sys.argv) > 1 else "llama7b_b1")
    measure(cfg, int(sys.argv[2]) if len(sys.argv) > 2 else None, int(sys.argv[3]) if len(sys.argv) > 3 else 64,
            log=lambda m: print(m, flush=True))
