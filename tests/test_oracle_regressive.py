"""Pins for the MLP regressive block (the components ablation: Sec. 3.2 last paragraph and
Sec. 4.3 "Ablations on Components" replace the Attention Decoder by an MLP over the two
input vectors concatenated), read as h_i = h_{i-1} + SiLU(W_r [RMSNorm_r(h_{i-1}); e_{i-1}] + b_r).

- closed form: with the state half of W_r zero, the embedding half alpha I and head MLPs
  that add nothing (W1 = 0, b1 = -200), the state at node n is h_0 plus the sum over the
  tokens m on n's root path of SiLU(alpha e(tok_m) + b_r), element by element, and its
  drafted logits are W_lm RMSNorm_f(state); planted mistakes (no recursion, the two halves
  swapped, the root token at every depth) fail it;
- with the embedding half zero the block cannot see the previous token: every node of a
  depth gets the same logits, so every parent expands the same children;
- greedy speculative output equals greedy autoregressive output.
"""
import inspect
import textwrap

import numpy as np
import pytest
import torch

import synth
import oracle
import oracle.clover as oc
from tests.test_oracle_base import _torch_forward_full


def _rms(x, g, eps):
    return x / np.sqrt(np.mean(x * x) + eps) * g


def _cfg(**kw):
    return synth.tiny_test_config(regressive="mlp", ab="none", topk=(3, 2, 2), tree_tokens=12, **kw)


def mlp_path_sum_pin(alpha=1.7, seed=21):
    cfg = _cfg()
    w = synth.make_weights(cfg, seed=seed, perturb=True)
    d = cfg.d_model
    w["rb.w"] = torch.cat([torch.zeros(d, d), torch.eye(d) * alpha], dim=1)
    for j in range(cfg.n_spec_heads):
        w[f"head{j}.w1"] = w[f"head{j}.w1"] * 0
        w[f"head{j}.b1"] = torch.full_like(w[f"head{j}.b1"], -200.0)
    o = oracle.CloverOracle(cfg, w)
    prompt = synth.make_prompt(cfg, n=9)
    st = o.prefill(prompt)
    h0 = _torch_forward_full(cfg, w, prompt, residual=True)[-1]
    W = {k: v.double().numpy() for k, v in w.items()}
    a = W["rb.w"][0, d]  # alpha as stored (fp32)
    c = o.draft(st)
    err = float(np.max(np.abs(st.h0 - h0)))
    for n, logits in c.row_logits.items():
        s = h0.copy()
        m = n
        while m >= 0:
            row = W["lm_head"][c.token[m]]
            z = a * row / np.linalg.norm(row) + W["rb.b"]
            s = s + z / (1 + np.exp(-z))
            m = c.parent[m]
        want = W["lm_head"] @ _rms(s, W["final_norm"], cfg.rms_eps)
        err = max(err, float(np.max(np.abs(logits - want))))
    assert len(c.row_logits) == 1 + 3 + 6
    return err


def test_mlp_regressive_path_sum_closed_form():
    assert mlp_path_sum_pin() < 1e-10


def _mutated(fn, old, new):
    src = textwrap.dedent(inspect.getsource(fn))
    assert src.count(old) == 1, old
    ns = dict(vars(oc))
    exec(compile(src.replace(old, new), f"<mutated {fn.__name__}>", "exec"), ns)
    return ns[fn.__name__]


@pytest.mark.parametrize("target,old,new", [
    ("regressive_mlp", "x = np.concatenate([a, prec.store(e)])", "x = np.concatenate([prec.store(e), a])"),
    ("draft", "state[len(depth) - 1] = s", "state[len(depth) - 1] = st.h0"),
    ("draft", 'rc_embed(self.w["lm_head"], token[n]), self.w', 'rc_embed(self.w["lm_head"], token[0]), self.w'),
])
def test_mlp_path_sum_pin_catches(monkeypatch, target, old, new):
    assert mlp_path_sum_pin() < 1e-10
    if target == "draft":
        monkeypatch.setattr(oc.CloverOracle, "draft", _mutated(oc.CloverOracle.draft, old, new))
    else:
        monkeypatch.setattr(oc, target, _mutated(getattr(oc, target), old, new))
    assert mlp_path_sum_pin() > 1e-6


def test_without_the_embedding_half_the_block_ignores_the_previous_token():
    cfg = _cfg()
    w = synth.make_weights(cfg, seed=3, perturb=True)
    d = cfg.d_model
    w["rb.w"] = torch.cat([w["rb.w"][:, :d], torch.zeros(d, d)], dim=1)
    o = oracle.CloverOracle(cfg, w)
    st = o.prefill(synth.make_prompt(cfg, n=10))
    c = o.draft(st)
    for depth in (1, 2):
        rows = [lg for n, lg in c.row_logits.items() if c.depth[n] == depth]
        assert len(rows) > 1
        for lg in rows[1:]:
            assert np.array_equal(lg, rows[0])
    # with the embedding half in place the rows of a depth differ
    w2 = synth.make_weights(cfg, seed=3, perturb=True)
    c2 = oracle.CloverOracle(cfg, w2).draft(o.prefill(synth.make_prompt(cfg, n=10)))
    rows2 = [lg for n, lg in c2.row_logits.items() if c2.depth[n] == 1]
    assert np.max(np.abs(rows2[0] - rows2[1])) > 1e-6


@pytest.mark.parametrize("seed,ab", [(0, "none"), (1, "default")])
def test_mlp_regressive_speculative_equals_greedy(seed, ab):
    cfg = synth.tiny_test_config(regressive="mlp", ab=ab, topk=(3, 2, 2), tree_tokens=12)
    o = oracle.CloverOracle(cfg, synth.make_weights(cfg, seed=seed, perturb=True))
    prompt = synth.make_prompt(cfg, seq=seed, n=12)
    spec, _ = o.generate(prompt, 14)
    assert spec == o.base.greedy_generate(prompt, 14)
