"""Pins for the Attention Decoder key-set readings (Eq. 1-2; Sec. 3.2).

- The multi-key decoder's attention equals torch's scaled-dot-product attention (a
  library routine) on the same projected query, keys and values.
- Path keys: a depth-1 node's root path is the root alone, so the first depth drafts
  exactly what the single-key reading drafts; deeper depths differ.
- Two-token keys make W_Q and W_K matter (unlike the single key, whose softmax weight
  is exactly 1): replacing W_Q changes the draft.
- For every key set, speculative output equals greedy autoregressive output.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import CloverOracle, attention_decoder, rc_embed
from oracle.model import Precision, rmsnorm


def _make(ad_keys, seed=0, **kw):
    cfg = synth.tiny_test_config(ad_keys=ad_keys, **kw)
    w = synth.make_weights(cfg, seed=seed, perturb=True)
    return cfg, w, CloverOracle(cfg, w)


def test_multi_key_decoder_matches_library_attention():
    cfg, w, o = _make("path", seed=3)
    H, hd = cfg.n_heads, cfg.head_dim
    rng = np.random.default_rng(1)
    h = rng.standard_normal(cfg.d_model)
    keys = np.stack([rc_embed(o.w["lm_head"], t) for t in (5, 17, 40)])
    prec = Precision("f32")
    got = attention_decoder(h, keys, o.w, H, hd, cfg.rms_eps, prec)
    a = rmsnorm(h, o.w["ad.norm"], cfg.rms_eps)
    q = torch.tensor(o.w["ad.wq"] @ a).reshape(H, 1, hd)
    K = torch.tensor(keys @ o.w["ad.wk"].T).reshape(-1, H, hd).transpose(0, 1)
    V = torch.tensor(keys @ o.w["ad.wv"].T).reshape(-1, H, hd).transpose(0, 1)
    att = torch.nn.functional.scaled_dot_product_attention(q, K, V).reshape(-1).numpy()
    assert np.max(np.abs(got - (h + o.w["ad.wo"] @ att))) < 1e-12


def test_path_keys_first_depth_equals_single_key():
    cfg, w, op = _make("path", seed=4)
    os_ = CloverOracle(cfg.with_(ad_keys="single"), w)
    prompt = synth.make_prompt(cfg, n=10)
    sp, ss = op.prefill(prompt), os_.prefill(prompt)
    cp, cs = op.draft(sp), os_.draft(ss)
    d1 = cp.depth <= 1
    assert np.array_equal(cp.token[d1], cs.token[d1]) and np.array_equal(cp.lp[d1], cs.lp[d1])
    assert np.array_equal(cp.row_logits[0], cs.row_logits[0])
    deeper = [n for n in cp.row_logits if cp.depth[n] >= 1]
    assert any(not np.allclose(cp.row_logits[n], cs.row_logits[n]) for n in deeper)


def test_two_token_keys_make_query_and_key_weights_matter():
    cfg, w, o = _make("two", seed=5)
    prompt = synth.make_prompt(cfg, n=10)
    base = o.draft(o.prefill(prompt))
    w2 = dict(w)
    w2["ad.wq"] = w2["ad.wq"] * 3.0
    o2 = CloverOracle(cfg, w2)
    other = o2.draft(o2.prefill(prompt))
    assert not np.allclose(base.row_logits[0], other.row_logits[0])
    # the single-key reading is blind to the same change (Eq. 1 read literally)
    cs = cfg.with_(ad_keys="single")
    s1, s2 = CloverOracle(cs, w), CloverOracle(cs, w2)
    assert np.array_equal(s1.draft(s1.prefill(prompt)).row_logits[0], s2.draft(s2.prefill(prompt)).row_logits[0])


@pytest.mark.parametrize("ad_keys", ["two", "path"])
@pytest.mark.parametrize("seed", [0, 1])
def test_key_sets_keep_greedy_output(ad_keys, seed):
    cfg, _, o = _make(ad_keys, seed=seed, topk=(3, 2, 2), tree_tokens=12)
    prompt = synth.make_prompt(cfg, seq=seed, n=12)
    spec, _ = o.generate(prompt, 14)
    assert spec == o.base.greedy_generate(prompt, 14)


def test_per_head_decoders_with_equal_weights_draft_like_the_shared_one():
    """Reading A6: one Attention Decoder shared by the heads, or one per head.  Per-head
    decoders whose weights all equal the shared decoder's draft exactly what the shared
    one drafts; giving head 2 its own weights changes depth 2 and leaves depth 1 alone."""
    cfg, w, o = _make("two", seed=6)
    cph = cfg.with_(ad_per_head=True)
    wph = {k: v for k, v in w.items() if not k.startswith("ad.")}
    for j in range(cfg.n_spec_heads):
        for f in ("norm", "wq", "wk", "wv", "wo"):
            wph[f"ad{j}.{f}"] = w[f"ad.{f}"]
    assert sorted(wph) == sorted(n for n, _ in synth.weight_specs(cph))
    prompt = synth.make_prompt(cfg, n=9)
    a = o.draft(o.prefill(prompt))
    oph = CloverOracle(cph, wph)
    b = oph.draft(oph.prefill(prompt))
    for f in ("token", "parent", "lp"):
        assert np.array_equal(getattr(a, f), getattr(b, f))
    wph["ad1.wv"] = wph["ad1.wv"] * 2.0
    oph2 = CloverOracle(cph, wph)
    c = oph2.draft(oph2.prefill(prompt))
    assert np.array_equal(c.row_logits[0], a.row_logits[0])            # depth 1: decoder ad0
    assert not np.allclose(c.row_logits[1], a.row_logits[1])           # depth 2: decoder ad1
