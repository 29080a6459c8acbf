"""Pins for the oracle's Medusa draft (the paper's baseline speculator).

Each pin holds by the method's definition, not by retyping the oracle:
- greedy speculative output equals greedy autoregressive output (Sec. 1, 2.1);
- the candidate tree is the Cartesian product of the heads' top-k sets (Sec. 1, 2.3):
  brute force over every root path;
- Sec. 4.3: Clover with the Attention Decoder, the Regressive Connection and the
  Augmenting Block removed is Medusa.  With their output projections zeroed the
  Augmenting Block and the Attention Decoder are exactly the identity, so the Clover
  oracle then drafts the very tree the Medusa oracle drafts, step after step.
"""
import itertools

import numpy as np
import pytest
import scipy.special

import oracle
import synth
from oracle import CloverOracle, MedusaOracle, topk_ids


def _medusa(seed=0, **kw):
    cfg = synth.tiny_test_config(draft="medusa", **kw)
    w = synth.make_weights(cfg, seed=seed, perturb=True)
    return cfg, w, MedusaOracle(cfg, w)


def test_medusa_weight_list_has_no_clover_parts():
    cfg = synth.tiny_test_config(draft="medusa")
    names = [n for n, _ in synth.weight_specs(cfg)]
    assert not any(n.startswith(("ab.", "ad.")) for n in names)
    assert [n for n in names if n.startswith("head")] == [f"head{j}.{p}" for j in range(3) for p in ("w1", "b1")]


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_medusa_speculative_equals_greedy_autoregressive(seed):
    cfg, _, o = _medusa(seed, topk=(3, 2, 2), tree_tokens=12)
    prompt = synth.make_prompt(cfg, seq=seed, n=12)
    spec, _ = o.generate(prompt, 14)
    assert spec == o.base.greedy_generate(prompt, 14)


@pytest.mark.parametrize("topk", [(4, 3, 2), (2, 2, 2), (3, 1, 2)])
def test_medusa_tree_is_cartesian_product(topk):
    cfg, _, o = _medusa(3, topk=topk)
    st = o.prefill(synth.make_prompt(cfg, n=10))
    c = o.draft(st)
    H = len(topk)
    assert len(c.token) == 1 + sum(int(np.prod(topk[:j + 1])) for j in range(H))
    kids = [list(topk_ids(c.head_logits[j], topk[j])) for j in range(H)]
    # every root path of depth j spells one element of K_1 x ... x K_j, each exactly once
    for j in range(1, H + 1):
        paths = []
        for n in np.nonzero(c.depth == j)[0]:
            p, toks = int(n), []
            while p > 0:
                toks.append(int(c.token[p])); p = int(c.parent[p])
            paths.append(tuple(toks[::-1]))
        assert sorted(paths) == sorted(itertools.product(*[[int(t) for t in kids[i]] for i in range(j)]))
    # children of one parent are head j's top-k in rank order; lp adds logp_j in fp32
    for n in range(1, len(c.token)):
        j, par = int(c.depth[n]), int(c.parent[n])
        sib = [i for i in range(len(c.token)) if c.parent[i] == par]
        assert [int(c.token[i]) for i in sib] == [int(t) for t in kids[j - 1]]
        logp = c.head_logits[j - 1] - scipy.special.logsumexp(c.head_logits[j - 1])
        want = np.float64(c.lp[par]) + logp[c.token[n]]
        assert abs(float(c.lp[n]) - want) <= 2e-7 * max(1.0, abs(want))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_clover_without_its_three_components_is_medusa(dtype):
    """Sec. 4.3: zero the Augmenting Block's attention and MLP output projections and the
    Attention Decoder's output projection; the Clover oracle's candidate trees, verify
    trees and emitted tokens then equal the Medusa oracle's on the same base and heads."""
    cfg_m = synth.tiny_test_config(draft="medusa", dtype=dtype, topk=(3, 2, 2), tree_tokens=12)
    cfg_c = cfg_m.with_(draft="clover")
    wc = synth.make_weights(cfg_c, seed=5, perturb=True)
    for n in ("ab.wo", "ab.w_down", "ad.wo"):
        wc[n] = wc[n] * 0
    wm = {n: wc[n] for n, _ in synth.weight_specs(cfg_m)}
    oc, om = CloverOracle(cfg_c, wc), MedusaOracle(cfg_m, wm)
    prompt = synth.make_prompt(cfg_m, n=14)
    sc, sm = oc.prefill(prompt), om.prefill(prompt)
    assert sc.t0 == sm.t0 and np.array_equal(sc.h0, sm.h0)
    for _ in range(5):
        ec, dc = oc.step(sc)
        em, dm = om.step(sm)
        for f in ("token", "parent", "depth", "lp"):
            assert np.array_equal(getattr(dc["cands"], f), getattr(dm["cands"], f)), f
        assert np.array_equal(dc["tree"].tokens, dm["tree"].tokens)
        assert ec == em
        assert np.array_equal(sc.h0, sm.h0)


def test_make_oracle_picks_the_speculator():
    cfg, w, _ = _medusa()
    assert isinstance(oracle.make_oracle(cfg, w), MedusaOracle)
    cfg_c = cfg.with_(draft="clover")
    assert isinstance(oracle.make_oracle(cfg_c, synth.make_weights(cfg_c)), CloverOracle)


def _decode(o, prompt, steps=4):
    st = o.prefill(prompt)
    trace = [(st.t0, st.h0.copy())]
    for _ in range(steps):
        em, det = o.step(st)
        trace.append((em, det["cands"].token.copy(), det["cands"].lp.copy(), det["tree"].tokens.copy(),
                      st.h0.copy()))
    return trace


def _same(a, b):
    assert len(a) == len(b)
    for x, y in zip(a, b):
        for u, v in zip(x, y):
            assert np.array_equal(np.asarray(u), np.asarray(v))


@pytest.mark.parametrize("variant,zeroed", [("attn", ("ab.w_down",)), ("mlp", ("ab.wo",)),
                                            ("none", ("ab.wo", "ab.w_down"))])
def test_augmenting_block_variants_are_the_full_block_with_a_half_removed(variant, zeroed):
    """Sec. 4.3 explores the Augmenting Block as a whole layer, its attention half, its MLP
    half, or none.  A half contributes exactly nothing when its output projection is zero,
    so each variant must draft, verify and emit exactly what the full block does with the
    other half's output projection zeroed."""
    cfg_v = synth.tiny_test_config(ab=variant, topk=(3, 2, 2), tree_tokens=12)
    cfg_f = cfg_v.with_(ab="full")
    wf = synth.make_weights(cfg_f, seed=6, perturb=True)
    for n in zeroed:
        wf[n] = wf[n] * 0
    wv = {n: wf[n] for n, _ in synth.weight_specs(cfg_v)}
    prompt = synth.make_prompt(cfg_v, n=13)
    _same(_decode(CloverOracle(cfg_v, wv), prompt), _decode(CloverOracle(cfg_f, wf), prompt))


def test_medusa_heads_on_the_augmenting_block_are_clover_without_ad_and_rc():
    """Sec. 4.3: Clover without the Attention Decoder (and with it the Regressive
    Connection) keeps the Augmenting Block and drafts with parallel heads.  The Clover
    oracle with a zero decoder output projection drafts exactly that Cartesian tree."""
    cfg_m = synth.tiny_test_config(draft="medusa", ab="full", topk=(3, 2, 2), tree_tokens=12)
    cfg_c = cfg_m.with_(draft="clover", ab="default")
    wc = synth.make_weights(cfg_c, seed=7, perturb=True)
    wc["ad.wo"] = wc["ad.wo"] * 0
    wm = {n: wc[n] for n, _ in synth.weight_specs(cfg_m)}
    prompt = synth.make_prompt(cfg_m, n=11)
    _same(_decode(MedusaOracle(cfg_m, wm), prompt), _decode(CloverOracle(cfg_c, wc), prompt))


def _per_head_cfg(**kw):
    return synth.tiny_test_config(draft="medusa", medusa_lm="per_head", topk=(3, 2, 2), tree_tokens=12, **kw)


def test_per_head_lm_heads_equal_to_the_target_give_the_shared_draft():
    """Sec. 3.4: the original Medusa gives every head its own LM head, Clover shares the
    target's.  With each head's LM head set to the target's the two readings draft the same
    candidates, log-probabilities and logits."""
    cfg = _per_head_cfg()
    w = synth.make_weights(cfg, seed=5, perturb=True)
    for j in range(cfg.n_spec_heads):
        w[f"head{j}.lm"] = w["lm_head"].clone()
    shared = cfg.with_(medusa_lm="shared")
    ws = {k: v for k, v in w.items() if not k.endswith(".lm")}
    a, b = oracle.MedusaOracle(cfg, w), oracle.MedusaOracle(shared, ws)
    prompt = synth.make_prompt(cfg, n=11)
    ca, cb = a.draft(a.prefill(prompt)), b.draft(b.prefill(prompt))
    assert np.array_equal(ca.token, cb.token) and np.array_equal(ca.lp, cb.lp)
    for la, lb in zip(ca.head_logits, cb.head_logits):
        assert np.array_equal(la, lb)


def test_each_head_reads_its_own_lm_head():
    """Head j's LM head scaled by c_j scales head j's logits by c_j exactly (every head
    reads the state and the final norm the same way), and no other head's."""
    cfg = _per_head_cfg()
    w = synth.make_weights(cfg, seed=6, perturb=True)
    scales = (1.0, 2.0, 4.0)
    for j in range(cfg.n_spec_heads):
        w[f"head{j}.lm"] = w["lm_head"] * scales[j]
    o = oracle.MedusaOracle(cfg, w)
    c = o.draft(o.prefill(synth.make_prompt(cfg, n=11)))
    base = oracle.MedusaOracle(cfg.with_(medusa_lm="shared"), {k: v for k, v in w.items() if not k.endswith(".lm")})
    cb = base.draft(base.prefill(synth.make_prompt(cfg, n=11)))
    for j in range(cfg.n_spec_heads):
        assert np.array_equal(c.head_logits[j], scales[j] * cb.head_logits[j]), j


@pytest.mark.parametrize("seed", [0, 1])
def test_per_head_lm_heads_speculative_equals_greedy(seed):
    cfg = _per_head_cfg()
    o = oracle.MedusaOracle(cfg, synth.make_weights(cfg, seed=seed, perturb=True))
    prompt = synth.make_prompt(cfg, seq=seed, n=12)
    spec, _ = o.generate(prompt, 14)
    assert spec == o.base.greedy_generate(prompt, 14)
