"""Invariant pins for the oracle's speculate-and-verify step."""
import numpy as np
import pytest

import synth
import oracle
from oracle import CloverOracle, attention_decoder, rc_embed
from oracle.model import Precision


def _make(seed=0, **kw):
    cfg = synth.tiny_test_config(**kw)
    w = synth.make_weights(cfg, seed=seed, perturb=True)
    return cfg, CloverOracle(cfg, w)


@pytest.mark.parametrize("seed,kv", [(0, 2), (1, 1)])
def test_tree_verify_equals_sequential_decode(seed, kv):
    """Sec. 2.2: tree-masked verification scores every node as if its root path
    were decoded sequentially."""
    cfg, o = _make(seed, n_kv_heads=kv)
    st = o.prefill(synth.make_prompt(cfg, n=10))
    cands = o.draft(st)
    tree = oracle.build_tree(cands.depth, cands.token, cands.parent, cands.lp, 25, st.L)
    ver = o.verify(st, tree)
    for i in range(len(tree.tokens)):
        path = []
        j = i
        while j >= 0:
            path.append(int(tree.tokens[j])); j = tree.parent[j]
        seq = st.tokens + path[::-1]
        ref = o.base.forward_full(seq)[-1]
        assert np.max(np.abs(ver.logits[i] - ref)) < 1e-10


@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_speculative_equals_greedy_autoregressive(seed):
    cfg, o = _make(seed, topk=(3, 2, 2), tree_tokens=12)
    prompt = synth.make_prompt(cfg, seq=seed, n=12)
    spec, _ = o.generate(prompt, 14)
    assert spec == o.base.greedy_generate(prompt, 14)


def test_planted_trees_accept_every_length():
    """Plant the greedy continuation at chosen depths: acceptance length 1..H+1."""
    cfg, o = _make(4)
    prompt = synth.make_prompt(cfg, n=12)
    ar = o.base.greedy_generate(prompt, 12)
    H = cfg.n_spec_heads
    for A in range(1, H + 2):
        st = o.prefill(prompt)
        assert st.t0 == ar[0]
        # root, then a decoy branch, then the true chain truncated after A-1 correct tokens
        toks = [st.t0, (ar[1] + 1) % cfg.vocab]
        par = [-1, 0]
        prev = 0
        for d in range(1, H + 1):
            t = ar[d] if d < A else (ar[d] + 3) % cfg.vocab
            toks.append(t); par.append(prev); prev = len(toks) - 1
        tree = o.planted_tree(st, toks, par)
        emitted, acc, _ = o.step_tree(st, tree)
        assert len(acc) == A
        assert emitted == ar[1:A + 1]
        # the state continues exactly like greedy decoding
        spec = [st.t0]
        while len(spec) < 6:
            e, _ = o.step(st)
            spec.extend(e)
        assert spec[:6] == ar[A:A + 6]


def test_commit_kv_equals_autoregressive_prefill():
    """After speculative steps the committed KV equals a prefill of the same tokens."""
    cfg, o = _make(5)
    st = o.prefill(synth.make_prompt(cfg, n=10))
    for _ in range(4):
        o.step(st)
    ref = o.prefill(st.tokens)
    assert ref.t0 == st.t0
    for (k, v), (rk, rv) in zip(st.kv, ref.kv):
        assert k.shape == rk.shape and np.max(np.abs(k - rk)) < 1e-10 and np.max(np.abs(v - rv)) < 1e-10
    assert np.max(np.abs(st.ab_kv[0] - ref.ab_kv[0])) < 1e-10
    assert np.max(np.abs(st.h0 - ref.h0)) < 1e-10


def test_ab_over_tree_then_compaction_equals_commit_time_ab():
    """Running the Augmenting Block over the whole tree (tree mask) and keeping the
    accepted rows gives what running it over the accepted rows does."""
    cfg, o = _make(6)
    prompt = synth.make_prompt(cfg, n=10)
    ar = o.base.greedy_generate(prompt, 5)
    st = o.prefill(prompt)
    tree = o.planted_tree(st, [st.t0, 1, ar[1], 2, ar[2], ar[3]], [-1, 0, 0, 2, 2, 4])
    ver = o.verify(st, tree)
    acc, bonus = oracle.accept(tree.tokens, tree.parent, ver.target)
    assert acc == [0, 2, 4, 5]
    h_tree, k_tree, _ = o.ab_forward(ver.x_last, tree.pos, st.ab_kv, tree.mask)
    L0 = st.L
    o.commit(st, tree, ver, acc, bonus)
    assert np.max(np.abs(h_tree[acc[-1]] - st.h0)) < 1e-10
    assert np.max(np.abs(k_tree[acc] - st.ab_kv[0][L0:])) < 1e-10


def test_attention_decoder_single_key_closed_form():
    """Eq. 1-2 with one key: the softmax weight is exactly 1, so h_i = h + W_O W_V e and
    neither W_Q nor W_K changes the result."""
    cfg, o = _make(7)
    rng = np.random.default_rng(0)
    h = rng.standard_normal(cfg.d_model)
    e = rc_embed(o.w["lm_head"], 17)
    prec = Precision("f32")
    out = attention_decoder(h, e, o.w, cfg.n_heads, cfg.head_dim, cfg.rms_eps, prec)
    assert np.allclose(out, h + o.w["ad.wo"] @ (o.w["ad.wv"] @ e), atol=1e-14)
    w2 = dict(o.w)
    w2["ad.wq"] = rng.standard_normal(w2["ad.wq"].shape)
    w2["ad.wk"] = rng.standard_normal(w2["ad.wk"].shape)
    assert np.array_equal(attention_decoder(h, e, w2, cfg.n_heads, cfg.head_dim, cfg.rms_eps, prec), out)
    # with two keys the weights do matter (the path variant is not degenerate)
    two = np.stack([e, rc_embed(o.w["lm_head"], 3)])
    a = attention_decoder(h, two, o.w, cfg.n_heads, cfg.head_dim, cfg.rms_eps, prec)
    b = attention_decoder(h, two, w2, cfg.n_heads, cfg.head_dim, cfg.rms_eps, prec)
    assert np.max(np.abs(a - b)) > 1e-6


def test_rc_embedding_is_unit_row():
    cfg, o = _make(8)
    for t in (0, 5, cfg.vocab - 1):
        e = rc_embed(o.w["lm_head"], t)
        assert abs(np.linalg.norm(e) - 1) < 1e-14
        assert np.allclose(e * np.linalg.norm(o.w["lm_head"][t]), o.w["lm_head"][t], atol=1e-15)


def test_draft_structure():
    cfg, o = _make(9, topk=(4, 3, 2), tree_tokens=41)
    st = o.prefill(synth.make_prompt(cfg, n=10))
    c = o.draft(st)
    assert len(c.depth) == 41
    assert np.all(c.lp[1:] <= 0)
    for i in range(1, 41):
        assert c.lp[i] <= c.lp[c.parent[i]]          # cumulative log-prob never rises
        assert c.depth[i] == c.depth[c.parent[i]] + 1
    # children of one parent are the head's top-k in order of logit
    for n, logits in c.row_logits.items():
        kids = [i for i in range(41) if c.parent[i] == n]
        assert list(c.token[kids]) == list(oracle.topk_ids(logits, len(kids)))
        assert np.all(np.diff(logits[c.token[kids]]) <= 0)
    # depth-j rows use head j-1 on the AD state; siblings share the parent's AD state
    assert set(c.row_logits) == {i for i in range(41) if c.depth[i] < 3}


def test_bf16_precision_mode_runs_and_matches_f32_loosely():
    cfg = synth.tiny_test_config(dtype="bf16")
    w = synth.make_weights(cfg, seed=1, perturb=True)
    ob = CloverOracle(cfg, w)
    of = CloverOracle(cfg.with_(dtype="f32"), w)
    toks = synth.make_prompt(cfg, n=10)
    lb, lf = ob.base.forward_full(toks), of.base.forward_full(toks)
    d = np.max(np.abs(lb - lf))
    assert 0 < d < 5e-2


def test_tiny_workload_sixteen_steps_equal_greedy():
    """The 2-layer, d=256 workload: 16 speculative steps reproduce greedy decoding."""
    cfg = synth.get_config("tiny_fp32")
    o = CloverOracle(cfg, synth.make_weights(cfg))
    prompt = synth.make_prompt(cfg)
    st = o.prefill(prompt)
    for _ in range(16):
        o.step(st)
    n_new = st.L - len(prompt) + 1
    assert st.tokens[len(prompt):] + [st.t0] == o.base.greedy_generate(prompt, n_new)


@pytest.mark.parametrize("draft", ["clover", "medusa"])
def test_identity_heads_draft_the_targets_next_token_logits(draft):
    """Sec. 3.3-3.4: the heads share the target's final norm and LM head and read the
    state of the last committed token.  With no Augmenting Block, a zero decoder output
    projection (the decoder then adds exactly zero) and head MLPs that add nothing
    (W1 = 0, b1 = -200: SiLU(-200) is about -3e-85, below half an ulp of any state entry),
    every node's head logits must be the target's own next-token logits after the prompt,
    as a plain causal forward of the prompt gives them.  So every node of depth j-1 gets
    the target's top-k_j as children, with the target's log-probabilities added in fp32,
    and the root is the target's greedy choice."""
    import torch
    cfg = synth.tiny_test_config(draft=draft, ab="none", topk=(3, 2, 2), tree_tokens=12)
    w = synth.make_weights(cfg, seed=9, perturb=True)
    if draft == "clover":
        w["ad.wo"] = w["ad.wo"] * 0
    for j in range(cfg.n_spec_heads):
        w[f"head{j}.w1"] = w[f"head{j}.w1"] * 0
        w[f"head{j}.b1"] = torch.full_like(w[f"head{j}.b1"], -200.0)
    o = oracle.make_oracle(cfg, w)
    prompt = synth.make_prompt(cfg, n=13)
    st = o.prefill(prompt)
    ref = o.base.forward_full(prompt)[-1]
    assert st.t0 == int(np.argmax(ref))
    logp = (ref - oracle.logsumexp(ref)).astype(np.float32)
    c = o.draft(st)
    if draft == "medusa":
        for lg in c.head_logits:
            assert np.max(np.abs(lg - ref)) <= 1e-12
    else:
        assert len(c.row_logits) > 0
        for lg in c.row_logits.values():
            assert np.max(np.abs(lg - ref)) <= 1e-12
    idx = 1
    level = [0]
    for j, k in enumerate(cfg.topk, start=1):
        want = np.lexsort((np.arange(len(ref)), -ref))[:k]
        nxt = []
        for n in level:
            for t in want:
                assert c.depth[idx] == j and c.parent[idx] == n and c.token[idx] == t
                assert c.lp[idx] == np.float32(np.float32(c.lp[n]) + logp[t])
                nxt.append(idx)
                idx += 1
        level = nxt
    assert idx == len(c.token)


def _rms(x, g, eps):
    return x / np.sqrt(np.mean(x * x) + eps) * g


def path_sum_pin(alphas=(0.7, -1.3, 2.1), seed=11):
    """Closed form of the Clover draft (Sec. 3.1 Regressive Connection; Sec. 3.2 Eq. 1-2
    and the recursion of h_i; Sec. 3.4 shared LM head).  With the single-key decoder the
    softmax weight is exactly 1, so each depth adds W_O W_V e(token) to the state it
    receives, and the state passed on is the decoder's output.  Without an Augmenting
    Block, h_0 is the target's residual at the last prompt row.  So the decoder output at
    node n is

        s(n) = h_0 + sum over the tokens m on n's root path (root and n included) of
               W_O W_V e(tok_m),  e(t) = W_lm[t] / ||W_lm[t]||,

    and the head of n's depth (head j for nodes of depth j, 0-based) turns it into logits
    W_lm RMSNorm_f(s + SiLU(W1_j s + b1_j)).  With W1_j = alpha_j I the MLP acts element by
    element, so a mix-up of heads, a missing residual or a swapped order of decoder and MLP
    changes the values.  Returns the largest error over every drafted row."""
    import torch
    cfg = synth.tiny_test_config(ab="none", topk=(3, 2, 2), tree_tokens=12)
    w = synth.make_weights(cfg, seed=seed, perturb=True)
    d = cfg.d_model
    for j, a in enumerate(alphas[:cfg.n_spec_heads]):
        w[f"head{j}.w1"] = torch.eye(d) * a
    o = CloverOracle(cfg, w)
    prompt = synth.make_prompt(cfg, n=11)
    st = o.prefill(prompt)
    # h_0 without an Augmenting Block: the residual after the last target layer at the
    # prompt's last row, from the torch float64 forward that pins the base model
    from tests.test_oracle_base import _torch_forward_full
    h0 = _torch_forward_full(cfg, w, prompt, residual=True)[-1]
    W = {k: v.double().numpy() for k, v in w.items()}
    ov = W["ad.wo"] @ W["ad.wv"]
    c = o.draft(st)
    err = float(np.max(np.abs(st.h0 - h0)))
    for n, logits in c.row_logits.items():
        s = h0.copy()
        m = n
        while m >= 0:
            row = W["lm_head"][c.token[m]]
            s = s + ov @ (row / np.linalg.norm(row))
            m = c.parent[m]
        j = int(c.depth[n])
        z = W[f"head{j}.w1"][0, 0] * s + W[f"head{j}.b1"]  # alpha_j as stored (fp32)
        r = s + z / (1 + np.exp(-z))
        want = W["lm_head"] @ _rms(r, W["final_norm"], cfg.rms_eps)
        err = max(err, float(np.max(np.abs(logits - want))))
    assert len(c.row_logits) == 1 + 3 + 6
    return err


def test_clover_draft_equals_path_sum_closed_form():
    assert path_sum_pin() < 1e-10
