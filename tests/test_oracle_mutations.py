"""Planted mistakes in the oracle must be caught by the pins (CPU only).

Each case patches one plausible error into the oracle and checks that the
invariant used as its pin no longer holds.
"""
import numpy as np
import pytest

import synth
import oracle
import oracle.clover as oc
import oracle.model as om
from tests.test_oracle_base import _torch_forward_full


def _base_err(cfg, w):
    toks = synth.make_prompt(cfg, n=16)
    got = om.BaseModel(cfg, {k: v.double().numpy() for k, v in w.items()}).forward_full(toks)
    return np.max(np.abs(got - _torch_forward_full(cfg, w, toks)))


def _tree_err(o, cfg):
    st = o.prefill(synth.make_prompt(cfg, n=10))
    c = o.draft(st)
    tree = oracle.build_tree(c.depth, c.token, c.parent, c.lp, 20, st.L)
    ver = o.verify(st, tree)
    err = 0.0
    for i in range(len(tree.tokens)):
        path, j = [], i
        while j >= 0:
            path.append(int(tree.tokens[j])); j = tree.parent[j]
        err = max(err, np.max(np.abs(ver.logits[i] - o.base.forward_full(st.tokens + path[::-1])[-1])))
    return err


def _rope_wrong_sign(x, pos, theta):
    hd = x.shape[-1]; half = hd // 2
    inv = theta ** (-np.arange(half) * 2.0 / hd)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv[None, :]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c + x2 * s, x2 * c - x1 * s], axis=-1)


def _attention_no_scale(q, k, v, visible):
    return om.attention.__wrapped__(q * np.sqrt(q.shape[-1]), k, v, visible) if hasattr(om.attention, "__wrapped__") \
        else _ATT(q * np.sqrt(q.shape[-1]), k, v, visible)


_ATT = om.attention


def _rmsnorm_no_gain(x, g, eps):
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)


def _mask_parent_only(parent):
    T = len(parent)
    m = np.eye(T, dtype=bool)
    for i in range(T):
        if parent[i] >= 0:
            m[i, parent[i]] = True
            m[i, 0] = True
    return m


@pytest.mark.parametrize("target,mut", [("rope", _rope_wrong_sign), ("attention", _attention_no_scale),
                                        ("rmsnorm", _rmsnorm_no_gain)])
def test_base_pin_catches(monkeypatch, target, mut):
    cfg = synth.tiny_test_config()
    w = synth.make_weights(cfg, seed=3, perturb=True)
    assert _base_err(cfg, w) < 1e-10
    monkeypatch.setattr(om, target, mut)
    assert _base_err(cfg, w) > 1e-6


def test_tree_pin_catches_wrong_mask(monkeypatch):
    cfg = synth.tiny_test_config()
    o = oracle.CloverOracle(cfg, synth.make_weights(cfg, seed=2, perturb=True))
    assert _tree_err(o, cfg) < 1e-10
    monkeypatch.setattr(oc, "tree_mask", _mask_parent_only)
    assert _tree_err(o, cfg) > 1e-6


def test_tree_pin_catches_wrong_positions(monkeypatch):
    cfg = synth.tiny_test_config()
    o = oracle.CloverOracle(cfg, synth.make_weights(cfg, seed=2, perturb=True))
    real = oc.build_tree

    def shifted(*a, **k):
        t = real(*a, **k)
        t.pos = t.pos + 1
        return t
    monkeypatch.setattr(oc, "build_tree", shifted)
    monkeypatch.setattr(oracle, "build_tree", shifted)
    assert _tree_err(o, cfg) > 1e-6


def test_spec_pin_catches_wrong_compaction(monkeypatch):
    """Committing tree slots in their own order instead of the accepted path breaks
    output equality with greedy decoding once a multi-token path is accepted."""
    cfg = synth.tiny_test_config()
    o = oracle.CloverOracle(cfg, synth.make_weights(cfg, seed=4, perturb=True))
    prompt = synth.make_prompt(cfg, n=12)
    ar = o.base.greedy_generate(prompt, 8)

    def run():
        st = o.prefill(prompt)
        tree = o.planted_tree(st, [st.t0, 0, ar[1], ar[2], ar[3]], [-1, 0, 0, 2, 3])
        out = [st.t0] + o.step_tree(st, tree)[0]
        while len(out) < 8:
            out += o.step(st)[0]
        return out[:8]
    assert run() == ar
    real = o.commit

    def bad_commit(st, tree, ver, acc, bonus):
        return real(st, tree, ver, list(range(len(acc))), bonus)
    monkeypatch.setattr(o, "commit", bad_commit)
    assert run() != ar


def test_acceptance_pin_catches_wrong_index():
    """Comparing a child's token with its own argmax instead of its parent's."""
    from tests.test_oracle_tree import _brute_accept

    def accept_own(tokens, parent, target):
        acc, cur = [0], 0
        while True:
            kids = [c for c in range(len(tokens)) if parent[c] == cur and tokens[c] == target[c]]
            if not kids:
                return acc, int(target[cur])
            acc.append(kids[0]); cur = kids[0]
    tokens, parent, target = [9, 4, 6, 5], [-1, 0, 0, 2], [6, 4, 5, 0]
    assert oracle.accept(tokens, parent, target)[0] == _brute_accept(tokens, parent, target) == [0, 2, 3]
    assert accept_own(tokens, parent, target)[0] != _brute_accept(tokens, parent, target)


def _prefill_state_of_wrong_row(self, prompt, slot=0):
    st = _PREFILL(self, prompt, slot)
    n = len(prompt)
    x, _ = self.base.forward_rows(prompt, np.arange(n), None, np.tril(np.ones((n, n), dtype=bool)))
    st.h0 = x[-2].copy()  # the state of the token before the last committed one
    return st


def _head_logits_without_final_norm(self, j, s):
    r = oc.head_mlp(s, self.w[f"head{j}.w1"], self.w[f"head{j}.b1"], self.prec)
    return self.prec.store(r[None, :])[0] @ self.w["lm_head"].T


_PREFILL = oc.CloverOracle.prefill


@pytest.mark.parametrize("draft", ["clover", "medusa"])
@pytest.mark.parametrize("attr,mut", [("prefill", _prefill_state_of_wrong_row),
                                      ("head_logits", _head_logits_without_final_norm)])
def test_identity_head_pin_catches(monkeypatch, draft, attr, mut):
    from tests.test_oracle_clover import test_identity_heads_draft_the_targets_next_token_logits as pin
    monkeypatch.setattr(oc.CloverOracle, attr, mut)
    with pytest.raises(AssertionError):
        pin(draft)


def _mutated_method(cls, name, old, new):
    """A copy of cls.name with one planted mistake: the source text old replaced by new
    (old must occur exactly once, so the mutation tracks the oracle's text)."""
    import inspect
    import textwrap
    src = textwrap.dedent(inspect.getsource(getattr(cls, name)))
    assert src.count(old) == 1, (name, old)
    ns = dict(vars(oc))
    exec(compile(src.replace(old, new), f"<mutated {name}>", "exec"), ns)
    return ns[name]


# plausible mistakes in the Clover draft composition (Sec. 3.1, 3.2 Eq. 1-2)
_DRAFT_MUTATIONS = {
    # no recursion: every depth's decoder reads h_0 instead of its parent's output
    "no_recursion": ("draft", "state[len(depth) - 1] = s", "state[len(depth) - 1] = st.h0"),
    # the root token's embedding at every depth instead of the node's own token
    "root_token_embedded": ("ad_keys", 'e = rc_embed(self.w["lm_head"], token[n])',
                            'e = rc_embed(self.w["lm_head"], token[0])'),
    # the next depth receives the head MLP's output instead of the decoder's
    "mlp_output_propagated": ("draft", "state[len(depth) - 1] = s",
                              'state[len(depth) - 1] = head_mlp(s, self.w[f"head{j - 1}.w1"], '
                              'self.w[f"head{j - 1}.b1"], self.prec)'),
    # depth j drafted with the next head's MLP
    "wrong_head": ("draft", "logits = self.head_logits(j - 1, s)",
                   "logits = self.head_logits(j % c.n_spec_heads, s)"),
}


@pytest.mark.parametrize("which", sorted(_DRAFT_MUTATIONS))
def test_path_sum_pin_catches(monkeypatch, which):
    from tests.test_oracle_clover import path_sum_pin
    assert path_sum_pin() < 1e-10
    name, old, new = _DRAFT_MUTATIONS[which]
    monkeypatch.setattr(oc.CloverOracle, name, _mutated_method(oc.CloverOracle, name, old, new))
    assert path_sum_pin() > 1e-6


def _head_mlp_no_residual(s, w1, b1, prec):
    return om.silu(prec.store(s) @ w1.T + b1)


def test_path_sum_pin_catches_mlp_without_residual(monkeypatch):
    from tests.test_oracle_clover import path_sum_pin
    monkeypatch.setattr(oc, "head_mlp", _head_mlp_no_residual)
    assert path_sum_pin() > 1e-6
