"""Pins for speculative sampling (temperature > 0).

- Philox4x32-10 words are uniform (chi-square over the top and the low byte).
- Gumbel-max over the generator's draws samples softmax(logits / temperature): the
  frequencies of 60000 draws match the softmax (chi-square), and a tiny temperature
  reduces to the argmax.
- Lossless acceptance: with a planted tree holding every vocabulary token below the root,
  the root's draw is always accepted and the second emitted token must be distributed as the target's
  p(t2 | prompt, t1) averaged over t1 ~ p(t1 | prompt) -- computed exactly by full forwards --
  and not as p(t2 | prompt), which a walk that drew the second token at the wrong node
  would give (the same statistic rejects that alternative).
- The speculative output still equals plain decoding when the temperature makes every
  draw the argmax.
"""
import numpy as np
import pytest
import scipy.special
import scipy.stats

import synth
from oracle import CloverOracle
from oracle import sampling


def _chi2_p(counts, probs):
    """p-value of observed counts against probabilities (cells with expectation < 5 merged)."""
    counts, probs = np.asarray(counts, dtype=np.float64), np.asarray(probs, dtype=np.float64)
    n = counts.sum()
    exp = probs * n
    big = exp >= 5
    obs = np.append(counts[big], counts[~big].sum())
    ex = np.append(exp[big], exp[~big].sum())
    if ex[-1] == 0:
        obs, ex = obs[:-1], ex[:-1]
    return scipy.stats.chisquare(obs, ex * obs.sum() / ex.sum()).pvalue


def test_philox_words_are_uniform():
    n = 1 << 17
    x = sampling.philox4x32_10_w0(np.arange(n, dtype=np.uint64), 3, 7, 1, 12345, 0)
    for byte in (x >> np.uint32(24), x & np.uint32(0xFF)):
        counts = np.bincount(byte.astype(np.int64), minlength=256)
        assert _chi2_p(counts, np.full(256, 1 / 256)) > 1e-4
    u = sampling.uniform_from_bits(x)
    assert u.dtype == np.float32 and float(u.min()) > 0.0 and float(u.max()) < 1.0
    # the key and every counter word change the stream
    y = sampling.philox4x32_10_w0(np.arange(n, dtype=np.uint64), 3, 7, 1, 12346, 0)
    z = sampling.philox4x32_10_w0(np.arange(n, dtype=np.uint64), 3, 8, 1, 12345, 0)
    assert np.mean(x == y) < 1e-3 and np.mean(x == z) < 1e-3


def test_uniform_mapping_is_exact_and_open_at_the_extreme_words():
    """U must stay strictly inside (0, 1) for every 32-bit word, so the Gumbel noise is
    finite; the extremes are the words with the top 23 bits all zero or all one, which a
    uniform sample of 2^17 words almost never reaches."""
    words = np.array([0, 0x1FF, 0x200, 0xFFFFFE00, 0xFFFFFF00, 0xFFFFFFFF], dtype=np.uint32)
    u = sampling.uniform_from_bits(words)
    assert u.dtype == np.float32
    assert np.all(u > 0) and np.all(u < 1)
    # exact: U = (m + 1/2) / 2^23 with m = word >> 9, compared in float64
    m = (words >> np.uint32(9)).astype(np.float64)
    assert np.array_equal(u.astype(np.float64), (m + 0.5) / 2.0 ** 23)
    assert float(u[0]) == 2.0 ** -24 and float(u[-1]) == 1.0 - 2.0 ** -24
    with np.errstate(all="raise"):
        g = sampling.gumbel_from_bits(words)
    assert np.all(np.isfinite(g))
    # monotone in the top 23 bits: words 0, 0x200 and 0xFFFFFFFF give rising noise, and
    # the low 9 bits do not matter (0xFFFFFE00 and 0xFFFFFFFF share their top 23 bits)
    assert g[0] < g[2] < g[5] and g[3] == g[5] and g[0] == g[1]


def test_gumbel_max_samples_the_softmax():
    rng = np.random.default_rng(0)
    logits = rng.standard_normal(12).astype(np.float32) * 1.5
    tau, n = 0.7, 60000
    draws = sampling.sample_tokens(np.tile(logits, (n, 1)), tau, 99, 0, np.arange(n), 2, 5)
    counts = np.bincount(draws, minlength=12)
    assert all(int(draws[s]) == sampling.sample_token(logits, tau, 99, 0, s, 2, 5) for s in (0, 1, n - 1))
    probs = scipy.special.softmax(logits.astype(np.float64) / tau)
    assert _chi2_p(counts, probs) > 1e-4
    # a temperature far below the logit gaps leaves the argmax
    for step in range(50):
        assert sampling.sample_token(logits, 1e-5, 7, 0, step, 0, 0) == int(np.argmax(logits))


def test_planted_tree_sampling_is_lossless():
    cfg = synth.tiny_test_config(temperature=0.5, topk=(3, 2, 2), tree_tokens=98)
    w = synth.make_weights(cfg, seed=4, perturb=True)
    o = CloverOracle(cfg, w)
    V = cfg.vocab
    prompt = synth.make_prompt(cfg, n=6)
    st0 = o.prefill(prompt)
    # every token below the root: the root's draw is always a child, whose own draw is the bonus
    tokens = [st0.t0] + list(range(V))
    parents = [-1] + [0] * V
    base = o.base
    pre = prompt + [st0.t0]
    p1 = scipy.special.softmax(base.forward_full(pre)[-1] / cfg.temperature)
    p2_given = np.stack([scipy.special.softmax(base.forward_full(pre + [t])[-1] / cfg.temperature)
                         for t in range(V)])
    p2 = p1 @ p2_given
    p2_wrong = p1  # the second token drawn at the root again: p(t2 | prompt, t0)
    n = 3000
    first, second = np.zeros(V), np.zeros(V)
    for seed in range(n):
        o.cfg = cfg.with_(sample_seed=seed)
        st = _copy_state(st0)
        emitted, acc, _ = o.step_tree(st, o.planted_tree(st, tokens, parents))
        assert len(acc) == 2 and len(emitted) == 2  # the root's draw is always a child
        first[emitted[0]] += 1
        second[emitted[1]] += 1
    assert _chi2_p(first, p1) > 1e-4
    assert _chi2_p(second, p2) > 1e-4
    assert _chi2_p(second, p2_wrong) < 1e-6


def _copy_state(st):
    import copy
    return copy.deepcopy(st)


def test_cold_sampling_equals_greedy_decoding():
    cfg = synth.tiny_test_config(temperature=1e-6, topk=(3, 2, 2), tree_tokens=12, sample_seed=5)
    w = synth.make_weights(cfg, seed=2, perturb=True)
    o = CloverOracle(cfg, w)
    prompt = synth.make_prompt(cfg, n=10)
    spec, _ = o.generate(prompt, 12)
    assert spec == o.base.greedy_generate(prompt, 12)
