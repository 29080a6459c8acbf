"""Pins for tree construction, the tree mask and greedy acceptance (pure host logic)."""
import itertools

import numpy as np
import pytest

import synth
from oracle import accept, build_tree, tree_mask


def _full_expansion(topk, rng):
    """A candidate list in creation order from random per-row log-probabilities."""
    depth, token, parent, lp = [0], [5], [-1], [np.float32(0)]
    for j, k in enumerate(topk, start=1):
        for n in [i for i in range(len(depth)) if depth[i] == j - 1]:
            logp = np.sort(np.log(rng.dirichlet(np.ones(k + 3))))[::-1][:k].astype(np.float32)
            toks = rng.choice(1000, size=k, replace=False)
            for t, l in zip(toks, logp):
                depth.append(j); token.append(int(t)); parent.append(n)
                lp.append(np.float32(lp[n] + l))
    return np.array(depth), np.array(token), np.array(parent), np.array(lp, dtype=np.float32)


@pytest.mark.parametrize("topk,count", [((4, 3, 2), 40), ((8, 4, 2), 104), ((8, 4, 2, 2), 232),
                                        ((4, 2, 2), 28), ((16, 4, 2), 208)])
def test_node_counts(topk, count):
    d, _, _, _ = _full_expansion(topk, np.random.default_rng(0))
    assert len(d) - 1 == count
    assert [int(np.sum(d == j)) for j in range(len(topk))] == list(np.cumprod((1,) + topk[:-1]))
    cfg = synth.CONFIGS["tiny_fp32"].with_(topk=topk)
    assert cfg.n_candidates() == count


def test_mask_is_ancestor_matrix():
    parent = [-1, 0, 0, 1, 1, 2, 3, 6]
    m = tree_mask(parent)
    for i in range(len(parent)):
        anc = set()
        j = i
        while j >= 0:
            anc.add(j); j = parent[j]
        assert set(np.nonzero(m[i])[0]) == anc
    assert np.array_equal(m, np.tril(m))          # parents precede children
    # a chain is the causal lower triangle; a single root is one AR step
    assert np.array_equal(tree_mask([-1, 0, 1, 2, 3]), np.tril(np.ones((5, 5), dtype=bool)))
    assert np.array_equal(tree_mask([-1]), np.ones((1, 1), dtype=bool))


@pytest.mark.parametrize("topk,T", [((4, 3, 2), 41), ((4, 3, 2), 20), ((8, 4, 2), 64),
                                    ((8, 4, 2, 2), 64), ((4, 2, 2), 16), ((16, 4, 2), 128)])
def test_truncation_brute_force(topk, T):
    rng = np.random.default_rng(len(topk) * 100 + T)
    d, tok, par, lp = _full_expansion(topk, rng)
    tree = build_tree(d, tok, par, lp, T, L=37)
    # brute force over all root paths: rank every non-root node by its path score
    keys = []
    for i in range(1, len(d)):
        path = []
        j = i
        while j > 0:
            path.append(j); j = par[j]
        keys.append((-float(lp[i]), len(path), i))
    kept = sorted(i for _, _, i in sorted(keys)[: T - 1])
    assert list(tree.src) == [0] + kept
    # ancestor-closed, BFS ordered, positions L + depth, mask from parents
    assert all(tree.parent[i] < i for i in range(1, T))
    assert np.all(np.diff(tree.depth) >= 0)
    assert np.array_equal(tree.pos, 37 + tree.depth)
    for i in range(1, T):
        assert tree.tokens[i] == tok[tree.src[i]]
        assert tree.src[tree.parent[i]] == par[tree.src[i]]
    assert np.array_equal(tree.mask, tree_mask(tree.parent))


def test_truncation_ties_prefer_shallow_then_early():
    # all candidates with equal score: the first T-1 in creation order are kept
    d, tok, par, lp = _full_expansion((3, 2), np.random.default_rng(5))
    lp = np.zeros_like(lp)
    tree = build_tree(d, tok, par, lp, 6, 0)
    assert list(tree.src) == [0, 1, 2, 3, 4, 5]


def _brute_accept(tokens, parent, target):
    best = [0]
    for i in range(len(tokens)):
        path = []
        j = i
        while j >= 0:
            path.append(j); j = parent[j]
        path = path[::-1]
        if all(tokens[path[a + 1]] == target[path[a]] for a in range(len(path) - 1)):
            if len(path) > len(best):
                best = path
    return best


def test_acceptance_brute_force():
    rng = np.random.default_rng(6)
    for trial in range(300):
        T = int(rng.integers(1, 30))
        parent = [-1] + [int(rng.integers(0, i)) for i in range(1, T)]
        # siblings carry distinct tokens, as top-k children do
        tokens = [0] * T
        for p in range(T):
            kids = [c for c in range(T) if parent[c] == p]
            for c, t in zip(kids, rng.choice(40, size=len(kids), replace=False)):
                tokens[c] = int(t)
        # targets hit a child's token often, so deep paths are exercised
        target = []
        for i in range(T):
            kids = [c for c in range(T) if parent[c] == i]
            hit = kids and rng.random() < 0.7
            target.append(tokens[int(rng.choice(kids))] if hit else int(rng.integers(0, 40)))
        acc, bonus = accept(tokens, parent, target)
        assert acc == _brute_accept(tokens, parent, target)
        assert bonus == target[acc[-1]]


def test_acceptance_duplicate_siblings_lowest_index():
    tokens = [9, 4, 4, 4]
    parent = [-1, 0, 0, 2]
    acc, bonus = accept(tokens, parent, [4, 7, 4, 1])
    assert acc == [0, 1] and bonus == 7
