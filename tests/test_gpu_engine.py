"""End-to-end parity of the C-ABI step against the oracle on seeded workloads."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.gpu_util import need_gpu, note

pytestmark = pytest.mark.gpu


def _engine(P, cfg, w, **kw):
    """An engine whose verify LM head also stores its logits (the parity checks read them)."""
    kw.setdefault("flags", P.FLAG_KEEP_LOGITS)
    return P.CloverEngine(cfg, {k: v.cuda() for k, v in w.items()}, **kw)


def _tiny(**kw):
    cfg = synth.get_config("tiny_fp32").with_(**kw)
    w = synth.make_weights(cfg, seed=0, perturb=True)
    return cfg, w


def test_tiny_fp32_sixteen_steps_match_oracle_and_greedy():
    P = need_gpu()
    note("engine tiny_fp32 16 steps")
    cfg, w = _tiny()
    eng = _engine(P, cfg, w)
    o = oracle.CloverOracle(cfg, w)
    prompt = synth.make_prompt(cfg)
    t0 = eng.prefill(0, prompt)
    st = o.prefill(prompt)
    assert t0 == st.t0
    h0 = eng.debug("h0", np.float32, (1, cfg.d_model))[0]
    assert np.max(np.abs(h0 - st.h0)) < 1e-4
    out = [t0]
    for step in range(16):
        ours = eng.step([0])[0]
        ref, det = o.step(st)
        if step < 3:
            cands = det["cands"]
            T = cfg.tree_tokens
            assert np.array_equal(eng.debug("cand_token", np.int32, (1, len(cands.token)))[0], cands.token)
            assert np.array_equal(eng.debug("tree_token", np.int32, (1, T))[0], det["tree"].tokens)
            assert np.array_equal(eng.debug("tree_parent", np.int32, (1, T))[0], det["tree"].parent)
            F = 1
            base = 0
            for j in range(1, cfg.n_spec_heads + 1):
                dl = eng.debug(f"draft_logits{j}", np.float32, (F, cfg.vocab))
                for f in range(F):
                    assert np.max(np.abs(dl[f] - cands.row_logits[base + f])) < 1e-4
                base += F
                F *= cfg.topk[j - 1]
            vl = eng.debug("verify_logits", np.float32, (T, cfg.vocab))
            assert np.max(np.abs(vl - det["ver"].logits)) < 1e-4
            assert np.array_equal(eng.debug("target", np.int32, (T,)), det["ver"].target)
        assert ours == ref, (step, ours, ref)
        out += ours
    assert eng.seq_len(0) == st.L
    assert out[: len(out)] == o.base.greedy_generate(prompt, len(out))
    # committed KV (compaction, rotary positions) equals the oracle's cache
    for layer in (0, cfg.n_layers - 1, cfg.n_layers):
        for pos in (0, 127, 128, st.L - 1):
            kv = st.kv[layer] if layer < cfg.n_layers else st.ab_kv
            for which in (0, 1):
                got = eng.debug_kv(0, layer, pos, bool(which))
                assert np.max(np.abs(got - kv[which][pos].reshape(-1))) < 1e-4, (layer, pos, which)


@pytest.mark.parametrize("ab_commit", [False, True])
def test_planted_trees_accept_every_length(ab_commit):
    """Planted trees force every acceptance length; greedy decoding continues exactly.  With
    CLOVER_FLAG_AB_COMMIT the Augmenting Block runs over the accepted rows at commit instead
    of over the tree: the next draft's state h_0 must still be the oracle's (Sec. 3.3)."""
    P = need_gpu()
    note(f"engine planted trees, ab_commit={ab_commit}")
    cfg, w = _tiny()
    o = oracle.CloverOracle(cfg, w)
    prompt = synth.make_prompt(cfg, seq=3)
    ar = o.base.greedy_generate(prompt, 12)
    H = cfg.n_spec_heads
    eng = _engine(P, cfg, w, flags=P.FLAG_KEEP_LOGITS | (P.FLAG_AB_COMMIT if ab_commit else 0))
    for A in range(1, H + 2):
        t0 = eng.prefill(0, prompt)
        assert t0 == ar[0]
        st = o.prefill(prompt)
        toks, par, prev = [t0, (ar[1] + 1) % cfg.vocab], [-1, 0], 0
        for d in range(1, H + 1):
            toks.append(ar[d] if d < A else (ar[d] + 3) % cfg.vocab)
            par.append(prev)
            prev = len(toks) - 1
        got = eng.verify_tree(0, toks, par)
        assert got == ar[1:A + 1], (A, got)
        assert eng.debug("acc_len", np.int32, (1,))[0] == A
        o.step_tree(st, o.planted_tree(st, toks, par))
        h0 = eng.debug("h0", np.float32, (1, cfg.d_model))[0]
        assert np.max(np.abs(h0 - st.h0)) < 1e-4, A
        for layer in (0, cfg.n_layers):  # a target layer and the Augmenting Block
            for j in range(A):
                for which in (0, 1):
                    kv = st.kv[layer] if layer < cfg.n_layers else st.ab_kv
                    ref = kv[which][st.L - A + j].reshape(-1)
                    assert np.max(np.abs(eng.debug_kv(0, layer, st.L - A + j, bool(which)) - ref)) < 1e-4
        # then continue with drafted steps: still greedy
        out = []
        while len(out) < 6:
            out += eng.step([0])[0]
        assert out[:6] == ar[A + 1:A + 7]
        eng.release(0)


def test_batch_of_three_sequences():
    P = need_gpu()
    note("engine batch 3")
    cfg, w = _tiny(batch=3)
    eng = _engine(P, cfg, w)
    o = oracle.CloverOracle(cfg, w)
    lens = [128, 77, 200]
    states, outs = [], []
    for s in range(3):
        prompt = synth.make_prompt(cfg, seq=s, n=lens[s])
        t0 = eng.prefill(s, prompt)
        st = o.prefill(prompt)
        assert t0 == st.t0
        states.append(st)
        outs.append([])
    for step in range(5):
        order = [2, 0, 1] if step % 2 else [0, 1, 2]
        got = eng.step(order)
        for b, s in enumerate(order):
            ref, _ = o.step(states[s])
            assert got[b] == ref, (step, s)
    # a single sequence may step alone afterwards
    ref, _ = o.step(states[1])
    assert eng.step([1])[0] == ref


def test_prefill_longer_than_one_chunk():
    P = need_gpu()
    note("engine long prefill")
    cfg, w = _tiny(max_context=1024)
    eng = _engine(P, cfg, w, prefill_chunk=128)
    o = oracle.CloverOracle(cfg, w)
    prompt = synth.make_prompt(cfg, n=300)
    assert eng.prefill(0, prompt) == o.prefill(prompt).t0


def test_error_paths_leave_state_unchanged():
    P = need_gpu()
    note("engine errors")
    cfg, w = _tiny(batch=2)
    eng = _engine(P, cfg, w)
    prompt = synth.make_prompt(cfg)
    with pytest.raises(P.CloverError) as e:
        eng.step([0])
    assert e.value.status == 3
    t0 = eng.prefill(0, prompt)
    with pytest.raises(P.CloverError) as e:
        eng.prefill(0, prompt)
    assert e.value.status == 3
    with pytest.raises(P.CloverError) as e:
        eng.prefill(1, [cfg.vocab])
    assert e.value.status == 1
    with pytest.raises(P.CloverError) as e:
        eng.prefill(1, [1] * (cfg.max_context))
    assert e.value.status == 2
    with pytest.raises(P.CloverError) as e:
        eng.verify_tree(0, [t0, 1, 2], [-1, 2, 0])
    assert e.value.status == 4
    with pytest.raises(P.CloverError) as e:
        eng.step([0, 0])
    assert e.value.status == 1
    assert eng.seq_len(0) == len(prompt)
    o = oracle.CloverOracle(cfg, w)
    st = o.prefill(prompt)
    assert eng.step([0])[0] == o.step(st)[0]


def test_two_engines_are_bit_identical():
    P = need_gpu()
    note("engine determinism")
    cfg, w = _tiny()
    prompt = synth.make_prompt(cfg, seq=5)
    runs = []
    for _ in range(2):
        eng = _engine(P, cfg, w)
        eng.prefill(0, prompt)
        toks = [eng.step([0])[0] for _ in range(4)]
        runs.append((toks, eng.debug("verify_logits", np.float32, (cfg.tree_tokens, cfg.vocab)),
                     eng.debug("draft_logits3", np.float32, (12, cfg.vocab))))
        eng.close()
    assert runs[0][0] == runs[1][0]
    assert np.array_equal(runs[0][1], runs[1][1])
    assert np.array_equal(runs[0][2], runs[1][2])


def _bf16_small():
    return synth.CloverConfig(name="small_bf16", n_layers=3, d_model=512, n_heads=4, n_kv_heads=2,
                              head_dim=128, ffn_dim=1024, vocab=4096, dtype="bf16", topk=(4, 2, 2),
                              tree_tokens=20, batch=1, prompt_len=(100, 100), steps=6, max_context=512)


def _margin_k(logits, k):
    """Gap between the k-th and (k+1)-th largest values (the top-k decision's margin)."""
    v = np.sort(logits)[::-1]
    return float(v[k - 1] - v[k]) if k < len(v) else np.inf


def teacher_forced_step(eng, o, states, tol, stats):
    """One step of every sequence 0..B-1 on the GPU, with the oracle teacher-forced onto it.

    Each oracle drafts from its own state; draft logits are compared for every depth whose
    frontier nodes (the candidates of all shallower depths) agree with the GPU's, and where
    they disagree the oracle's own top-k decision there must be a near tie (margin < 2 tol).
    The oracle then verifies the GPU's tree (all T rows compared), checks that its own
    acceptance agrees with the GPU's unless a target is a near tie, and commits the GPU's
    accepted path and bonus, so the next step starts from the same tokens on both sides and
    every step is compared.  stats counts compared rows and near-tie decisions."""
    c = o.cfg
    B, T, V, H = len(states), c.tree_tokens, c.vocab, c.n_spec_heads
    got = eng.step(list(range(B)))
    n_cand = 1 + c.n_candidates()
    gtok = eng.debug("cand_token", np.int32, (eng.c.max_batch, n_cand))
    trees = eng.debug("tree_token", np.int32, (eng.c.max_batch, T))
    parents = eng.debug("tree_parent", np.int32, (eng.c.max_batch, T))
    vl = eng.debug("verify_logits", np.float32, (B * T, V))
    accs = eng.debug("acc", np.int32, (eng.c.max_batch, H + 1))
    alen = eng.debug("acc_len", np.int32, (eng.c.max_batch,))
    medusa = getattr(c, "draft", "clover") == "medusa"
    F = 1
    dl = []
    for j in range(1, H + 1):
        rows = B if medusa else B * F
        dl.append(eng.debug(f"draft_logits{j}", np.float32, (rows, V)))
        F *= c.topk[j - 1]
    for b, st in enumerate(states):
        cands = o.draft(st)
        F, base = 1, 0
        for j in range(1, H + 1):
            if medusa:
                err = float(np.max(np.abs(dl[j - 1][b] - cands.head_logits[j - 1])))
                assert err < tol, (b, j, err)
                stats["draft_rows"] += 1
                continue
            if not np.array_equal(gtok[b, :base + F], cands.token[:base + F]):
                # a near tie in a shallower top-k made different frontier nodes
                assert min(_margin_k(cands.row_logits[n], c.topk[cands.depth[n]])
                           for n in cands.row_logits if cands.depth[n] < j - 1) < 2 * tol, (b, j)
                stats["draft_ties"] += 1
                break
            for f in range(F):
                err = float(np.max(np.abs(dl[j - 1][b * F + f] - cands.row_logits[base + f])))
                assert err < tol, (b, j, f, err)
                stats["draft_rows"] += 1
            base += F
            F *= c.topk[j - 1]
        tree = o.planted_tree(st, trees[b], parents[b])
        ver = o.verify(st, tree)
        err = float(np.max(np.abs(vl[b * T:(b + 1) * T] - ver.logits)))
        assert err < tol, (b, err)
        stats["verify_rows"] += T
        acc_g = [int(a) for a in accs[b, :alen[b]]]
        acc_o, bonus_o = oracle.accept(tree.tokens, tree.parent, ver.target)
        emitted_g = got[b]
        assert emitted_g == [int(tree.tokens[i]) for i in acc_g[1:]] + [emitted_g[-1]]
        if acc_o != acc_g or bonus_o != emitted_g[-1]:
            top2 = np.sort(ver.logits[sorted(set(acc_o) | set(acc_g))], axis=1)[:, -2:]
            assert float(np.min(top2[:, 1] - top2[:, 0])) < 2 * tol, (b, acc_o, acc_g)
            stats["target_ties"] += 1
        o.commit(st, tree, ver, acc_g, emitted_g[-1])
        stats["steps"] += 1
    return got


def test_bf16_small_model_within_tolerance():
    """bf16 storage: draft and verify logits within 2e-2 of the oracle (which rounds at
    the same storage points) at every step; the oracle is teacher-forced onto the GPU's
    trees and accepted paths, and its own discrete decisions must agree wherever they are
    not near ties."""
    P = need_gpu()
    note("engine bf16 small")
    cfg = _bf16_small()
    w = synth.make_weights(cfg, seed=2, perturb=True)
    eng = _engine(P, cfg, w)
    o = oracle.CloverOracle(cfg, w)
    prompt = synth.make_prompt(cfg, n=100)
    t0 = eng.prefill(0, prompt)
    st = o.prefill(prompt)
    assert t0 == st.t0
    stats = dict(steps=0, draft_rows=0, verify_rows=0, draft_ties=0, target_ties=0)
    for _ in range(6):
        teacher_forced_step(eng, o, [st], 2e-2, stats)
    note(f"bf16 small: {stats}")
    assert stats["steps"] == 6 and stats["verify_rows"] == 6 * cfg.tree_tokens
    assert stats["draft_rows"] >= 6 * 5  # at least the root and depth-1 rows of every step


def _kv_close(got, ref, layer=0):
    """Committed bf16 K/V against the oracle's.  Layer 0 sees the same bf16 inputs on both
    sides, so its values differ at most by one bf16 step where the fp32 and fp64 sums round
    apart; deeper layers inherit the residual stream's low-bit differences and may differ
    by up to two bf16 steps (2^-7 relative each, taken at magnitude 1 below 1)."""
    if layer == 0:
        return float(np.max(np.abs(got - ref) / (np.abs(ref) + 0.05))) <= 1.0 / 64
    return bool(np.all(np.abs(got - ref) <= 2.0 ** -6 * np.maximum(np.abs(ref), 1.0)))


def _random_tree(rng, T, H, vocab):
    """Seeded tree of T nodes, depth <= H, parents before children."""
    depth, parents = [0], [-1]
    for i in range(1, T):
        cand = [j for j in range(i) if depth[j] < H]
        p = int(rng.choice(cand))
        parents.append(p)
        depth.append(depth[p] + 1)
    return [int(t) for t in rng.integers(0, vocab, T)], parents


def test_bf16_128_row_verify_and_chunked_prefill():
    """A 128-token planted tree (128 verify rows) and a 300-token prompt (a 256-row prefill
    chunk and a 44-row one) run the register-blocked GEMM with each of its epilogues:
    rotary + paged KV append, SwiGLU, split-K partials and the LM head.  Committed K/V and
    the verify logits stay within the bf16 bounds of the oracle."""
    P = need_gpu()
    note("engine bf16 128-row verify")
    cfg = _bf16_small().with_(topk=(8, 4, 4), tree_tokens=128, max_context=1024)
    w = synth.make_weights(cfg, seed=4, perturb=True)
    eng = _engine(P, cfg, w)
    o = oracle.CloverOracle(cfg, w)
    prompt = synth.make_prompt(cfg, n=300)
    eng.prefill(0, prompt)
    st = o.prefill(prompt)
    for layer in (0, cfg.n_layers - 1):
        for pos in (0, 100, 255, 256, 299):
            for which in (0, 1):
                got = eng.debug_kv(0, layer, pos, bool(which))
                assert _kv_close(got, st.kv[layer][which][pos].reshape(-1), layer), (layer, pos, which)
    rng = np.random.default_rng(11)
    tokens, parents = _random_tree(rng, cfg.tree_tokens, cfg.n_spec_heads, cfg.vocab)
    tokens[0] = st.t0
    tree = o.planted_tree(st, tokens, parents)
    L = st.L
    got = eng.verify_tree(0, tokens, parents)
    ref, acc, ver = o.step_tree(st, tree)
    vl = eng.debug("verify_logits", np.float32, (cfg.tree_tokens, cfg.vocab))
    err = float(np.max(np.abs(vl - ver.logits)))
    note(f"128-row verify logits: max |err| {err:.3e}")
    assert err < 2e-2
    # the LM head's fused argmax equals the argmax of its own logits (lowest index on ties)
    assert np.array_equal(eng.debug("target", np.int32, (cfg.tree_tokens,)), np.argmax(vl, axis=1))
    top2 = np.sort(ver.logits, axis=1)[:, -2:]
    if np.min(top2[:, 1] - top2[:, 0]) >= 4e-2:  # no near tie decides a target
        assert got == ref
    # the committed K/V of the GPU's accepted path are its tree nodes' K/V (the oracle's
    # tree-node values, taken at the GPU's own acceptance)
    acc_g = eng.debug("acc", np.int32, (1, cfg.n_spec_heads + 1))[0][:len(got)]
    for j, node in enumerate(acc_g):
        for which in (0, 1):
            g = eng.debug_kv(0, 0, L + j, bool(which))
            assert _kv_close(g, ver.kv[0][which][node].reshape(-1)), (j, which)


def test_bf16_batch_of_eight_verify_rows():
    """Eight sequences of 20-token trees verify as one 160-row forward (register-blocked
    GEMMs whose rows belong to different sequences and KV blocks); each sequence's draft and
    verify logits match its own oracle within the bf16 tolerance."""
    P = need_gpu()
    note("engine bf16 batch 8")
    cfg = _bf16_small().with_(batch=8)
    w = synth.make_weights(cfg, seed=5, perturb=True)
    eng = _engine(P, cfg, w)
    o = oracle.CloverOracle(cfg, w)
    lens = [60, 41, 90, 77, 33, 128, 50, 99]
    states = []
    for s in range(8):
        prompt = synth.make_prompt(cfg, seq=s, n=lens[s])
        eng.prefill(s, prompt)
        states.append(o.prefill(prompt))
    B, T, V = 8, cfg.tree_tokens, cfg.vocab
    got = eng.step(list(range(B)))
    trees = eng.debug("tree_token", np.int32, (B, T))
    parents = eng.debug("tree_parent", np.int32, (B, T))
    vl = eng.debug("verify_logits", np.float32, (B * T, V))
    assert np.array_equal(eng.debug("target", np.int32, (B * T,)), np.argmax(vl, axis=1))
    d1 = eng.debug("draft_logits1", np.float32, (B, V))
    compared = 0
    for b in range(B):
        ref, det = o.step(states[b])
        # the root's head-1 logits depend only on this sequence's h0 and t0
        assert float(np.max(np.abs(d1[b] - det["cands"].row_logits[0]))) < 2e-2, b
        if not (np.array_equal(trees[b], det["tree"].tokens) and np.array_equal(parents[b], det["tree"].parent)):
            continue  # a near tie in the draft or the truncation separated the trees
        err = float(np.max(np.abs(vl[b * T:(b + 1) * T] - det["ver"].logits)))
        assert err < 2e-2, (b, err)
        compared += 1
        top2 = np.sort(det["ver"].logits, axis=1)[:, -2:]
        if np.min(top2[:, 1] - top2[:, 0]) >= 4e-2:
            assert got[b] == ref, b
    assert compared >= 3
    note(f"batch 8: {compared} sequences compared")


@pytest.mark.parametrize("B,T,topk", [(16, 64, (8, 4, 2)), (16, 128, (16, 4, 2)), (48, 128, (16, 4, 2))])
def test_bf16_large_batches_verify_rows(B, T, topk):
    """Sixteen or forty-eight sequences verify 1024, 2048 or 6144 tree rows in one forward (the
    batch x tree cost surface's largest cells: register-blocked GEMMs at those row counts with
    every epilogue, attention over many paged sequences); each sequence's draft and verify
    logits stay within the bf16 tolerance of its oracle over two teacher-forced steps."""
    P = need_gpu()
    note(f"engine bf16 batch {B}, T={T}")
    cfg = _bf16_small().with_(batch=B, topk=topk, tree_tokens=T, max_context=512)
    w = synth.make_weights(cfg, seed=12, perturb=True)
    eng = _engine(P, cfg, w)
    o = oracle.CloverOracle(cfg, w)
    states = []
    for s in range(B):
        prompt = synth.make_prompt(cfg, seq=s, n=20 + (17 * s) % 300)
        assert eng.prefill(s, prompt) == (st := o.prefill(prompt)).t0
        states.append(st)
    stats = dict(steps=0, draft_rows=0, verify_rows=0, draft_ties=0, target_ties=0)
    for _ in range(2):
        teacher_forced_step(eng, o, states, 2e-2, stats)
    note(f"batch {B}, T={T}: {stats}")
    assert stats["steps"] == 2 * B and stats["verify_rows"] == 2 * B * T
    eng.close()


def ab_flag(P, ab_commit):
    return P.FLAG_AB_COMMIT if ab_commit else 0


@pytest.mark.parametrize("ab_commit", [False, True])
def test_graph_replay_matches_eager_launches(ab_commit):
    """The step's phases replay as HIP graphs captured per batch size; every replay,
    with host work and batch-size changes in between, matches eager launches bit for bit."""
    P = need_gpu()
    note("engine graph vs eager")
    cfg, w = _tiny(batch=2)
    prompts = [synth.make_prompt(cfg, seq=s, n=100 + 30 * s) for s in range(2)]
    g = _engine(P, cfg, w, flags=P.FLAG_KEEP_LOGITS | ab_flag(P, ab_commit))
    e = _engine(P, cfg, w, flags=P.FLAG_EAGER | P.FLAG_KEEP_LOGITS | ab_flag(P, ab_commit))
    for s in range(2):
        assert g.prefill(s, prompts[s]) == e.prefill(s, prompts[s])
    schedule = [[0], [0, 1], [1], [0, 1], [0], [1, 0], [0, 1]]
    for i, seqs in enumerate(schedule):
        if i == 3:
            g.set_flags(P.FLAG_EAGER | P.FLAG_KEEP_LOGITS | ab_flag(P, ab_commit))  # eager in the middle
        if i == 5:
            g.set_flags(P.FLAG_KEEP_LOGITS | ab_flag(P, ab_commit))  # graphs again after
        a, b = g.step(seqs), e.step(seqs)
        assert a == b, (i, seqs, a, b)
        rows = len(seqs) * cfg.tree_tokens
        va = g.debug("verify_logits", np.float32, (rows, cfg.vocab))
        vb = e.debug("verify_logits", np.float32, (rows, cfg.vocab))
        assert np.array_equal(va, vb), i
        assert np.array_equal(g.debug("h0", np.float32, (2, cfg.d_model)), e.debug("h0", np.float32, (2, cfg.d_model)))
        torch.cuda.synchronize()
    assert g.seq_len(0) == e.seq_len(0) and g.seq_len(1) == e.seq_len(1)


def test_medusa_tiny_fp32_sixteen_steps_match_oracle_and_greedy():
    """The Medusa baseline on the same kernels: heads on x_N of the last committed token,
    one LM-head pass for all heads, Cartesian candidate tree.  Head logits within 1e-4 of
    the oracle, candidate and verify trees exact, tokens equal to the oracle's and to
    plain greedy decoding; committed KV equals the oracle's."""
    P = need_gpu()
    note("engine medusa tiny_fp32 16 steps")
    cfg = synth.get_config("tiny_fp32_medusa")
    w = synth.make_weights(cfg, seed=0, perturb=True)
    eng = _engine(P, cfg, w)
    o = oracle.MedusaOracle(cfg, w)
    prompt = synth.make_prompt(cfg)
    t0 = eng.prefill(0, prompt)
    st = o.prefill(prompt)
    assert t0 == st.t0
    assert np.max(np.abs(eng.debug("h0", np.float32, (1, cfg.d_model))[0] - st.h0)) < 1e-4
    out = [t0]
    T = cfg.tree_tokens
    for step in range(16):
        ours = eng.step([0])[0]
        ref, det = o.step(st)
        cands = det["cands"]
        for j in range(1, cfg.n_spec_heads + 1):
            dl = eng.debug(f"draft_logits{j}", np.float32, (1, cfg.vocab))[0]
            assert np.max(np.abs(dl - cands.head_logits[j - 1])) < 1e-4, (step, j)
        n = len(cands.token)
        for f, dt in (("token", np.int32), ("parent", np.int32), ("depth", np.int32)):
            assert np.array_equal(eng.debug(f"cand_{f}", dt, (1, n))[0], getattr(cands, f)), (step, f)
        assert np.array_equal(eng.debug("tree_token", np.int32, (1, T))[0], det["tree"].tokens)
        assert np.array_equal(eng.debug("tree_parent", np.int32, (1, T))[0], det["tree"].parent)
        vl = eng.debug("verify_logits", np.float32, (T, cfg.vocab))
        assert np.max(np.abs(vl - det["ver"].logits)) < 1e-4
        assert ours == ref, (step, ours, ref)
        out += ours
    assert eng.seq_len(0) == st.L
    assert out == o.base.greedy_generate(prompt, len(out))
    for layer in (0, cfg.n_layers - 1):
        for pos in (0, 127, 128, st.L - 1):
            for which in (0, 1):
                got = eng.debug_kv(0, layer, pos, bool(which))
                assert np.max(np.abs(got - st.kv[layer][which][pos].reshape(-1))) < 1e-4, (layer, pos, which)
    with pytest.raises(P.CloverError):
        eng.debug_kv(0, cfg.n_layers, 0, False)  # no Augmenting Block cache in Medusa mode


def test_logits_are_stored_only_with_keep_logits():
    """Without CLOVER_FLAG_KEEP_LOGITS the verify LM head stores only its argmax keys: the
    logits buffer keeps what the last flagged step wrote while the targets move on.  With
    the flag set again (the captured graphs are rebuilt) the logits are fresh and match
    the oracle."""
    P = need_gpu()
    note("engine keep-logits flag")
    cfg, w = _tiny(batch=1)
    eng = _engine(P, cfg, w, flags=0)
    o = oracle.CloverOracle(cfg, w)
    prompt = synth.make_prompt(cfg, n=90)
    st = o.prefill(prompt)
    assert eng.prefill(0, prompt) == st.t0
    T, V = cfg.tree_tokens, cfg.vocab
    eng.set_flags(P.FLAG_KEEP_LOGITS)
    assert eng.step([0])[0] == o.step(st)[0]
    kept = eng.debug("verify_logits", np.float32, (T, V))
    eng.set_flags(0)
    for _ in range(2):
        ref, det = o.step(st)
        assert eng.step([0])[0] == ref
        assert np.array_equal(eng.debug("target", np.int32, (T,)), det["ver"].target)
        assert np.array_equal(eng.debug("verify_logits", np.float32, (T, V)), kept)
    eng.set_flags(P.FLAG_KEEP_LOGITS)
    ref, det = o.step(st)
    assert eng.step([0])[0] == ref
    assert float(np.max(np.abs(eng.debug("verify_logits", np.float32, (T, V)) - det["ver"].logits))) < 1e-4
    eng.close()


def test_medusa_bf16_batch_of_three_within_tolerance():
    """bf16 Medusa over three sequences of different lengths: each sequence's head logits
    and verify logits within 2e-2 of its oracle at every step, with the oracle
    teacher-forced onto the GPU's trees and accepted paths."""
    P = need_gpu()
    note("engine medusa bf16 batch 3")
    cfg = _bf16_small().with_(draft="medusa", batch=3)
    w = synth.make_weights(cfg, seed=8, perturb=True)
    eng = _engine(P, cfg, w)
    o = oracle.MedusaOracle(cfg, w)
    lens = [100, 37, 64]
    states = []
    for s in range(3):
        prompt = synth.make_prompt(cfg, seq=s, n=lens[s])
        assert eng.prefill(s, prompt) == (st := o.prefill(prompt)).t0
        states.append(st)
    stats = dict(steps=0, draft_rows=0, verify_rows=0, draft_ties=0, target_ties=0)
    for _ in range(3):
        teacher_forced_step(eng, o, states, 2e-2, stats)
    note(f"medusa bf16 batch 3: {stats}")
    assert stats["steps"] == 9 and stats["draft_rows"] == 9 * cfg.n_spec_heads
    assert stats["verify_rows"] == 9 * cfg.tree_tokens


@pytest.mark.parametrize("draft,ab,ad_keys,per_head,regressive", [
    ("clover", "attn", "single", False, "attention"), ("clover", "mlp", "single", False, "attention"),
    ("clover", "none", "single", False, "attention"), ("medusa", "full", "single", False, "attention"),
    ("clover", "default", "two", False, "attention"), ("clover", "default", "path", False, "attention"),
    ("clover", "default", "two", True, "attention"), ("clover", "default", "single", False, "mlp"),
    ("clover", "none", "single", False, "mlp")])
def test_speculator_variants_match_oracle(draft, ab, ad_keys, per_head, regressive):
    """The Augmenting Block variants of Sec. 4.3 (attention half, MLP half, none) under the
    Clover draft, the Augmenting Block feeding parallel heads (Clover without Attention
    Decoder and Regressive Connection), the two-token and root-path key sets of the
    Attention Decoder, one decoder per head, and the MLP regressive block of the components
    ablation (with and without the Augmenting Block): tiny fp32, six steps, draft logits of
    every frontier row and verify logits within 1e-4, candidate and verify trees exact,
    tokens equal to the oracle's and to greedy decoding."""
    P = need_gpu()
    note(f"engine variant draft={draft} ab={ab} ad_keys={ad_keys} per_head={per_head} regressive={regressive}")
    cfg = synth.get_config("tiny_fp32").with_(draft=draft, ab=ab, ad_keys=ad_keys, ad_per_head=per_head,
                                              regressive=regressive)
    w = synth.make_weights(cfg, seed=1, perturb=True)
    eng = _engine(P, cfg, w)
    o = oracle.make_oracle(cfg, w)
    prompt = synth.make_prompt(cfg, seq=2)
    assert eng.prefill(0, prompt) == (st := o.prefill(prompt)).t0
    assert np.max(np.abs(eng.debug("h0", np.float32, (1, cfg.d_model))[0] - st.h0)) < 1e-4
    T, out = cfg.tree_tokens, [st.t0]
    for step in range(6):
        ours = eng.step([0])[0]
        ref, det = o.step(st)
        n = len(det["cands"].token)
        if draft == "clover":
            F, base = 1, 0
            for j in range(1, cfg.n_spec_heads + 1):
                dl = eng.debug(f"draft_logits{j}", np.float32, (F, cfg.vocab))
                for f in range(F):
                    assert np.max(np.abs(dl[f] - det["cands"].row_logits[base + f])) < 1e-4, (step, j, f)
                base += F
                F *= cfg.topk[j - 1]
        assert np.array_equal(eng.debug("cand_token", np.int32, (1, n))[0], det["cands"].token), step
        assert np.array_equal(eng.debug("tree_token", np.int32, (1, T))[0], det["tree"].tokens), step
        vl = eng.debug("verify_logits", np.float32, (T, cfg.vocab))
        assert np.max(np.abs(vl - det["ver"].logits)) < 1e-4, step
        assert np.max(np.abs(eng.debug("h0", np.float32, (1, cfg.d_model))[0] - st.h0)) < 1e-4, step
        assert ours == ref, (step, ours, ref)
        out += ours
    assert out == o.base.greedy_generate(prompt, len(out))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_medusa_per_head_lm_heads_match_oracle(dtype):
    """The original Medusa's per-head LM heads (Sec. 3.4): one LM-head pass per head, each
    with its own weights.  Head logits and verify logits within the dtype's tolerance over
    four steps, trees exact, tokens equal to the oracle's (fp32) and to greedy decoding."""
    P = need_gpu()
    note(f"engine Medusa per-head LM heads {dtype}")
    cfg = (synth.get_config("tiny_fp32") if dtype == "f32" else _bf16_small()).with_(
        draft="medusa", medusa_lm="per_head", batch=2)
    w = synth.make_weights(cfg, seed=13, perturb=True)
    eng = _engine(P, cfg, w)
    o = oracle.make_oracle(cfg, w)
    tol = 1e-4 if dtype == "f32" else 2e-2
    states = []
    for s in range(2):
        prompt = synth.make_prompt(cfg, seq=s, n=90 + 20 * s)
        assert eng.prefill(s, prompt) == (st := o.prefill(prompt)).t0
        states.append(st)
    stats = dict(steps=0, draft_rows=0, verify_rows=0, draft_ties=0, target_ties=0)
    for _ in range(4):
        teacher_forced_step(eng, o, states, tol, stats)
    note(f"Medusa per-head LM heads {dtype}: {stats}")
    assert stats["steps"] == 8 and stats["draft_rows"] == 8 * cfg.n_spec_heads
    if dtype == "f32":
        assert stats["target_ties"] == 0
    eng.close()


@pytest.mark.parametrize("which", ["tiny_fp32", "small_bf16_t128"])
def test_sampled_targets_match_oracle_sampler(which):
    """Speculative sampling (temperature 0.8): every tree node's target is a Gumbel-max draw
    fused into the LM head's argmax epilogue.  On the GPU's own verify logits the oracle's
    sampler (its own Philox4x32-10 and Gumbel transform) reproduces every target exactly
    wherever the top two perturbed scores are not within 1e-4 of each other; the step counter
    of each slot advances once per step; end to end, tokens equal the oracle's while no draw
    is that close.  Two sequences (slots 0 and 1); the bf16 case verifies 2 x 128 rows on the
    register-blocked kernel."""
    P = need_gpu()
    note(f"engine sampling {which}")
    if which == "tiny_fp32":
        cfg, w = _tiny(batch=2, temperature=0.8, sample_seed=1234)
        tol = 1e-4
    else:
        cfg = _bf16_small().with_(batch=2, topk=(8, 4, 4), tree_tokens=128, max_context=1024,
                                  temperature=0.8, sample_seed=77)
        w = synth.make_weights(cfg, seed=9, perturb=True)
        tol = 2e-2
    from oracle import sampling
    eng = _engine(P, cfg, w)
    o = oracle.CloverOracle(cfg, w)
    T, V = cfg.tree_tokens, cfg.vocab
    states, same = [], [True, True]
    for s in range(2):
        prompt = synth.make_prompt(cfg, seq=s, n=60 + 17 * s)
        t0 = eng.prefill(s, prompt)
        st = o.prefill(prompt, slot=s)
        states.append(st)
        if t0 != st.t0:  # only a near-tie among the perturbed scores may separate them
            sc = np.sort(sampling.gumbel_scores(o.base.logits(o.base.forward_rows(prompt, np.arange(len(prompt)), None,
                         np.tril(np.ones((len(prompt),) * 2, dtype=bool)))[0][-1:])[0], cfg.temperature,
                         cfg.sample_seed, 1, 0, s, 0))
            assert sc[-1] - sc[-2] < 2 * tol / cfg.temperature, s
            same[s] = False
    near = 0
    for k in range(4):
        got = eng.step([0, 1])
        assert list(eng.debug("sample_step", np.int32, (2,))) == [k + 1, k + 1]
        vl = eng.debug("verify_logits", np.float32, (2 * T, V)).reshape(2, T, V)
        tg = eng.debug("target", np.int32, (2 * T,)).reshape(2, T)
        for s in range(2):
            scores = sampling.gumbel_scores(vl[s], cfg.temperature, cfg.sample_seed, 0, k, s, np.arange(T))
            want = np.argmax(scores, axis=1)
            top2 = np.sort(scores, axis=1)[:, -2:]
            clear = (top2[:, 1] - top2[:, 0]) >= 1e-4
            near += int(np.sum(~clear))
            assert np.array_equal(tg[s][clear], want[clear]), (k, s)
            if same[s]:
                ref, det = o.step(states[s])
                sc = np.sort(sampling.gumbel_scores(det["ver"].logits, cfg.temperature, cfg.sample_seed, 0, k, s,
                                                    np.arange(T)), axis=1)
                if np.min(sc[:, -1] - sc[:, -2]) >= 2 * tol / cfg.temperature and \
                        np.array_equal(eng.debug("tree_token", np.int32, (2, T))[s], det["tree"].tokens):
                    assert got[s] == ref, (k, s)
                else:
                    same[s] = False
    note(f"sampling {which}: {near} near-tie draws skipped")


def test_context_fills_then_step_is_refused_and_slot_is_reused():
    """A sequence steps until its next tree no longer fits (committed tokens + T >
    max_context): every step before that matches the oracle, the refused step returns
    CAPACITY and leaves the sequence as it was, and a released slot takes a new prompt."""
    P = need_gpu()
    note("engine capacity: fill one sequence's context")
    cfg, w = _tiny(batch=1)
    T, cap = cfg.tree_tokens, 200
    eng = _engine(P, cfg, w, max_context=cap)
    o = oracle.CloverOracle(cfg, w)
    prompt = synth.make_prompt(cfg, n=cap - T - 6)
    st = o.prefill(prompt)
    assert eng.prefill(0, prompt) == st.t0
    steps = 0
    while True:
        L = eng.seq_len(0)
        if L + T > cap:
            with pytest.raises(P.CloverError) as e:
                eng.step([0])
            assert e.value.status == 2
            assert eng.seq_len(0) == L
            break
        assert eng.step([0])[0] == o.step(st)[0], steps
        assert eng.seq_len(0) == st.L
        steps += 1
        assert steps < 10
    assert steps >= 1
    eng.release(0)
    prompt2 = synth.make_prompt(cfg, seq=1, n=40)
    st2 = o.prefill(prompt2)
    assert eng.prefill(0, prompt2) == st2.t0
    for _ in range(3):
        assert eng.step([0])[0] == o.step(st2)[0]
    eng.close()
