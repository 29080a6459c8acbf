"""End-to-end parity of the C-ABI step against the oracle on seeded workloads."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.gpu_util import need_gpu, note

pytestmark = pytest.mark.gpu


def _engine(P, cfg, w, **kw):
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


def test_planted_trees_accept_every_length():
    P = need_gpu()
    note("engine planted trees")
    cfg, w = _tiny()
    o = oracle.CloverOracle(cfg, w)
    prompt = synth.make_prompt(cfg, seq=3)
    ar = o.base.greedy_generate(prompt, 12)
    H = cfg.n_spec_heads
    eng = _engine(P, cfg, w)
    for A in range(1, H + 2):
        t0 = eng.prefill(0, prompt)
        assert t0 == ar[0]
        toks, par, prev = [t0, (ar[1] + 1) % cfg.vocab], [-1, 0], 0
        for d in range(1, H + 1):
            toks.append(ar[d] if d < A else (ar[d] + 3) % cfg.vocab)
            par.append(prev)
            prev = len(toks) - 1
        got = eng.verify_tree(0, toks, par)
        assert got == ar[1:A + 1], (A, got)
        assert eng.debug("acc_len", np.int32, (1,))[0] == A
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


def test_bf16_small_model_within_tolerance():
    """bf16 storage: logits within 2e-2 of the oracle (which rounds at the same
    storage points); discrete results compared while no decision is a near tie."""
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
    tol = 2e-2
    for step in range(6):
        ours = eng.step([0])[0]
        ref, det = o.step(st)
        cands = det["cands"]
        F, base = 1, 0
        for j in range(1, cfg.n_spec_heads + 1):
            dl = eng.debug(f"draft_logits{j}", np.float32, (F, cfg.vocab))
            for f in range(F):
                err = np.max(np.abs(dl[f] - cands.row_logits[base + f]))
                assert err < tol, (step, j, f, err)
            base += F
            F *= cfg.topk[j - 1]
        T = cfg.tree_tokens
        same_tree = np.array_equal(eng.debug("tree_token", np.int32, (1, T))[0], det["tree"].tokens)
        if not same_tree:
            # only a near tie in the draft may separate the trees
            margins = [np.sort(l)[::-1] for l in cands.row_logits.values()]
            assert min(m[k - 1] - m[k] for m, k in zip(margins, [cfg.topk[cands.depth[n]] for n in cands.row_logits])) < 2 * tol
            break
        vl = eng.debug("verify_logits", np.float32, (T, cfg.vocab))
        assert np.max(np.abs(vl - det["ver"].logits)) < tol
        top2 = np.sort(det["ver"].logits, axis=1)[:, -2:]
        if np.min(top2[:, 1] - top2[:, 0]) < 2 * tol:
            break
        assert ours == ref, step


def test_graph_replay_matches_eager_launches():
    """The step's phases replay as HIP graphs captured per batch size; every replay,
    with host work and batch-size changes in between, matches eager launches bit for bit."""
    P = need_gpu()
    note("engine graph vs eager")
    cfg, w = _tiny(batch=2)
    prompts = [synth.make_prompt(cfg, seq=s, n=100 + 30 * s) for s in range(2)]
    g = _engine(P, cfg, w)
    e = _engine(P, cfg, w, flags=P.FLAG_EAGER)
    for s in range(2):
        assert g.prefill(s, prompts[s]) == e.prefill(s, prompts[s])
    schedule = [[0], [0, 1], [1], [0, 1], [0], [1, 0], [0, 1]]
    for i, seqs in enumerate(schedule):
        if i == 3:
            g.set_flags(P.FLAG_EAGER)      # eager in the middle, graphs again after
        if i == 5:
            g.set_flags(0)
        a, b = g.step(seqs), e.step(seqs)
        assert a == b, (i, seqs, a, b)
        rows = len(seqs) * cfg.tree_tokens
        va = g.debug("verify_logits", np.float32, (rows, cfg.vocab))
        vb = e.debug("verify_logits", np.float32, (rows, cfg.vocab))
        assert np.array_equal(va, vb), i
        assert np.array_equal(g.debug("h0", np.float32, (2, cfg.d_model)), e.debug("h0", np.float32, (2, cfg.d_model)))
        torch.cuda.synchronize()
    assert g.seq_len(0) == e.seq_len(0) and g.seq_len(1) == e.seq_len(1)
