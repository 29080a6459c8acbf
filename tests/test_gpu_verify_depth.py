"""Full-depth parity at the benchmarked model shapes (bf16).

At the 7B shape (32 layers, d_model 4096) and the 80-layer GQA shape (d_model 8192, 64
query / 8 KV heads), with a 64-token prompt, the engine runs:

1. prefill, then one drafted speculate-and-verify step (Sec. 2.1, 3);
2. a planted 64-node tree holding the target's two best continuations at every depth
   below the root (`clover_verify_tree`), so a path of full length is accepted and
   compacted;
3. (7B shape) one more drafted step, whose draft starts from the Augmenting Block state
   the planted step committed.

The residual-stream trace (`clover_debug_trace`) records what enters every layer, the
residual after the last layer and the Augmenting Block's output, for every launch.  The
float64 oracle then runs every layer on the GPU's own inputs to that layer (teacher
forcing per layer), over the prompt and each step's tree against the KV the passes before
committed, and compares the layer's output with the GPU's input to the next layer.  It
streams the model one layer at a time: each layer's weights are drawn again on the device
from the per-tensor seeded generators the engine's weights came from (a subset of
`synth.make_weights` is the same values), converted to float64 on the host, used for all
rows, and dropped, so float64 copies of the whole model never coexist.

Checked against the oracle:
- every layer (and the Augmenting Block) on every pass: the rms and the largest element of
  out - GPU within LAYER_RMS_TOL and LAYER_MAX_TOL of the rms of the layer's own increment;
- the first token after the prompt; every drafted root row from the GPU's h_0; all 64
  verify rows of every step from the GPU's x_N: logits max-abs <= 2e-2;
- targets = argmax and acceptance (exact; against the oracle's own logits wherever no
  decision is within 2 x tol of a tie);
- the committed K/V of the planted path on every layer, within one bf16 step;
- (7B shape) the free-running end-to-end forward (the oracle's own residual stream through
  all 32 layers): within the noise floor that two valid accumulation orders of the same
  bf16 precision model show at this depth (oracle/noise_floor.py).

Checked on the GPU alone (bit-exact): after the planted step, on every layer, each accepted
node's K and V in its tree slot equal the committed slot's, byte for byte (the accepted
nodes sit at tree indices past the accepted length, so compaction leaves their sources in
place).
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from oracle.clover import attention_decoder, head_mlp, rc_embed
from oracle.model import BaseModel, LayerWeights, Precision, layer_forward
from tests.gpu_util import need_gpu, note

pytestmark = pytest.mark.gpu

LOGIT_TOL = 2e-2
PROMPT = 64
# One layer on identical inputs: the GPU and the oracle round to bf16 at the same points but
# accumulate in different orders (fp32 vs fp64), so an element whose value lies within the
# accumulation difference of a bf16 rounding boundary rounds one step (2^-8 relative) apart,
# and the GPU also rounds the attention probabilities to bf16.  Bounds on the layer's output
# error relative to the rms of the layer's increment (what the layer adds to the stream): the
# error's rms (one-step roundings of a small fraction of elements, each about 2^-9 of the
# element, carried through one layer's products) and its largest element (the increments
# are heavy-tailed: a relative error near 2^-9 on the largest elements of the increment is
# about 1e-2 of the increment's rms).
LAYER_RMS_TOL, LAYER_MAX_TOL = 5e-3, 5e-2
# End to end through 32 layers: the drift between two valid accumulation orders of the bf16
# precision model, measured by oracle/noise_floor.py at the 7B shape over 64 rows, is 0.15
# max-abs and 0.021 mean-abs on the logits; the bounds allow three times that.
E2E_MAX, E2E_MEAN = 0.46, 0.063
# (workload, drafted step after the planted one)
WORKLOADS = [("llama7b_b1", True), ("large_gqa_b1", False)]


def _fetch(cfg, names):
    """float64 host copies of the named weights, drawn again on the device."""
    w = synth.make_weights(cfg, seed=0, device="cuda", names=set(names))
    out = {n: t.double().cpu().numpy() for n, t in w.items()}
    del w
    return out


def _planted_tree(rng, T, H, root, top2_after, vocab):
    """T nodes: H + 1 decoy children of the root first, then the binary tree of the target's
    two best continuations at every depth down to H (top2_after(path) gives them for the
    tokens below the root), then random decoys under nodes of depth < H.  Every continuation
    node's index exceeds the longest acceptance, H + 1, and the path the verify accepts
    follows its own argmax whenever that is one of the two best of the probe that chose
    the children (two forward passes of different row counts differ in the last bits, so
    the probe's best may lose a near tie)."""
    tokens, parents, depth = [root], [-1], [0]
    first = top2_after([])
    for _ in range(H + 1):
        t = int(rng.integers(0, vocab))
        while t in first:
            t = int(rng.integers(0, vocab))
        tokens.append(t); parents.append(0); depth.append(1)
    level = [(0, [])]
    for d in range(1, H + 1):
        nxt = []
        for node, path in level:
            for t in (first if node == 0 else top2_after(path)):
                tokens.append(int(t)); parents.append(node); depth.append(d)
                nxt.append((len(tokens) - 1, path + [int(t)]))
        level = nxt
    assert len(tokens) <= T
    while len(tokens) < T:
        p = int(rng.choice([i for i in range(len(tokens)) if depth[i] < H]))
        tokens.append(int(rng.integers(0, vocab))); parents.append(p); depth.append(depth[p] + 1)
    return tokens, parents


def _gpu_step_record(eng, cfg, B_rows):
    T, V, H = cfg.tree_tokens, cfg.vocab, cfg.n_spec_heads
    acc_len = int(eng.debug("acc_len", np.int32, (eng.c.max_batch,))[0])
    return dict(
        tree_token=eng.debug("tree_token", np.int32, (eng.c.max_batch, T))[0].copy(),
        tree_parent=eng.debug("tree_parent", np.int32, (eng.c.max_batch, T))[0].copy(),
        logits=eng.debug("verify_logits", np.float32, (T, V)).astype(np.float64),
        target=eng.debug("target", np.int32, (T,)).copy(),
        acc=[int(a) for a in eng.debug("acc", np.int32, (eng.c.max_batch, H + 1))[0][:acc_len]],
        L=eng.seq_len(0),
    )


@pytest.fixture(scope="module", params=WORKLOADS, ids=[w for w, _ in WORKLOADS])
def run(request):
    P = need_gpu()
    name, third_step = request.param
    cfg = synth.get_config(name).with_(batch=1, prompt_len=(PROMPT, PROMPT))
    T, H, V, d = cfg.tree_tokens, cfg.n_spec_heads, cfg.vocab, cfg.d_model
    note(f"full-depth {name}: weights on device")
    w = synth.make_weights(cfg, seed=0, device="cuda")
    eng = P.CloverEngine(cfg, w, max_batch=2, max_context=PROMPT + 4 * T + 64, free_source=True,
                         flags=P.FLAG_KEEP_LOGITS)
    del w
    torch.cuda.empty_cache()
    rows = max(PROMPT, T)
    buf = torch.zeros((cfg.n_layers + 2) * rows * d, dtype=torch.float32, device="cuda")

    def trace(n):
        return buf[:(cfg.n_layers + 2) * n * d].view(cfg.n_layers + 2, n, d).double().cpu().numpy()

    eng.set_trace(buf)
    prompt = synth.make_prompt(cfg, n=PROMPT)
    r = {"cfg": cfg, "prompt": prompt, "steps": []}
    note(f"full-depth {name}: prefill and a drafted step")
    r["t0"] = eng.prefill(0, prompt)
    r["trace_prompt"] = trace(PROMPT)
    out1 = eng.step([0])
    s1 = _gpu_step_record(eng, cfg, 1)
    s1["draft_root"] = eng.debug("draft_logits1", np.float32, (2, V))[0].astype(np.float64)
    s1["out"], s1["L_before"], s1["trace"] = out1[0], PROMPT, trace(T)
    r["steps"].append(s1)
    committed = prompt + [int(s1["tree_token"][a]) for a in s1["acc"]]
    root = out1[0][-1]
    # the target's two best continuations after the root and each path below it, from
    # prefills of slot 1 (untraced; the prefill's LM-head row is kept with the logits)
    eng.set_trace(None)

    def top2_after(path):
        eng.prefill(1, committed + [root] + path)
        row = eng.debug("verify_logits", np.float32, (1, V))[0]
        eng.release(1)
        return [int(t) for t in np.lexsort((np.arange(V), -row))[:2]]

    rng = np.random.default_rng(7)
    toks, pars = _planted_tree(rng, T, H, root, top2_after, V)
    eng.set_trace(buf)
    note(f"full-depth {name}: planted tree of the target's top-2 continuations, {len(toks)} nodes")
    L2 = eng.seq_len(0)
    out2 = eng.verify_tree(0, toks, pars)
    s2 = _gpu_step_record(eng, cfg, 1)
    s2["out"], s2["L_before"], s2["trace"] = out2, L2, trace(T)
    A2 = len(s2["acc"])
    # byte-exact compaction on every layer (the Augmenting Block's is layer n_layers)
    n_kv_layers = cfg.n_layers + (1 if cfg.ab_kind in ("full", "attn") else 0)
    s2["kv_committed"] = {}
    mism = 0
    for layer in range(n_kv_layers):
        for j in range(A2):
            for which in (0, 1):
                dst = eng.debug_kv(0, layer, L2 + j, bool(which))
                src = eng.debug_kv(0, layer, L2 + s2["acc"][j], bool(which))
                mism += int(not np.array_equal(dst.view(np.uint32), src.view(np.uint32)))
                s2["kv_committed"][(layer, j, which)] = dst.astype(np.float64)
    s2["compaction_mismatches"] = mism
    r["steps"].append(s2)
    if third_step:
        out3 = eng.step([0])
        s3 = _gpu_step_record(eng, cfg, 1)
        s3["draft_root"] = eng.debug("draft_logits1", np.float32, (2, V))[0].astype(np.float64)
        s3["out"], s3["L_before"], s3["trace"] = out3[0], L2 + A2, trace(T)
        r["steps"].append(s3)
    eng.set_trace(None)
    eng.close()
    del eng, buf
    torch.cuda.empty_cache()
    r["oracle"] = _oracle_pass(cfg, r, free_running=third_step)
    return r


def _oracle_pass(cfg, r, free_running):
    """Every layer on the GPU's inputs to it (and, with free_running, the oracle's own residual
    stream beside), over the prompt and each step's tree, one layer at a time."""
    prec = Precision(cfg.dtype)
    nh, nkv, hd, eps, theta = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.rms_eps, cfg.rope_theta
    n = len(r["prompt"])
    NL = cfg.n_layers
    causal = np.tril(np.ones((n, n), dtype=bool))
    passes = [(np.arange(n), causal, None, r["trace_prompt"])]
    for s in r["steps"]:
        depth = np.zeros(len(s["tree_parent"]), dtype=np.int64)
        for i in range(1, len(depth)):
            depth[i] = depth[s["tree_parent"][i]] + 1
        passes.append((s["L_before"] + depth, oracle.tree_mask(s["tree_parent"]), s["acc"], s["trace"]))
    o = {"layer_err": [], "tree_kv": []}
    free = [p[3][0].copy() for p in passes] if free_running else None

    def run_stack(lw, inputs, kind):
        """One layer over every pass with this layer's cache; returns outputs and tree K/V."""
        attn, mlp = kind in ("full", "attn"), kind in ("full", "mlp")
        z = np.zeros((0, nkv, hd))
        kp = vp = z
        outs, kvs = [], []
        for (pos, mask, acc, _), x in zip(passes, inputs):
            xo, k, v = layer_forward(x, pos, lw, kp, vp, mask, nh, nkv, hd, eps, theta, prec, attn=attn, mlp=mlp)
            outs.append(xo)
            kvs.append((k, v))
            if attn:
                keep = np.arange(len(x)) if acc is None else np.asarray(acc)
                kp, vp = np.concatenate([kp, k[keep]]), np.concatenate([vp, v[keep]])
        return outs, kvs

    def compare(idx_in, idx_out, outs):
        """(rms, max) of the error over every pass, relative to the rms of the increment."""
        e_rms = e_max = 0.0
        for (_, _, _, tr), xo in zip(passes, outs):
            inc = tr[idx_out] - tr[idx_in]
            scale = float(np.sqrt(np.mean(inc * inc)))
            err = xo - tr[idx_out]
            e_rms = max(e_rms, float(np.sqrt(np.mean(err * err))) / scale)
            e_max = max(e_max, float(np.max(np.abs(err))) / scale)
        return e_rms, e_max

    fields = list(LayerWeights.__dataclass_fields__)
    for layer in range(NL):
        lw = LayerWeights.from_dict(_fetch(cfg, [f"layer{layer}.{f}" for f in fields]), f"layer{layer}")
        outs, kvs = run_stack(lw, [p[3][layer] for p in passes], "full")
        o["layer_err"].append(compare(layer, layer + 1, outs))
        o["tree_kv"].append(kvs[2])  # the planted pass
        if free_running:
            free, _ = run_stack(lw, free, "full")
        del lw
        if layer % 8 == 7:
            note(f"{cfg.name} oracle: {layer + 1} of {NL} layers, worst layer error so far "
                 f"rms {max(e[0] for e in o['layer_err']):.3e}, max {max(e[1] for e in o['layer_err']):.3e}")
    kind = cfg.ab_kind
    wab = _fetch(cfg, [f"ab.{f}" for f in fields])
    outs, kvs = run_stack(LayerWeights.from_dict(wab, "ab", partial=True), [p[3][NL] for p in passes], kind)
    o["ab_err"] = compare(NL, NL + 1, outs)
    o["tree_kv"].append(kvs[2])
    head = ["final_norm", "lm_head", "ad.norm", "ad.wq", "ad.wk", "ad.wv", "ad.wo", "head0.w1", "head0.b1"]
    w = _fetch(cfg, head)
    base = BaseModel(cfg.with_(n_layers=0), {"final_norm": w["final_norm"], "lm_head": w["lm_head"]})
    o["t0_logits"] = base.logits(r["trace_prompt"][NL][-1:])[0]
    o["verify_logits"] = [base.logits(s["trace"][NL]) for s in r["steps"]]
    if free_running:
        o["free_logits"] = [base.logits(x) for x in free[1:]]

    def draft_root(h0, t):
        e = rc_embed(w["lm_head"], int(t))
        s = attention_decoder(h0, e, w, cfg.n_heads, cfg.head_dim, cfg.rms_eps, prec)
        return base.logits(head_mlp(s, w["head0.w1"], w["head0.b1"], prec)[None, :])[0]

    # drafted steps read h_0 = the block's output at the last committed row of the pass before
    o["draft_root"] = {0: draft_root(r["trace_prompt"][NL + 1][-1], r["t0"])}
    if len(r["steps"]) > 2:
        s2 = r["steps"][1]
        o["draft_root"][2] = draft_root(s2["trace"][NL + 1][s2["acc"][-1]], s2["out"][-1])
    return o


def _margin(logits):
    top2 = np.sort(logits, axis=-1)[..., -2:]
    return top2[..., 1] - top2[..., 0]


@pytest.mark.timeout(900)
def test_every_layer_matches_oracle_on_its_own_inputs(run):
    o, cfg = run["oracle"], run["cfg"]
    errs = np.asarray(o["layer_err"])  # [layer][rms, max]
    note(f"{cfg.name}: per-layer error / rms(increment): rms worst {errs[:, 0].max():.3e} (layer "
         f"{int(errs[:, 0].argmax())}), median {np.median(errs[:, 0]):.3e}; max worst {errs[:, 1].max():.3e} "
         f"(layer {int(errs[:, 1].argmax())}), median {np.median(errs[:, 1]):.3e}; Augmenting Block "
         f"rms {o['ab_err'][0]:.3e}, max {o['ab_err'][1]:.3e}")
    assert errs[:, 0].max() <= LAYER_RMS_TOL, int(errs[:, 0].argmax())
    assert errs[:, 1].max() <= LAYER_MAX_TOL, int(errs[:, 1].argmax())
    assert o["ab_err"][0] <= LAYER_RMS_TOL and o["ab_err"][1] <= LAYER_MAX_TOL


@pytest.mark.timeout(900)
def test_lm_head_targets_and_drafted_roots_from_gpu_states(run):
    r, o = run, run["oracle"]
    cfg = r["cfg"]
    if _margin(o["t0_logits"]) >= 2 * LOGIT_TOL:
        assert r["t0"] == int(np.argmax(o["t0_logits"]))
    for i, s in enumerate(r["steps"]):
        err = float(np.max(np.abs(s["logits"] - o["verify_logits"][i])))
        note(f"{cfg.name} step {i}: LM head over all 64 rows from the GPU's x_N: max |err| {err:.3e}")
        assert err <= LOGIT_TOL, (i, err)
        # the fused argmax is the argmax of the stored logits (lowest index on ties)
        assert np.array_equal(s["target"], np.argmax(s["logits"], axis=1)), i
        clear = _margin(o["verify_logits"][i]) >= 2 * LOGIT_TOL
        assert np.array_equal(s["target"][clear], np.argmax(o["verify_logits"][i], axis=1)[clear]), i
    for i, ref in o["draft_root"].items():
        err = float(np.max(np.abs(r["steps"][i]["draft_root"] - ref)))
        note(f"{cfg.name} step {i}: drafted root row from the GPU's h_0: max |err| {err:.3e}")
        assert err <= LOGIT_TOL, (i, err)


@pytest.mark.timeout(900)
def test_acceptance_and_planted_path(run):
    r, o = run, run["oracle"]
    cfg = r["cfg"]
    for i, s in enumerate(r["steps"]):
        acc, bonus = oracle.accept(s["tree_token"], s["tree_parent"], s["target"])
        assert acc == s["acc"] and bonus == s["out"][-1], i
        assert s["out"][:-1] == [int(s["tree_token"][a]) for a in s["acc"][1:]]
        acc_o, bonus_o = oracle.accept(s["tree_token"], s["tree_parent"], np.argmax(o["verify_logits"][i], axis=1))
        if acc_o != s["acc"] or bonus_o != s["out"][-1]:
            on_path = sorted(set(acc_o) | set(s["acc"]))
            assert float(np.min(_margin(o["verify_logits"][i][on_path]))) < 2 * LOGIT_TOL, (i, acc_o, s["acc"])
    s2 = r["steps"][1]
    note(f"{cfg.name} planted step: accepted {s2['acc']}")
    assert len(s2["acc"]) == cfg.n_spec_heads + 1, s2["acc"]


@pytest.mark.timeout(900)
def test_compaction_bit_exact_and_committed_kv(run):
    r, o = run, run["oracle"]
    cfg = r["cfg"]
    s2 = r["steps"][1]
    assert s2["compaction_mismatches"] == 0
    worst = 0.0
    for (layer, j, which), got in s2["kv_committed"].items():
        ref = o["tree_kv"][layer][which][s2["acc"][j]].reshape(-1)
        worst = max(worst, float(np.max(np.abs(got - ref) / (np.abs(ref) + 0.05))))
    note(f"{cfg.name} committed K/V of the planted path ({len(s2['acc'])} rows) on {len(o['tree_kv'])} "
         f"layers: max |err| / (|ref| + 0.05) = {worst:.3e}")
    # both sides hold bf16 values computed from the same layer input; they may differ by one
    # bf16 step where the fp32 and fp64 sums fall on either side of a rounding boundary
    assert worst <= 1.0 / 64


@pytest.mark.timeout(900)
def test_end_to_end_within_the_precision_noise_floor(run):
    r, o = run, run["oracle"]
    if "free_logits" not in o:
        pytest.skip("end-to-end pass only at the 7B shape")
    for i, s in enumerate(r["steps"]):
        d = np.abs(s["logits"] - o["free_logits"][i])
        note(f"{r['cfg'].name} step {i}: end-to-end logits through {r['cfg'].n_layers} layers: "
             f"max |err| {d.max():.3e}, mean {d.mean():.3e}")
        assert d.max() <= E2E_MAX and d.mean() <= E2E_MEAN, i
