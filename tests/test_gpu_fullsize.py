"""Parity at the full 7B-shape workload, in the launch configuration the benchmark times.

Workload: 32 layers, d_model 4096, 32 heads of 128, SwiGLU 11008, vocab 125696, bf16,
Clover heads with top-k (8, 4, 2) truncated to a 64-token tree, batch 1, 1024-token
prompt, HIP-graph replay (the engine's default).  The float64 oracle cannot run the
whole 7B forward in a test, so it recomputes sampled outputs one by one from the
GPU's own inputs to that stage, and the discrete stages are checked exactly:

- draft: the root's head-1 logits (Regressive Connection, Attention Decoder, head MLP,
  final norm, shared LM head) from h0 and t0 (Sec. 3.1-3.4);
- top-k children of every frontier row of every depth, their cumulative log-probs, and
  the truncated tree and its ancestor mask, from the GPU's draft logits;
- verify: final norm + LM head on sampled tree rows from the residual after the last
  layer, and target = argmax of every row;
- acceptance from the tree and targets, and the emitted tokens;
- KV compaction: layer 0's committed K/V rows of the accepted nodes equal the oracle's
  layer-0 K/V of those tokens at their committed positions (embedding, RMSNorm, QKV,
  rotary, paged append and compaction).
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from oracle.clover import attention_decoder, head_mlp, rc_embed, topk_ids
from oracle.model import BaseModel, LayerWeights, layer_forward, logsumexp
from tests.gpu_util import need_gpu, note

pytestmark = pytest.mark.gpu

LOGIT_TOL = 2e-2  # bf16 workloads: max-abs on logits


def _f64(t):
    return t.double().cpu().numpy()


@pytest.fixture(scope="module")
def run():
    P = need_gpu()
    cfg = synth.get_config("llama7b_b1")
    note(f"full-size workload {cfg.name}: weights on device")
    w = synth.make_weights(cfg, seed=0, device="cuda")
    L0 = cfg.prompt_len[0]
    eng = P.CloverEngine(cfg, w, max_batch=1, max_context=L0 + 256)
    prompt = synth.make_prompt(cfg, seq=0, n=L0)
    note("prefill 1024 tokens")
    t0 = eng.prefill(0, prompt)
    h0 = eng.debug("h0", np.float32, (1, cfg.d_model))[0].astype(np.float64)
    L = eng.seq_len(0)
    note("one graph-replayed step")
    eng.step([0])  # warm-up step: captures the graphs
    t0 = int(eng.debug("t0", np.int32, (1,))[0])
    h0 = eng.debug("h0", np.float32, (1, cfg.d_model))[0].astype(np.float64)
    L = eng.seq_len(0)
    out = eng.step([0])[0]
    T, H, V, d = cfg.tree_tokens, cfg.n_spec_heads, cfg.vocab, cfg.d_model
    ncand = 1
    F = 1
    for k in cfg.topk:
        F *= k
        ncand += F
    r = {
        "cfg": cfg, "t0": t0, "h0": h0, "L": L, "out": out,
        "cand_token": eng.debug("cand_token", np.int32, (1, ncand))[0],
        "cand_parent": eng.debug("cand_parent", np.int32, (1, ncand))[0],
        "cand_depth": eng.debug("cand_depth", np.int32, (1, ncand))[0],
        "cand_lp": eng.debug("cand_lp", np.float32, (1, ncand))[0],
        "tree_token": eng.debug("tree_token", np.int32, (1, T))[0],
        "tree_parent": eng.debug("tree_parent", np.int32, (1, T))[0],
        "tree_depth": eng.debug("tree_depth", np.int32, (1, T))[0],
        "tree_pos": eng.debug("tree_pos", np.int32, (1, T))[0],
        "tree_mask": eng.debug("tree_mask", np.uint64, (1, T, (T + 63) // 64))[0],
        "target": eng.debug("target", np.int32, (1, T))[0],
        "acc": eng.debug("acc", np.int32, (1, H + 1))[0],
        "acc_len": int(eng.debug("acc_len", np.int32, (1,))[0]),
        "verify_logits": eng.debug("verify_logits", np.float32, (T, V)),
        "x_last": eng.debug("x_last", np.float32, (T, d)).astype(np.float64),
        "L_after": eng.seq_len(0),
    }
    F = 1
    for j in range(1, H + 1):
        r[f"draft_logits{j}"] = eng.debug(f"draft_logits{j}", np.float32, (F, V))
        F *= cfg.topk[j - 1]
    acc = r["acc"][: r["acc_len"]]
    r["kv0"] = [(eng.debug_kv(0, 0, L + j, False), eng.debug_kv(0, 0, L + j, True)) for j in range(len(acc))]
    note("oracle weights (float64) for the sampled checks")
    names = ["final_norm", "lm_head", "ad.norm", "ad.wq", "ad.wk", "ad.wv", "ad.wo",
             "head0.w1", "head0.b1"] + [f"layer0.{f}" for f in LayerWeights.__dataclass_fields__]
    r["w"] = {n: _f64(w[n]) for n in names}
    acc_tokens = [int(r["tree_token"][a]) for a in acc]
    r["emb_rows"] = _f64(w["emb"][torch.tensor(acc_tokens, device=w["emb"].device)])
    eng.close()
    del w
    torch.cuda.empty_cache()
    return r


def _lm_logits(r, rows):
    cfg = r["cfg"]
    base = BaseModel(cfg.with_(n_layers=0), {"final_norm": r["w"]["final_norm"], "lm_head": r["w"]["lm_head"]})
    return base.logits(np.atleast_2d(rows))


def test_fullsize_draft_root_row_matches_oracle(run):
    r = run
    cfg, w = r["cfg"], r["w"]
    prec = oracle.model.Precision(cfg.dtype)
    e = rc_embed(w["lm_head"], r["t0"])
    s = attention_decoder(r["h0"], e, w, cfg.n_heads, cfg.head_dim, cfg.rms_eps, prec)
    rr = head_mlp(s, w["head0.w1"], w["head0.b1"], prec)
    ref = _lm_logits(r, rr)[0]
    got = r["draft_logits1"][0]
    err = float(np.max(np.abs(got - ref)))
    note(f"draft root row: max |err| {err:.3e}")
    assert err <= LOGIT_TOL


def test_fullsize_topk_lp_and_tree_exact(run):
    r = run
    cfg = r["cfg"]
    tok, par, dep, lp = r["cand_token"], r["cand_parent"], r["cand_depth"], r["cand_lp"]
    assert tok[0] == r["t0"] and par[0] == -1 and dep[0] == 0
    # children of the frontier rows of each depth, in creation order
    idx = 1
    frontier = [0]
    for j in range(1, cfg.n_spec_heads + 1):
        k = cfg.topk[j - 1]
        dl = r[f"draft_logits{j}"]
        nxt = []
        for f, node in enumerate(frontier):
            logits = dl[f].astype(np.float64)
            want = topk_ids(logits, k)
            logp = logits - logsumexp(logits)
            for c in range(k):
                assert dep[idx] == j and par[idx] == node
                assert tok[idx] == want[c], (j, f, c)
                exp_lp = np.float32(np.float32(lp[node]) + np.float32(logp[want[c]]))
                assert abs(float(lp[idx]) - float(exp_lp)) <= 1e-4
                nxt.append(idx)
                idx += 1
        frontier = nxt
    assert idx == len(tok)
    tree = oracle.build_tree(dep, tok, par, lp, cfg.tree_tokens, r["L"])
    assert np.array_equal(r["tree_token"], tree.tokens)
    assert np.array_equal(r["tree_parent"], tree.parent)
    assert np.array_equal(r["tree_depth"], tree.depth)
    assert np.array_equal(r["tree_pos"], tree.pos)
    m = oracle.tree_mask(tree.parent)
    T = cfg.tree_tokens
    words = np.zeros((T, (T + 63) // 64), dtype=np.uint64)
    for i in range(T):
        for j in range(T):
            if m[i, j]:
                words[i, j // 64] |= np.uint64(1) << np.uint64(j % 64)
    assert np.array_equal(r["tree_mask"], words)


def test_fullsize_verify_lm_head_rows_and_targets(run):
    r = run
    vl = r["verify_logits"]
    assert np.array_equal(r["target"], np.argmax(vl, axis=1))
    rows = [0, 1, 9, 33, 63]
    ref = _lm_logits(r, r["x_last"][rows])
    err = float(np.max(np.abs(vl[rows] - ref)))
    note(f"verify LM-head rows {rows}: max |err| {err:.3e}")
    assert err <= LOGIT_TOL


def test_fullsize_acceptance_and_emitted_tokens(run):
    r = run
    acc, bonus = oracle.accept(r["tree_token"], r["tree_parent"], r["target"])
    assert list(r["acc"][: r["acc_len"]]) == list(acc)
    emitted = [int(r["tree_token"][a]) for a in acc[1:]] + [int(bonus)]
    assert list(r["out"]) == emitted
    assert r["L_after"] == r["L"] + len(acc)


def test_fullsize_layer0_committed_kv(run):
    r = run
    cfg, w = r["cfg"], r["w"]
    prec = oracle.model.Precision(cfg.dtype)
    lw = LayerWeights.from_dict(w, "layer0")
    acc = r["acc"][: r["acc_len"]]
    z = np.zeros((0, cfg.n_kv_heads, cfg.head_dim))
    for j, node in enumerate(acc):
        pos = r["L"] + j  # committed position = L + depth of the accepted node
        assert r["tree_pos"][node] == pos
        _, k, v = layer_forward(r["emb_rows"][j : j + 1], np.array([pos]), lw, z, z, np.ones((1, 1), dtype=bool),
                                cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.rms_eps, cfg.rope_theta, prec)
        for got, ref in ((r["kv0"][j][0], k.reshape(-1)), (r["kv0"][j][1], v.reshape(-1))):
            rel = np.abs(got - ref) / (np.abs(ref) + 0.05)
            # both sides hold bf16 values; they may differ by one bf16 step where the
            # fp32 and fp64 sums fall on either side of a rounding boundary
            assert float(np.max(rel)) <= 1.0 / 64, (j, float(np.max(rel)))
