"""Parity at the full benchmark workloads, in the launch configuration the benchmark times.

Workloads (bf16, HIP-graph replay, the engine's default):
- llama7b_b1: 32 layers, d_model 4096, 32 heads of 128, SwiGLU 11008, vocab 125696,
  Clover heads with top-k (8, 4, 2) truncated to a 64-token tree, batch 1, 1024-token
  prompt;
- llama7b_b8: the same model, 8 sequences with seeded prompt lengths in 2048..4096 on
  the paged KV cache, 512 verify rows;
- large_gqa_b1: 80 layers, d_model 8192, 64 query / 8 KV heads of 128, SwiGLU 28672,
  4 Clover heads with top-k (8, 4, 2, 2), batch 1, 2048-token prompt;
- llama7b_b8 with speculative sampling at temperature 0.8 (`bench.py --workload llama7b_b8
  --temperature 0.8`): the 512-row LM head's sampled argmax epilogue at full size;
- llama7b_b1_medusa (`bench.py --draft medusa`): the Medusa heads on x_N of the last
  committed token and their Cartesian-product tree, at the 7B shape.

The float64 oracle cannot run these forwards in a test, so it recomputes sampled
outputs one by one from the GPU's own inputs to that stage, and the discrete stages
are checked exactly, for every sequence of the batch:

- draft: the root's head-1 logits (Regressive Connection, Attention Decoder, head MLP,
  final norm, shared LM head) from h0 and t0 (Sec. 3.1-3.4); for Medusa every head's
  logits (head MLP on h0, final norm, shared LM head);
- top-k children of every frontier row of every depth, their cumulative log-probs, and
  the truncated tree and its ancestor mask, from the GPU's draft logits;
- verify: final norm + LM head on sampled tree rows from the residual after the last
  layer, and target = argmax of every row (with sampling: on sampled rows, the oracle's
  Gumbel-max draw from the GPU's logits, wherever the top two perturbed scores are not
  within 1e-4);
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
WORKLOADS = ["llama7b_b1", "llama7b_b8", "large_gqa_b1", "llama7b_b8@0.8", "llama7b_b1_medusa"]


def _f64(t):
    return t.double().cpu().numpy()


@pytest.fixture(scope="module", params=WORKLOADS)
def run(request):
    P = need_gpu()
    name, _, temp = request.param.partition("@")
    cfg = synth.get_config(name)
    if temp:
        cfg = cfg.with_(temperature=float(temp), sample_seed=31)
    B, T, H, V, d = cfg.batch, cfg.tree_tokens, cfg.n_spec_heads, cfg.vocab, cfg.d_model
    lens = [cfg.prompt_len[0]] if B == 1 else synth.make_prompt_lengths(cfg)
    note(f"full-size workload {cfg.name}: weights on device, prompts {lens}")
    w = synth.make_weights(cfg, seed=0, device="cuda")
    # the oracle's copies of what the sampled checks read, taken before packing frees the
    # device sources (the large model's weights and their packed copies would not both fit)
    medusa = cfg.draft == "medusa"
    heads = [f"head{j}.{k}" for j in range(cfg.n_spec_heads if medusa else 1) for k in ("w1", "b1")]
    names = (["final_norm", "lm_head"] + ([] if medusa else ["ad.norm", "ad.wq", "ad.wk", "ad.wv", "ad.wo"])
             + heads + [f"layer0.{f}" for f in LayerWeights.__dataclass_fields__])
    host = {n: _f64(w[n]) for n in names}
    emb = w["emb"].cpu()
    eng = P.CloverEngine(cfg, w, max_batch=B, max_context=max(lens) + 256, free_source=True,
                         flags=P.FLAG_KEEP_LOGITS)
    del w
    torch.cuda.empty_cache()
    for b in range(B):
        note(f"prefill sequence {b}: {lens[b]} tokens")
        eng.prefill(b, synth.make_prompt(cfg, seq=b, n=lens[b]))
    seqs = list(range(B))
    note("one graph-replayed step")
    eng.step(seqs)  # warm-up step: captures the graphs
    t0 = eng.debug("t0", np.int32, (B,))
    sample_step = eng.debug("sample_step", np.int32, (B,))  # the counters the next step draws with
    h0 = eng.debug("h0", np.float32, (B, d)).astype(np.float64)
    L = [eng.seq_len(b) for b in seqs]
    out = eng.step(seqs)
    ncand, F = 1, 1
    for k in cfg.topk:
        F *= k
        ncand += F
    r = {
        "cfg": cfg, "B": B, "t0": t0, "h0": h0, "L": L, "out": out, "sample_step": sample_step,
        "cand_token": eng.debug("cand_token", np.int32, (B, ncand)),
        "cand_parent": eng.debug("cand_parent", np.int32, (B, ncand)),
        "cand_depth": eng.debug("cand_depth", np.int32, (B, ncand)),
        "cand_lp": eng.debug("cand_lp", np.float32, (B, ncand)),
        "tree_token": eng.debug("tree_token", np.int32, (B, T)),
        "tree_parent": eng.debug("tree_parent", np.int32, (B, T)),
        "tree_depth": eng.debug("tree_depth", np.int32, (B, T)),
        "tree_pos": eng.debug("tree_pos", np.int32, (B, T)),
        "tree_mask": eng.debug("tree_mask", np.uint64, (B, T, (T + 63) // 64)),
        "target": eng.debug("target", np.int32, (B * T,)).reshape(B, T),
        "acc": eng.debug("acc", np.int32, (B, H + 1)),
        "acc_len": eng.debug("acc_len", np.int32, (B,)),
        "verify_logits": eng.debug("verify_logits", np.float32, (B * T, V)).reshape(B, T, V),
        "x_last": eng.debug("x_last", np.float32, (B * T, d)).astype(np.float64).reshape(B, T, d),
        "L_after": [eng.seq_len(b) for b in seqs],
        "w": host,
    }
    F = 1
    for j in range(1, H + 1):
        rows = 1 if medusa else F  # Medusa: one row per head and sequence, whatever the depth
        r[f"draft_logits{j}"] = eng.debug(f"draft_logits{j}", np.float32, (B * rows, V)).reshape(B, rows, V)
        F *= cfg.topk[j - 1]
    r["kv0"], r["emb_rows"] = [], []
    for b in seqs:
        acc = r["acc"][b][: r["acc_len"][b]]
        r["kv0"].append([(eng.debug_kv(b, 0, L[b] + j, False), eng.debug_kv(b, 0, L[b] + j, True))
                         for j in range(len(acc))])
        toks = [int(r["tree_token"][b][a]) for a in acc]
        r["emb_rows"].append(emb[torch.tensor(toks)].double().numpy())
    eng.close()
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
    if cfg.draft == "medusa":
        for b in range(r["B"]):
            for j in range(cfg.n_spec_heads):
                rr = head_mlp(r["h0"][b], w[f"head{j}.w1"], w[f"head{j}.b1"], prec)
                err = float(np.max(np.abs(r[f"draft_logits{j + 1}"][b][0] - _lm_logits(r, rr)[0])))
                note(f"{cfg.name} Medusa head {j + 1} of sequence {b}: max |err| {err:.3e}")
                assert err <= LOGIT_TOL, (b, j)
        return
    for b in range(r["B"]):
        e = rc_embed(w["lm_head"], int(r["t0"][b]))
        s = attention_decoder(r["h0"][b], e, w, cfg.n_heads, cfg.head_dim, cfg.rms_eps, prec)
        rr = head_mlp(s, w["head0.w1"], w["head0.b1"], prec)
        ref = _lm_logits(r, rr)[0]
        err = float(np.max(np.abs(r["draft_logits1"][b][0] - ref)))
        note(f"{cfg.name} draft root row of sequence {b}: max |err| {err:.3e}")
        assert err <= LOGIT_TOL, b


def test_fullsize_topk_lp_and_tree_exact(run):
    r = run
    cfg = r["cfg"]
    T = cfg.tree_tokens
    for b in range(r["B"]):
        tok, par, dep, lp = r["cand_token"][b], r["cand_parent"][b], r["cand_depth"][b], r["cand_lp"][b]
        assert tok[0] == r["t0"][b] and par[0] == -1 and dep[0] == 0
        # children of the frontier rows of each depth, in creation order
        idx = 1
        frontier = [0]
        for j in range(1, cfg.n_spec_heads + 1):
            k = cfg.topk[j - 1]
            dl = r[f"draft_logits{j}"][b]
            nxt = []
            for f, node in enumerate(frontier):
                # Medusa: every node of the depth expands with the head's one list
                logits = dl[0 if cfg.draft == "medusa" else f].astype(np.float64)
                want = topk_ids(logits, k)
                logp = logits - logsumexp(logits)
                for c in range(k):
                    assert dep[idx] == j and par[idx] == node
                    assert tok[idx] == want[c], (b, j, f, c)
                    exp_lp = np.float32(np.float32(lp[node]) + np.float32(logp[want[c]]))
                    assert abs(float(lp[idx]) - float(exp_lp)) <= 1e-4
                    nxt.append(idx)
                    idx += 1
            frontier = nxt
        assert idx == len(tok)
        tree = oracle.build_tree(dep, tok, par, lp, T, r["L"][b])
        assert np.array_equal(r["tree_token"][b], tree.tokens), b
        assert np.array_equal(r["tree_parent"][b], tree.parent), b
        assert np.array_equal(r["tree_depth"][b], tree.depth), b
        assert np.array_equal(r["tree_pos"][b], tree.pos), b
        m = oracle.tree_mask(tree.parent)
        words = np.zeros((T, (T + 63) // 64), dtype=np.uint64)
        for i in range(T):
            for j in range(T):
                if m[i, j]:
                    words[i, j // 64] |= np.uint64(1) << np.uint64(j % 64)
        assert np.array_equal(r["tree_mask"][b], words), b


def test_fullsize_verify_lm_head_rows_and_targets(run):
    r = run
    cfg = r["cfg"]
    rows = [0, 1, 9, 33, 63]
    for b in range(r["B"]):
        vl = r["verify_logits"][b]
        if cfg.temperature > 0:
            # the draws of sampled rows: node n of sequence slot b at this step's counter
            from oracle import sampling
            sc = sampling.gumbel_scores(vl[rows], cfg.temperature, cfg.sample_seed, sampling.DOMAIN_VERIFY,
                                        int(r["sample_step"][b]), b, np.asarray(rows))
            want = np.argmax(sc, axis=1)
            top2 = np.sort(sc, axis=1)[:, -2:]
            clear = (top2[:, 1] - top2[:, 0]) >= 1e-4
            assert np.array_equal(r["target"][b][rows][clear], want[clear]), b
        else:
            assert np.array_equal(r["target"][b], np.argmax(vl, axis=1)), b
        ref = _lm_logits(r, r["x_last"][b][rows])
        err = float(np.max(np.abs(vl[rows] - ref)))
        note(f"{r['cfg'].name} verify LM-head rows {rows} of sequence {b}: max |err| {err:.3e}")
        assert err <= LOGIT_TOL, b


def test_fullsize_acceptance_and_emitted_tokens(run):
    r = run
    for b in range(r["B"]):
        acc, bonus = oracle.accept(r["tree_token"][b], r["tree_parent"][b], r["target"][b])
        assert list(r["acc"][b][: r["acc_len"][b]]) == list(acc), b
        emitted = [int(r["tree_token"][b][a]) for a in acc[1:]] + [int(bonus)]
        assert list(r["out"][b]) == emitted, b
        assert r["L_after"][b] == r["L"][b] + len(acc), b


def test_fullsize_layer0_committed_kv(run):
    r = run
    cfg, w = r["cfg"], r["w"]
    prec = oracle.model.Precision(cfg.dtype)
    lw = LayerWeights.from_dict(w, "layer0")
    z = np.zeros((0, cfg.n_kv_heads, cfg.head_dim))
    for b in range(r["B"]):
        acc = r["acc"][b][: r["acc_len"][b]]
        for j, node in enumerate(acc):
            pos = r["L"][b] + j  # committed position = L + depth of the accepted node
            assert r["tree_pos"][b][node] == pos
            _, k, v = layer_forward(r["emb_rows"][b][j: j + 1], np.array([pos]), lw, z, z,
                                    np.ones((1, 1), dtype=bool), cfg.n_heads, cfg.n_kv_heads,
                                    cfg.head_dim, cfg.rms_eps, cfg.rope_theta, prec)
            for got, ref in ((r["kv0"][b][j][0], k.reshape(-1)), (r["kv0"][b][j][1], v.reshape(-1))):
                rel = np.abs(got - ref) / (np.abs(ref) + 0.05)
                # both sides hold bf16 values; they may differ by one bf16 step where the
                # fp32 and fp64 sums fall on either side of a rounding boundary
                assert float(np.max(rel)) <= 1.0 / 64, (b, j, float(np.max(rel)))
