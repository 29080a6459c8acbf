"""Clover speculator, token tree, verification and acceptance (oracle side).

Test infrastructure only.  Follows Sec. 3 of the paper:

* Regressive Connection (Sec. 3.1, 3.4): the embedding of a speculated token is
  its row of the LM-head weight after normalisation; read here as row-wise L2
  normalisation.
* Attention Decoder (Sec. 3.2, Eq. 1-2): Q from the RMS-normalised hidden state
  h_{i-1}, K and V from e_{i-1}; h_i = h_{i-1} + Attention(Q, K, V).  Read
  literally, the key set is the single vector e_{i-1}, so the softmax weight is
  exactly 1.  The attention has the base model's head layout and an output
  projection; its weights are shared by all heads.  Two other readings of the key
  set are selectable (``ad_keys``): the two vectors {RMSNorm(h), e} and the
  embeddings of every token on the node's root path.
* Per-head MLP (Sec. 3.2, Sec. 4.1 "Medusa initialisation"): read as the Medusa
  residual block r = h + SiLU(W1 h + b1), one per head.
* Shared LM head (Sec. 3.4): every head reuses the target's final norm and LM
  head.
* Augmenting Block (Sec. 3.3): one extra decoder layer over the residual stream
  after the last base layer, with its own KV cache; its output at the last
  committed position is h_0.
* Token tree (Sec. 2.2): per-depth top-k expansion, truncation to the
  configured number of verify tokens by cumulative log-probability, mask =
  ancestor-or-self matrix.  The paper names no tree construction or sampling
  algorithm (Sec. 4.1), so this one is a reading.
* Verification and greedy acceptance (Sec. 2.1): the target's argmax at each
  node decides which child, if any, is kept; the accepted path plus one bonus
  token is emitted, so outputs equal plain greedy decoding.

Pins of the head composition (tests/test_oracle_clover.py): the single-key closed form
of the Attention Decoder; the reduction with identity heads (no Augmenting Block, zero
decoder output projection, an MLP that adds nothing), where every node's head logits
must be the target's own next-token logits after the prompt; and the path-sum closed
form, where with the single key, no Augmenting Block and head MLPs W1_j = alpha_j I
every drafted row must equal W_lm RMSNorm_f(s + SiLU(alpha_j s + b1_j)) with
s = h_0 + sum of W_O W_V e(tok) over the node's root path.  That one fixes the
recursion of the decoder state, the token embedded at each depth, the head used at
each depth, the order of decoder and MLP and the MLP's residual form; planted mistakes
in each fail it.  What remains a reading rather than a pinned fact is the choice of
these forms themselves (the architecture figure is not available).
"""
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from . import sampling
from .model import BaseModel, LayerWeights, Precision, layer_forward, logsumexp, rmsnorm, silu


# --------------------------------------------------------------------------------------------
# small pure functions


def topk_ids(logits: np.ndarray, k: int) -> np.ndarray:
    """The k largest entries, ordered by value descending, then token id ascending."""
    ids = np.arange(logits.shape[0])
    order = np.lexsort((ids, -logits))
    return order[:k]


def rc_embed(w_lm: np.ndarray, token: int) -> np.ndarray:
    """Regressive Connection embedding: e(t) = W_lm[t] / max(||W_lm[t]||_2, 1e-12).

    Sec. 3.4: the one-hot token times the transposed, normalised LM-head weight.
    """
    row = w_lm[token]
    return row / max(float(np.sqrt(np.sum(row * row))), 1e-12)


def attention_decoder(h: np.ndarray, e_keys: np.ndarray, w: Dict[str, np.ndarray], n_heads: int,
                      head_dim: int, eps: float, prec: Precision) -> np.ndarray:
    """Sec. 3.2, Eq. 1-2.  h: [d] hidden state h_{i-1}; e_keys: [n_keys, d] token embeddings.

    Q = W_Q RMSNorm(h); K = W_K e; V = W_V e; h_i = h + W_O Attention(Q, K, V).
    """
    a = prec.store(rmsnorm(h, w["ad.norm"], eps))
    E = prec.store(np.atleast_2d(e_keys))
    q = (a @ w["ad.wq"].T).reshape(n_heads, head_dim)
    k = (E @ w["ad.wk"].T).reshape(-1, n_heads, head_dim)
    v = (E @ w["ad.wv"].T).reshape(-1, n_heads, head_dim)
    s = np.einsum("hd,khd->hk", q, k) / np.sqrt(head_dim)
    s = s - np.max(s, axis=1, keepdims=True)
    p = np.exp(s)
    p = p / np.sum(p, axis=1, keepdims=True)
    o = np.einsum("hk,khd->hd", p, v).reshape(-1)
    return h + prec.store(o) @ w["ad.wo"].T


def regressive_mlp(h: np.ndarray, e: np.ndarray, w: Dict[str, np.ndarray], eps: float,
                   prec: Precision) -> np.ndarray:
    """The MLP regressive block of the ablation (Sec. 3.2 last paragraph, Sec. 4.3): the two
    input vectors concatenated, h_i = h + SiLU(W_r [RMSNorm_r(h); e] + b_r)."""
    a = prec.store(rmsnorm(h, w["rb.norm"], eps))
    x = np.concatenate([a, prec.store(e)])
    return h + silu(x @ w["rb.w"].T + w["rb.b"])


def head_mlp(s: np.ndarray, w1: np.ndarray, b1: np.ndarray, prec: Precision) -> np.ndarray:
    """Per-head residual MLP block: r = s + SiLU(W1 s + b1)."""
    return s + silu(prec.store(s) @ w1.T + b1)


def tree_mask(parent: Sequence[int]) -> np.ndarray:
    """Ancestor-or-self matrix: mask[i][j] is True iff j == i or j is an ancestor of i."""
    T = len(parent)
    m = np.zeros((T, T), dtype=bool)
    for i in range(T):
        j = i
        while j >= 0:
            m[i, j] = True
            j = parent[j]
    return m


@dataclass
class Candidates:
    """Draft output in creation order (index 0 is the root)."""
    depth: np.ndarray
    token: np.ndarray
    parent: np.ndarray
    lp: np.ndarray                     # float32 cumulative log-probability
    row_logits: Dict[int, np.ndarray] = field(default_factory=dict)   # node -> head logits
    row_state: Dict[int, np.ndarray] = field(default_factory=dict)    # node -> AD output


@dataclass
class Tree:
    tokens: np.ndarray
    parent: np.ndarray
    depth: np.ndarray
    pos: np.ndarray
    mask: np.ndarray
    src: np.ndarray                    # candidate index of each tree node


def build_tree(depth, token, parent, lp, T: int, L: int) -> Tree:
    """Truncate the candidate tree to T verify tokens (root included).

    Non-root candidates are ranked by (lp descending, depth ascending, creation
    index ascending) and the first T-1 kept; the root and the kept nodes are then
    listed in creation order, which is breadth-first.  Positions are L + depth.
    """
    depth, token, parent = np.asarray(depth), np.asarray(token), np.asarray(parent)
    lp = np.asarray(lp, dtype=np.float32)
    n = len(depth)
    idx = np.arange(1, n)
    order = np.lexsort((idx, depth[1:], -lp[1:].astype(np.float64)))
    kept = np.sort(idx[order[: T - 1]])
    src = np.concatenate([[0], kept]).astype(np.int64)
    remap = {int(s): i for i, s in enumerate(src)}
    par = np.array([-1] + [remap[int(parent[s])] for s in kept], dtype=np.int64)
    dep = depth[src].astype(np.int64)
    return Tree(tokens=token[src].astype(np.int64), parent=par, depth=dep, pos=L + dep,
                mask=tree_mask(par), src=src)


def accept(tokens: Sequence[int], parent: Sequence[int], target: Sequence[int]):
    """Greedy acceptance (Sec. 2.1): follow the children whose token equals the
    target's argmax at their parent; the lowest-index matching child wins.

    Returns (acc, bonus): acc lists accepted node indices starting at the root,
    bonus is the target's argmax at the last accepted node.
    """
    acc = [0]
    cur = 0
    while True:
        nxt = None
        for c in range(len(tokens)):
            if parent[c] == cur and tokens[c] == target[cur]:
                nxt = c
                break
        if nxt is None:
            break
        acc.append(nxt)
        cur = nxt
    return acc, int(target[cur])


# --------------------------------------------------------------------------------------------
# stateful decoding


@dataclass
class SeqState:
    tokens: List[int]                                  # committed tokens, positions 0..L-1
    kv: List[Tuple[np.ndarray, np.ndarray]]           # per base layer, [L, n_kv, hd]
    ab_kv: Optional[Tuple[np.ndarray, np.ndarray]]     # Augmenting Block cache (None: no attention)
    h0: np.ndarray                                     # AB output at position L-1
    t0: int                                            # next token (root of the next tree)
    slot: int = 0                                      # sequence slot (sampling counters)
    steps: int = 0                                     # speculate-and-verify steps committed

    @property
    def L(self) -> int:
        return len(self.tokens)


@dataclass
class VerifyOut:
    logits: np.ndarray            # [T, V]
    target: np.ndarray            # [T] argmax, lowest id on ties
    x_last: np.ndarray            # [T, d] residual after the last base layer
    kv: List[Tuple[np.ndarray, np.ndarray]]   # per layer, tree-node K/V [T, n_kv, hd]


class CloverOracle:
    def __init__(self, cfg, weights):
        self.cfg = cfg
        self.w = {k: (v.double().numpy() if hasattr(v, "double") else np.asarray(v, dtype=np.float64))
                  for k, v in weights.items()}
        self.base = BaseModel(cfg, self.w)
        self.prec = self.base.prec
        self.ab_kind = getattr(cfg, "ab_kind", "full")
        self.ab = None if self.ab_kind == "none" else LayerWeights.from_dict(self.w, "ab", partial=True)

    # -- Augmenting Block -------------------------------------------------------------------
    def ab_forward(self, x_rows, pos, ab_kv, tail_visible):
        """Sec. 3.3 (and the variants of Sec. 4.3): the whole layer, its attention or MLP half,
        or none (the rows pass through).  Returns (h, k_new, v_new); k/v None without attention."""
        c = self.cfg
        if self.ab_kind == "none":
            return x_rows, None, None
        attn = self.ab_kind in ("full", "attn")
        kp, vp = ab_kv if attn else (None, None)
        return layer_forward(x_rows, np.asarray(pos), self.ab, kp, vp, tail_visible,
                             c.n_heads, c.n_kv_heads, c.head_dim, c.rms_eps, c.rope_theta,
                             self.prec, attn=attn, mlp=self.ab_kind in ("full", "mlp"))

    # -- prefill (Sec. 1: the prompt is processed in one pass and yields the first token) ---
    # -- the target's choice of token: greedy argmax, or a sample (oracle/sampling.py) -----
    def target_token(self, logits: np.ndarray, domain: int, step: int, slot: int, node: int) -> int:
        tau = float(getattr(self.cfg, "temperature", 0.0))
        if tau <= 0.0:
            return int(np.argmax(logits))
        return sampling.sample_token(logits, tau, int(getattr(self.cfg, "sample_seed", 0)), domain, step,
                                     slot, node)

    def prefill(self, prompt: Sequence[int], slot: int = 0) -> SeqState:
        n = len(prompt)
        causal = np.tril(np.ones((n, n), dtype=bool))
        x, kv = self.base.forward_rows(prompt, np.arange(n), None, causal)
        t0 = self.target_token(self.base.logits(x[-1:])[0], sampling.DOMAIN_PREFILL, 0, slot, 0)
        h, k, v = self.ab_forward(x, np.arange(n), self.base.empty_kv(), causal)
        return SeqState(tokens=list(prompt), kv=kv, ab_kv=None if k is None else (k, v),
                        h0=h[-1].copy(), t0=t0, slot=slot)

    # -- drafting (Sec. 3) ---------------------------------------------------------------
    def head_logits(self, j: int, s: np.ndarray) -> np.ndarray:
        r = head_mlp(s, self.w[f"head{j}.w1"], self.w[f"head{j}.b1"], self.prec)
        return self.base.logits(r[None, :])[0]

    def decoder_weights(self, j: int) -> Dict[str, np.ndarray]:
        """The Attention Decoder that drafts depth j: the shared ad.* set (Eq. 1 has no head
        index), or head j's own ad{j-1}.* set when the configuration gives each head one."""
        if not getattr(self.cfg, "ad_per_head", False) or getattr(self.cfg, "regressive", "attention") == "mlp":
            return self.w
        return {f"ad.{f}": self.w[f"ad{j - 1}.{f}"] for f in ("norm", "wq", "wk", "wv", "wo")}

    def ad_keys(self, h: np.ndarray, n: int, token, parent, wad) -> np.ndarray:
        """Key/value inputs of the Attention Decoder for node n with state h (Eq. 1; the key
        set is a reading): "single" {e(token_n)}; "two" {RMSNorm_ad(h), e(token_n)} (Sec. 3.2:
        two vectors per request or beam); "path" {e(t) for every token on n's root path,
        root first}."""
        kind = getattr(self.cfg, "ad_keys", "single")
        e = rc_embed(self.w["lm_head"], token[n])
        if kind == "single":
            return e[None, :]
        if kind == "two":
            a = self.prec.store(rmsnorm(h, wad["ad.norm"], self.cfg.rms_eps))
            return np.stack([a, e])
        path = []
        while n >= 0:
            path.append(rc_embed(self.w["lm_head"], token[n]))
            n = parent[n]
        return np.stack(path[::-1])

    def draft(self, st: SeqState) -> Candidates:
        c = self.cfg
        depth, token, parent = [0], [st.t0], [-1]
        lp = [np.float32(0.0)]
        state = {0: st.h0}
        out = Candidates(depth=None, token=None, parent=None, lp=None)
        for j in range(1, c.n_spec_heads + 1):
            frontier = [i for i in range(len(depth)) if depth[i] == j - 1]
            wad = self.decoder_weights(j)
            for n in frontier:
                if getattr(c, "regressive", "attention") == "mlp":
                    s = regressive_mlp(state[n], rc_embed(self.w["lm_head"], token[n]), self.w, c.rms_eps,
                                       self.prec)
                else:
                    s = attention_decoder(state[n], self.ad_keys(state[n], n, token, parent, wad), wad,
                                          c.n_heads, c.head_dim, c.rms_eps, self.prec)
                logits = self.head_logits(j - 1, s)
                logp = logits - logsumexp(logits)
                out.row_logits[n] = logits
                out.row_state[n] = s
                for t in topk_ids(logits, c.topk[j - 1]):
                    depth.append(j)
                    token.append(int(t))
                    parent.append(n)
                    lp.append(np.float32(np.float32(lp[n]) + np.float32(logp[t])))
                    state[len(depth) - 1] = s
        out.depth = np.array(depth)
        out.token = np.array(token)
        out.parent = np.array(parent)
        out.lp = np.array(lp, dtype=np.float32)
        return out

    # -- verification (Sec. 2.1, 2.2) ----------------------------------------------------
    def verify(self, st: SeqState, tree: Tree) -> VerifyOut:
        x, kv = self.base.forward_rows(tree.tokens, tree.pos, st.kv, tree.mask)
        logits = self.base.logits(x)
        tau = float(getattr(self.cfg, "temperature", 0.0))
        if tau > 0.0:  # node i's draw: counter (token, i, steps of the sequence, slot)
            target = sampling.sample_tokens(logits, tau, int(getattr(self.cfg, "sample_seed", 0)),
                                            sampling.DOMAIN_VERIFY, st.steps, st.slot, np.arange(len(logits)))
        else:
            target = np.argmax(logits, axis=1)
        return VerifyOut(logits=logits, target=target, x_last=x, kv=kv)

    # -- commit: compaction of the accepted KV entries and the Augmenting Block ------------
    def commit(self, st: SeqState, tree: Tree, ver: VerifyOut, acc: List[int], bonus: int):
        L, A = st.L, len(acc)
        acc = np.asarray(acc)
        st.kv = [(np.concatenate([kp, k[acc]]), np.concatenate([vp, v[acc]]))
                 for (kp, vp), (k, v) in zip(st.kv, ver.kv)]
        causal = np.tril(np.ones((A, A), dtype=bool))
        h, k, v = self.ab_forward(ver.x_last[acc], L + np.arange(A), st.ab_kv, causal)
        if k is not None:
            st.ab_kv = (np.concatenate([st.ab_kv[0], k]), np.concatenate([st.ab_kv[1], v]))
        st.h0 = h[-1].copy()
        st.tokens.extend(int(t) for t in tree.tokens[acc])
        st.t0 = bonus
        st.steps += 1

    def step_tree(self, st: SeqState, tree: Tree):
        """Verify a given tree, accept, commit.  Returns (emitted, acc, verify output)."""
        ver = self.verify(st, tree)
        acc, bonus = accept(tree.tokens, tree.parent, ver.target)
        emitted = [int(tree.tokens[i]) for i in acc[1:]] + [bonus]
        self.commit(st, tree, ver, acc, bonus)
        return emitted, acc, ver

    def step(self, st: SeqState):
        """One speculate-and-verify step.  Returns (emitted, details)."""
        cands = self.draft(st)
        tree = build_tree(cands.depth, cands.token, cands.parent, cands.lp,
                          self.cfg.tree_tokens, st.L)
        emitted, acc, ver = self.step_tree(st, tree)
        return emitted, dict(cands=cands, tree=tree, acc=acc, ver=ver)

    def planted_tree(self, st: SeqState, tokens: Sequence[int], parents: Sequence[int]) -> Tree:
        parent = np.asarray(parents, dtype=np.int64)
        depth = np.zeros(len(parent), dtype=np.int64)
        for i in range(1, len(parent)):
            depth[i] = depth[parent[i]] + 1
        return Tree(tokens=np.asarray(tokens, dtype=np.int64), parent=parent, depth=depth,
                    pos=st.L + depth, mask=tree_mask(parent), src=np.arange(len(parent)))

    def generate(self, prompt: Sequence[int], n_new: int, max_steps: int = 10_000):
        """Speculative greedy generation of at least n_new tokens (first token from prefill)."""
        st = self.prefill(prompt)
        out = [st.t0]
        steps = 0
        while len(out) < n_new and steps < max_steps:
            emitted, _ = self.step(st)
            out.extend(emitted)
            steps += 1
        return out[:n_new], st
