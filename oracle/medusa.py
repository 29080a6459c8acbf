"""Medusa draft on the same target model (oracle side; test infrastructure only).

The paper measures Clover against Medusa decoding (Sec. 1, Sec. 2.3, Sec. 4):
parallel MLP heads that all read the hidden state of the last transformer block,
head j speculating the token j places past the next one, and a token tree that
is the Cartesian product of the heads' candidates.  Sec. 4.4 states that Clover
with the Attention Decoder, the Regressive Connection and the Augmenting Block
removed is that architecture, so the heads here are the Clover head block
without those three parts:

* head j on the last committed token's x_N (the residual after the last base
  layer, the tensor the Augmenting Block would read): r_j = x + SiLU(W1_j x + b1_j),
  logits_j = W_lm RMSNorm_f(r_j) with the target's final norm and shared LM head;
* depth-j children of every depth-(j-1) node are head j's top-k_j tokens (value
  descending, token id ascending), lp(child) = lp(parent) + logp_j(token) in fp32,
  nodes created depth by depth, parents in creation order, children in rank order;
* truncation, verification, greedy acceptance and KV compaction as for Clover;
  there is no Augmenting Block, so after a step h_0 is x_N at the last accepted
  node.

Pins: speculative output equals greedy autoregressive output (the acceptance
rule makes this hold for any draft); every depth-j node's children carry exactly
head j's top-k_j tokens and log-probabilities (Cartesian structure); node
counts.  The head block itself is the Clover head block (same readings), so
its parity status is that of the Clover heads: parity unpinned beyond these.
"""
from typing import Sequence

import numpy as np

from .clover import Candidates, CloverOracle, SeqState, accept, topk_ids  # noqa: F401
from .model import BaseModel, logsumexp


class MedusaOracle(CloverOracle):
    def __init__(self, cfg, weights):
        self.cfg = cfg
        self.w = {k: (v.double().numpy() if hasattr(v, "double") else np.asarray(v, dtype=np.float64))
                  for k, v in weights.items()}
        self.base = BaseModel(cfg, self.w)
        self.prec = self.base.prec
        self.ab = None

    def prefill(self, prompt: Sequence[int]) -> SeqState:
        n = len(prompt)
        causal = np.tril(np.ones((n, n), dtype=bool))
        x, kv = self.base.forward_rows(prompt, np.arange(n), None, causal)
        t0 = int(np.argmax(self.base.logits(x[-1:])[0]))
        return SeqState(tokens=list(prompt), kv=kv, ab_kv=None, h0=x[-1].copy(), t0=t0)

    def draft(self, st: SeqState) -> Candidates:
        c = self.cfg
        H = c.n_spec_heads
        # every head reads the same state: its logits do not depend on the parent node
        head_logits = [self.head_logits(j, st.h0) for j in range(H)]
        head_logp = [lg - logsumexp(lg) for lg in head_logits]
        depth, token, parent = [0], [st.t0], [-1]
        lp = [np.float32(0.0)]
        for j in range(1, H + 1):
            kids = topk_ids(head_logits[j - 1], c.topk[j - 1])
            for n in [i for i in range(len(depth)) if depth[i] == j - 1]:
                for t in kids:
                    depth.append(j)
                    token.append(int(t))
                    parent.append(n)
                    lp.append(np.float32(np.float32(lp[n]) + np.float32(head_logp[j - 1][t])))
        out = Candidates(depth=np.array(depth), token=np.array(token), parent=np.array(parent),
                         lp=np.array(lp, dtype=np.float32))
        out.head_logits = head_logits
        return out

    def commit(self, st: SeqState, tree, ver, acc, bonus: int):
        acc = np.asarray(acc)
        st.kv = [(np.concatenate([kp, k[acc]]), np.concatenate([vp, v[acc]]))
                 for (kp, vp), (k, v) in zip(st.kv, ver.kv)]
        st.h0 = ver.x_last[acc[-1]].copy()
        st.tokens.extend(int(t) for t in tree.tokens[acc])
        st.t0 = bonus
