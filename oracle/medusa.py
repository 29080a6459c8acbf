"""Medusa draft on the same target model (oracle side; test infrastructure only).

The paper measures Clover against Medusa decoding (Sec. 1, Sec. 2.3, Sec. 4):
parallel MLP heads that all read the hidden state of the last transformer block,
head j speculating the token j places past the next one, and a token tree that
is the Cartesian product of the heads' candidates.  Sec. 4.3 states that Clover
with the Attention Decoder, the Regressive Connection and the Augmenting Block
removed is that architecture, so the heads here are the Clover head block
without the Attention Decoder and the Regressive Connection:

* every head reads the drafting state h_0 of the last committed token: x_N (the
  residual after the last base layer) when there is no Augmenting Block -- the
  Medusa baseline -- or the Augmenting Block's output when one is configured
  (Clover without Attention Decoder and Regressive Connection, Sec. 4.3);
* head j: r_j = h + SiLU(W1_j h + b1_j), logits_j = W_lm RMSNorm_f(r_j) with the
  target's final norm and shared LM head;
* depth-j children of every depth-(j-1) node are head j's top-k_j tokens (value
  descending, token id ascending), lp(child) = lp(parent) + logp_j(token) in fp32,
  nodes created depth by depth, parents in creation order, children in rank order;
* truncation, verification, greedy acceptance, KV compaction and the Augmenting
  Block's update of h_0 are those of the Clover oracle.

Pins: speculative output equals greedy autoregressive output (the acceptance
rule makes this hold for any draft); every depth-j node's children carry exactly
head j's top-k_j tokens and log-probabilities (Cartesian structure); node
counts; Clover with its output projections zeroed drafts the same trees.  The
head block itself is the Clover head block (same readings), pinned by the identity
heads reduction and by the path-sum closed form of the Clover oracle (its head MLP and
shared LM head are the ones used here).
"""
import numpy as np

from .clover import Candidates, CloverOracle, SeqState, head_mlp, topk_ids
from .model import logsumexp, rmsnorm


class MedusaOracle(CloverOracle):
    def head_logits(self, j: int, s: np.ndarray) -> np.ndarray:
        """Head j's MLP on the state, the shared final norm, then the shared LM head or, with
        per-head LM heads (the original Medusa, Sec. 3.4), head j's own."""
        if getattr(self.cfg, "medusa_lm", "shared") != "per_head":
            return super().head_logits(j, s)
        r = head_mlp(s, self.w[f"head{j}.w1"], self.w[f"head{j}.b1"], self.prec)
        return self.prec.store(rmsnorm(r, self.w["final_norm"], self.cfg.rms_eps)) @ self.w[f"head{j}.lm"].T

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
