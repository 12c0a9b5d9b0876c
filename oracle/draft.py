"""Plain CPU evaluation of the draft side: the Dynamic Gated Fusion front end
(Section 3.2), the draft's block stack (Section 3.3) and the draft-tree
construction of Section 3.1.

TEST INFRASTRUCTURE ONLY (see the package docstring).  float64.

Readings (the paper gives the steps in words, no formulas):

* DGF: h1 = W_h f (f the hidden state fed to the draft), h2 = W_e e (e the
  token embedding); a linear layer on the concatenation [h1 || h2] followed
  by a sigmoid gives g; the fused input is g * h1 + (1 - g) * h2 (the
  weighted sum).  No biases.
* The draft: DGF, then M Llama blocks with the same tree mask and positions
  as the target (its own KV cache), then its final RMSNorm and the target's
  lm_head.  Node u (token t_u, parent p) takes f = the draft's output
  feature at p (the residual stream after its last block) and e = E[t_u];
  the root takes the hidden state handed over with the accepted tokens.  The
  distribution of u's children is softmax of u's logits.
* Tree construction: the score of a node is the product of the draft
  probabilities along its path from the root (the root scores 1).  Each round
  the `width` highest-scoring nodes of the newest layer are expanded, each by
  its `width` most probable tokens (probability order, lower id first on
  ties), for `depth` rounds; then every node but the root is ranked by score
  (earlier-created first on ties) and the best n_tree - 1 join the root.
  Scores never increase along a path and a parent is created before its
  children, so the selection is ancestor-closed; the output lists the
  selected nodes in creation order (a topological order).
"""
from __future__ import annotations

import numpy as np

from .verify import OracleModel, _to_float, forward_tree, tree_info


def sigmoid(z):
    return 0.5 * (1.0 + np.tanh(0.5 * np.asarray(z)))


def dgf(feat, emb, w_hidden, w_embed, w_gate):
    """Dynamic Gated Fusion (Section 3.2) of hidden states ``feat`` [n][d] and
    token embeddings ``emb`` [n][d]; weights [d][d], [d][d], [d][2d]."""
    h1 = feat @ w_hidden.T
    h2 = emb @ w_embed.T
    g = sigmoid(np.concatenate([h1, h2], axis=-1) @ w_gate.T)
    return g * h1 + (1.0 - g) * h2


class DraftModel:
    """The draft's blocks as an OracleModel (its embed and lm_head are the
    target's) plus the DGF weights (raw arrays, bf16 bits or fp32)."""

    def __init__(self, blocks: OracleModel, w_hidden, w_embed, w_gate):
        self.blocks = blocks
        self.w_hidden, self.w_embed, self.w_gate = w_hidden, w_embed, w_gate

    def forward(self, kv, tokens, parents, feat_in):
        """Logits and output features of every node of a draft tree."""
        emb = self.blocks.embed(np.asarray(tokens), np.float64)
        x0 = dgf(np.asarray(feat_in, dtype=np.float64), emb, _to_float(self.w_hidden, np.float64),
                 _to_float(self.w_embed, np.float64), _to_float(self.w_gate, np.float64))
        out = forward_tree(self.blocks, kv, tokens, parents, x0=x0)
        return out["logits"], out["hidden"]


def _softmax(z):
    e = np.exp(z - z.max())
    return e / e.sum()


def build_tree(forward_fn, root_token, root_feature, depth, width, n_tree, trace=None):
    """Draft-tree construction (Section 3.1), literally: every generated node
    is kept until the final ranking.

    forward_fn(tokens, parents, feat_in) -> (logits [n][V], features [n][d])
    runs the draft over an ancestor-closed node list (parents index into it).
    Returns (tokens [n], parents [n], scores [n]) of the selected tree.
    ``trace``, when a list, receives each ranking decision as
    (kind, score of the last one taken, score of the first one left out)."""
    tok, par, score = [int(root_token)], [-1], [1.0]
    feat = {}
    frontier = [0]
    for _ in range(depth):
        order = sorted(frontier, key=lambda i: (-score[i], i))
        chosen = order[:width]
        if trace is not None and len(order) > width:
            trace.append(("expand", score[order[width - 1]], score[order[width]]))
        # the draft's output at the chosen nodes: one pass over them and
        # their ancestors, each fed its parent's feature
        sub = sorted({a for u in chosen for a in tree_info(par[: u + 1]).ancestors[u]})
        pos = {u: r for r, u in enumerate(sub)}
        f_in = np.stack([np.asarray(root_feature, dtype=np.float64) if u == 0 else feat[par[u]] for u in sub])
        logits, f_out = forward_fn([tok[u] for u in sub], [pos[par[u]] if u else -1 for u in sub], f_in)
        for u in sub:
            feat[u] = f_out[pos[u]]
        new = []
        for u in chosen:
            p = _softmax(np.asarray(logits[pos[u]], dtype=np.float64))
            top = sorted(range(len(p)), key=lambda t: (-p[t], t))
            if trace is not None and len(p) > width:
                trace.append(("child", p[top[width - 1]], p[top[width]]))
            for t in top[:width]:
                tok.append(t)
                par.append(u)
                score.append(score[u] * p[t])
                new.append(len(tok) - 1)
        frontier = new
    ranked = sorted(range(1, len(tok)), key=lambda i: (-score[i], i))
    if trace is not None and len(ranked) > n_tree - 1:
        trace.append(("select", score[ranked[n_tree - 2]], score[ranked[n_tree - 1]]))
    keep = sorted([0] + ranked[: n_tree - 1])
    index = {u: r for r, u in enumerate(keep)}
    return (np.array([tok[u] for u in keep]), np.array([index[par[u]] if u else -1 for u in keep]),
            np.array([score[u] for u in keep]))
