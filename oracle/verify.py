"""Plain CPU evaluation of one tree-verification step of a Llama-style target.

TEST INFRASTRUCTURE ONLY (see the package docstring).  float64 unless a
``dtype`` argument says otherwise.

What the step computes comes from Section 3.1 of the paper: the target takes
the candidate draft tokens, computes their logits in a single forward pass and
applies the acceptance rule; the accepted tokens start the next round.  The
paper names the target family (LLaMA2-Chat, Vicuna; Section 4 "Experiments")
but not its block structure, mask, positions or cache; the readings used here
are the standard Llama-2 decoder block and:

* node 0 is the root (the pending token), ``parents[0] = -1`` and
  ``0 <= parents[i] < i``;
* node i attends to every committed key plus the keys of its ancestors and
  itself (tree mask);
* node i sits at position ``P + depth(i) - 1`` (root depth 1);
* new keys/values are rounded to the cache dtype before any use;
* greedy acceptance (temperature 0, the exact-match criterion of Section 5
  "Verifying Draft Tokens"): node i is accepted iff its parent is accepted and
  its token equals the parent's argmax; the deepest accepted node wins, lowest
  index on ties; argmax ties go to the lowest token id.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

# ---------------------------------------------------------------------------
# storage conversions


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> exact float64 values."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _to_float(raw, dtype) -> np.ndarray:
    if isinstance(raw, tuple):          # (int8 codes, row scales)
        return dequantize_rows(raw[0], raw[1], dtype)
    if raw.dtype == np.uint16:
        return bf16_to_f64(raw).astype(dtype, copy=False)
    return np.asarray(raw).astype(dtype, copy=False)


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round each value to the nearest bf16 value, ties to even, from the
    value itself (no intermediate fp32 rounding).  Returns the same dtype."""
    x = np.asarray(x)
    src_dtype = x.dtype
    x64 = x.astype(np.float64)
    bits = x64.view(np.uint64)
    # fp64 has 52 stored mantissa bits, bf16 has 7: drop 45 with RNE.
    lsb = (bits >> np.uint64(45)) & np.uint64(1)
    rounded = (bits + np.uint64((1 << 44) - 1) + lsb) & ~np.uint64((1 << 45) - 1)
    out = rounded.view(np.float64)
    # Below the smallest normal (2^-126) bf16 spacing is fixed at 2^-133.
    tiny = np.abs(x64) < 2.0 ** -126
    if np.any(tiny):
        out = np.where(tiny, np.round(x64 * 2.0 ** 133) * 2.0 ** -133, out)
    return out.astype(src_dtype)


def round_cache(x: np.ndarray, kv_dtype: str) -> np.ndarray:
    """Value as stored in a KV cache of ``kv_dtype`` ('bf16', 'f32', 'f64')."""
    if kv_dtype == "bf16":
        return round_to_bf16(x)
    if kv_dtype == "f32":
        return x.astype(np.float32).astype(x.dtype)
    if kv_dtype in ("f64", "none"):
        return x
    raise ValueError(kv_dtype)


# ---------------------------------------------------------------------------
# model container


def dequantize_rows(q: np.ndarray, scale: np.ndarray, dtype=np.float64) -> np.ndarray:
    """Weight-only int8 (the int8 target of Section 4): W[r][c] = scale[r] *
    q[r][c], one scale per output row.  Exact in float64."""
    return np.asarray(q).astype(dtype) * np.asarray(scale).astype(dtype)[:, None]


class OracleModel:
    """Weights as raw arrays (bf16 bits, fp32, or int8 codes with per-row
    scales), matrices ``[out][in]``.

    ``layer_fn(l)`` returns a dict with wq, wk, wv, wo, w_gate, w_up, w_down,
    attn_norm, ffn_norm (and, for int8 matrices, ``<name>_scale``); it is
    called once per layer per forward pass so large models never hold more
    than one layer in float64.  ``lm_head_scale`` marks an int8 lm_head.
    """

    def __init__(self, cfg, layer_fn, embed_rows_fn, lm_head, final_norm, lm_head_scale=None):
        self.cfg = cfg
        self.layer_fn = layer_fn
        self.embed_rows_fn = embed_rows_fn
        self.lm_head = lm_head if lm_head_scale is None else (lm_head, lm_head_scale)
        self.final_norm = final_norm

    def layer(self, l: int, dtype) -> dict:
        raw = self.layer_fn(l)
        return {k: (dequantize_rows(v, raw[k + "_scale"], dtype) if k + "_scale" in raw else _to_float(v, dtype))
                for k, v in raw.items() if not k.endswith("_scale")}

    def embed(self, ids, dtype) -> np.ndarray:
        return _to_float(self.embed_rows_fn(np.asarray(ids)), dtype)


def empty_kv(cfg, dtype=np.float64):
    h, hd = cfg.n_heads, cfg.head_dim
    return [(np.zeros((h, 0, hd), dtype), np.zeros((h, 0, hd), dtype))
            for _ in range(cfg.n_layers)]


def kv_from_raw(layers, dtype=np.float64):
    """Cached K/V given as stored arrays ``[H][P][hd]`` per layer -> floats."""
    return [(_to_float(k, dtype), _to_float(v, dtype)) for k, v in layers]


# ---------------------------------------------------------------------------
# tree


@dataclass
class TreeInfo:
    parents: np.ndarray      # int [M]
    depth: np.ndarray        # int [M], root = 1
    ancestors: list          # list of sorted int arrays: ancestors of i and i itself


def tree_info(parents) -> TreeInfo:
    """Validate a draft tree given by parent indices and derive depths and
    ancestor sets.  Node 0 is the root (parent -1); node i >= 1 has a parent
    with a smaller index."""
    parents = np.asarray(parents, dtype=np.int64)
    m = len(parents)
    if m < 1:
        raise ValueError("empty tree")
    if parents[0] != -1:
        raise ValueError("node 0 must be the root (parent -1)")
    depth = np.zeros(m, dtype=np.int64)
    anc = [None] * m
    depth[0] = 1
    anc[0] = np.array([0])
    for i in range(1, m):
        p = int(parents[i])
        if not 0 <= p < i:
            raise ValueError("parent of node %d must be in [0, %d)" % (i, i))
        depth[i] = depth[p] + 1
        anc[i] = np.append(anc[p], i)
    return TreeInfo(parents, depth, anc)


# ---------------------------------------------------------------------------
# building blocks


def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def rope(x: np.ndarray, pos: np.ndarray, base: float) -> np.ndarray:
    """Rotary embedding, rotate-half pairing: element j pairs with j + hd/2
    and turns by angle pos * base^(-2j/hd).  x: [M][H][hd], pos: [M]."""
    hd = x.shape[-1]
    half = hd // 2
    j = np.arange(half, dtype=np.float64)
    theta = base ** (-2.0 * j / hd)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * theta[None, :]       # [M][half]
    c = np.cos(ang).astype(x.dtype)[:, None, :]
    s = np.sin(ang).astype(x.dtype)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def attention_node(q, k_ctx, v_ctx, k_tree, v_tree):
    """Softmax attention of one query per head over the committed keys and the
    query's visible tree keys.  q: [H][hd]; k_ctx, v_ctx: [H][P][hd];
    k_tree, v_tree: [H][n][hd].  Scores are scaled by 1/sqrt(hd)."""
    hd = q.shape[-1]
    scale = 1.0 / np.sqrt(hd)
    s_ctx = np.einsum("hpd,hd->hp", k_ctx, q) * scale
    s_tree = np.einsum("hnd,hd->hn", k_tree, q) * scale
    s = np.concatenate([s_ctx, s_tree], axis=1)
    s = s - np.max(s, axis=1, keepdims=True)
    w = np.exp(s)
    w = w / np.sum(w, axis=1, keepdims=True)
    p = k_ctx.shape[1]
    return (np.einsum("hp,hpd->hd", w[:, :p], v_ctx)
            + np.einsum("hn,hnd->hd", w[:, p:], v_tree))


def silu(z):
    return z / (1.0 + np.exp(-z))


# ---------------------------------------------------------------------------
# one forward pass over a tree


def forward_tree(model: OracleModel, kv, tokens, parents, dtype=np.float64, kv_dtype=None, x0=None):
    """Logits of every tree node after one pass of the decoder stack.

    kv: per layer (K, V) floats [H][P][hd] holding the committed cache.
    x0: the stack's input rows [M][d] (default: the tokens' embeddings).
    Returns dict(logits [M][V], new_k, new_v: per layer [M][H][hd] rounded to
    the cache dtype, tree: TreeInfo, pos, hidden: the residual stream after
    the last block [M][d])."""
    cfg = model.cfg
    kv_dtype = kv_dtype or cfg.kv_dtype
    info = tree_info(parents)
    tokens = np.asarray(tokens, dtype=np.int64)
    m = len(tokens)
    if len(info.parents) != m:
        raise ValueError("tokens and parents differ in length")
    if np.any(tokens < 0) or np.any(tokens >= cfg.vocab):
        raise ValueError("token id out of range")
    p_ctx = kv[0][0].shape[1]
    pos = p_ctx + info.depth - 1
    h, hd, d = cfg.n_heads, cfg.head_dim, cfg.d_model

    x = model.embed(tokens, dtype) if x0 is None else np.asarray(x0, dtype=dtype)   # [M][d]
    new_k, new_v = [], []
    for l in range(cfg.n_layers):
        w = model.layer(l, dtype)
        k_ctx, v_ctx = kv[l]
        k_ctx = k_ctx.astype(dtype, copy=False)
        v_ctx = v_ctx.astype(dtype, copy=False)
        u = rmsnorm(x, w["attn_norm"], cfg.rms_eps)
        q = (u @ w["wq"].T).reshape(m, h, hd)
        k = (u @ w["wk"].T).reshape(m, h, hd)
        v = (u @ w["wv"].T).reshape(m, h, hd)
        q = rope(q, pos, cfg.rope_base)
        k = round_cache(rope(k, pos, cfg.rope_base), kv_dtype)
        v = round_cache(v, kv_dtype)
        new_k.append(k)
        new_v.append(v)
        o = np.empty((m, h, hd), dtype=dtype)
        for i in range(m):
            a = info.ancestors[i]
            kt = np.transpose(k[a], (1, 0, 2))               # [H][n][hd]
            vt = np.transpose(v[a], (1, 0, 2))
            o[i] = attention_node(q[i], k_ctx, v_ctx, kt, vt)
        x = x + o.reshape(m, d) @ w["wo"].T
        u = rmsnorm(x, w["ffn_norm"], cfg.rms_eps)
        x = x + (silu(u @ w["w_gate"].T) * (u @ w["w_up"].T)) @ w["w_down"].T
        del w
    u = rmsnorm(x, _to_float(model.final_norm, dtype), cfg.rms_eps)
    logits = u @ _to_float(model.lm_head, dtype).T
    return dict(logits=logits, new_k=new_k, new_v=new_v, tree=info, pos=pos, hidden=x)


# ---------------------------------------------------------------------------
# acceptance and commit


def argmax_lowest(z: np.ndarray) -> np.ndarray:
    """Row-wise argmax taken on the fp32 values; ties go to the lowest id."""
    z32 = np.asarray(z).astype(np.float32)
    return np.argmax(z32, axis=-1).astype(np.int64)


def greedy_accept(tokens, parents, amax):
    """Greedy acceptance on a tree: node 0 is always accepted; node i is
    accepted when its parent is and its token equals the parent's argmax.
    The deepest accepted node wins (lowest index on ties).  Returns
    (accept_len, path root->best, bonus = argmax at best)."""
    info = tree_info(parents)
    tokens = np.asarray(tokens)
    m = len(tokens)
    ok = np.zeros(m, dtype=bool)
    ok[0] = True
    for i in range(1, m):
        p = info.parents[i]
        ok[i] = ok[p] and int(tokens[i]) == int(amax[p])
    best = 0
    for i in range(m):
        if ok[i] and info.depth[i] > info.depth[best]:
            best = i
    path = info.ancestors[best].copy()
    return int(info.depth[best]), path, int(amax[best])


def softmax_t(z: np.ndarray, temperature: float) -> np.ndarray:
    """Target distribution at temperature T > 0: softmax(z / T), float64."""
    z = np.asarray(z, dtype=np.float64) / float(temperature)
    e = np.exp(z - z.max())
    return e / e.sum()


def sample_inverse_cdf(p: np.ndarray, u: float) -> int:
    """The smallest token id v with cumsum(p)[v] > u * sum(p) (u in [0, 1))."""
    c = np.cumsum(np.asarray(p, dtype=np.float64))
    return int(np.searchsorted(c, u * c[-1], side="right"))


def accept_sampled(logits, tokens, parents, q, temperature, u_accept, u_bonus, trace=None):
    """Stochastic tree verification (temperature T > 0): recursive rejection
    sampling over each accepted node's children, the speculative sampling rule
    the paper applies (Section 3.1) and credits with preserving the target's
    output distribution (Section 5, "Verifying Draft Tokens").

    Reading used here (the paper gives no formula): the children of node u are
    independent draws from the draft distribution q[u]; the target
    distribution at u is p = softmax(logits[u] / T).  Starting at the root,
    the children of the current node are tried in index order; child c (token
    t) is accepted when u_accept[c] * q[u][t] < p[t]; a rejected child
    replaces p by the residual max(p - q[u], 0), renormalised.  When a child
    is accepted it becomes the current node; when none is, the bonus token is
    drawn from the current p by inverse CDF with u_bonus[current].
    Returns (accept_len, path root->last, bonus).

    ``trace``, when a list, receives every decision the walk takes, for tests
    that need the margin of a decision: ("accept", child, u*q[t], p[t], mass)
    per tried child and ("bonus", p, u, mass) at the end, where mass is the
    product of the residual totals since p was last a softmax."""
    info = tree_info(parents)
    tokens = np.asarray(tokens)
    m = len(tokens)
    children = [[c for c in range(m) if info.parents[c] == u] for u in range(m)]
    cur, path = 0, [0]
    while True:
        p = softmax_t(logits[cur], temperature)
        qu = np.asarray(q[cur], dtype=np.float64)
        moved, mass = False, 1.0
        for c in children[cur]:
            t = int(tokens[c])
            if trace is not None:
                trace.append(("accept", c, float(u_accept[c]) * qu[t], p[t], mass))
            if float(u_accept[c]) * qu[t] < p[t]:
                path.append(c)
                cur = c
                moved = True
                break
            r = np.maximum(p - qu, 0.0)
            s = r.sum()
            if s > 0:
                p = r / s
                mass *= s
        if not moved:
            if trace is not None:
                trace.append(("bonus", p, float(u_bonus[cur]), mass))
            return len(path), np.array(path), sample_inverse_cdf(p, float(u_bonus[cur]))


def verify_step(model, kv, tokens, parents, dtype=np.float64, kv_dtype=None):
    """One verification step: forward pass + argmax + greedy acceptance."""
    out = forward_tree(model, kv, tokens, parents, dtype=dtype, kv_dtype=kv_dtype)
    amax = argmax_lowest(out["logits"])
    n, path, bonus = greedy_accept(tokens, parents, amax)
    out.update(argmax=amax, accept_len=n, path=path, bonus=bonus)
    return out


def commit(kv, new_k, new_v, path):
    """Append the accepted nodes' keys/values (in path order) to the cache."""
    path = np.asarray(path)
    out = []
    for l, (k, v) in enumerate(kv):
        kk = np.transpose(new_k[l][path], (1, 0, 2))
        vv = np.transpose(new_v[l][path], (1, 0, 2))
        out.append((np.concatenate([k, kk.astype(k.dtype)], axis=1),
                    np.concatenate([v, vv.astype(v.dtype)], axis=1)))
    return out


def prefill(model, tokens, kv=None, dtype=np.float64, kv_dtype=None):
    """Run ``tokens`` as one chain through the stack and commit all of them.
    Returns (kv, logits of the chain)."""
    kv = kv if kv is not None else empty_kv(model.cfg, dtype)
    n = len(tokens)
    parents = np.arange(-1, n - 1)
    out = forward_tree(model, kv, tokens, parents, dtype=dtype, kv_dtype=kv_dtype)
    return commit(kv, out["new_k"], out["new_v"], np.arange(n)), out["logits"]


def greedy_decode(model, kv, root, n_tokens, dtype=np.float64, kv_dtype=None):
    """Plain greedy decoding, one token per pass: returns the ``n_tokens``
    tokens emitted starting with ``root`` and the final cache."""
    seq = [int(root)]
    while len(seq) < n_tokens + 1:
        out = forward_tree(model, kv, [seq[-1]], [-1], dtype=dtype, kv_dtype=kv_dtype)
        kv = commit(kv, out["new_k"], out["new_v"], [0])
        seq.append(int(argmax_lowest(out["logits"])[0]))
    return seq[:n_tokens], kv
