"""Pins of the CPU oracle against things other than itself (no GPU).

Each test checks the oracle against a fact the method or mathematics fixes:
hand-derived closed forms and worked examples (tests/golden/), an independent
Llama implementation, a library attention routine, and the invariants of tree
verification (chain == sequential decoding, tree == per-path decoding,
acceptance == brute force, verify+commit == greedy decoding).
"""
import math
import os

import numpy as np
import pytest
import torch

import oracle
import synth
from oracle import verify as ov
from tests.helpers import Weights, all_parent_arrays, small_cfg

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------------------
# input generator (not the method, but both sides trust it)

def test_generator_matches_python_restatement():
    got = synth.u64(7, 1234, 5, start=9)
    want = [synth.u64_py(7, 1234, 9 + i) for i in range(5)]
    assert [int(v) for v in got] == want
    a = synth.normal(5, 9, 1001, 0.02, "bf16")
    b = synth.normal(5, 9, 500, 0.02, "bf16", start=301)
    assert np.array_equal(a[301:801], b)
    f = synth.normal(5, 9, 200000, 1.0, "f32")
    assert abs(f.mean()) < 0.01 and abs(f.std() - 1.0) < 0.01


# ---------------------------------------------------------------------------
# storage rounding

def _golden_lines(name):
    with open(os.path.join(GOLDEN, name)) as fh:
        return [ln.strip() for ln in fh if ln.strip() and not ln.startswith("#")]


def test_bf16_rounding_golden():
    for ln in _golden_lines("bf16_rounding.txt"):
        lhs, rhs = ln.split("->")
        x = float(lhs)
        want = int(rhs, 16)
        got = ov.round_to_bf16(np.array([x]))[0]
        bits = (np.array([got], dtype=np.float32).view(np.uint32)[0] >> 16)
        assert int(bits) == want, (x, hex(int(bits)), hex(want))
        # the rounded value must itself be a bf16 value
        assert float(got) == float(ov.bf16_to_f64(np.array([want], dtype=np.uint16))[0])


def test_bf16_rounding_matches_torch_on_fp32_values():
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(100000) * np.exp(rng.uniform(-20, 20, 100000))).astype(np.float32)
    want = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = ov.round_to_bf16(x.astype(np.float64))
    assert np.array_equal(got, want)


# ---------------------------------------------------------------------------
# building blocks

def test_rope_golden_closed_form():
    for ln in _golden_lines("rope_hd4_base10000.txt"):
        lhs, rhs = ln.split("->")
        vals = lhs.split()
        pos = int(vals[0])
        x = np.array([float(v) for v in vals[1:]]).reshape(1, 1, 4)
        want = np.array([float(v) for v in rhs.split()])
        got = ov.rope(x, np.array([pos]), 10000.0)[0, 0]
        np.testing.assert_allclose(got, want, rtol=0, atol=1e-14)


def test_rope_properties():
    rng = np.random.default_rng(1)
    hd = 16
    q = rng.standard_normal((1, 3, hd))
    k = rng.standard_normal((1, 3, hd))
    # norm preserving
    for p in (0, 5, 1000):
        np.testing.assert_allclose(np.linalg.norm(ov.rope(q, np.array([p]), 1e4), axis=-1),
                                   np.linalg.norm(q, axis=-1), rtol=1e-13)
    np.testing.assert_array_equal(ov.rope(q, np.array([0]), 1e4), q)
    # <R_m q, R_n k> depends only on m - n
    def dot(m, n):
        return np.sum(ov.rope(q, np.array([m]), 1e4) * ov.rope(k, np.array([n]), 1e4), axis=-1)
    np.testing.assert_allclose(dot(7, 3), dot(104, 100), rtol=1e-10)
    assert not np.allclose(dot(7, 3), dot(7, 4))


def test_rmsnorm_closed_form():
    for c in (3.0, -0.25, 1e-4):
        x = np.full((1, 32), c)
        g = np.linspace(0.5, 2.0, 32)
        got = ov.rmsnorm(x, g, 1e-6)
        want = c / math.sqrt(c * c + 1e-6) * g
        np.testing.assert_allclose(got[0], want, rtol=1e-14)
    x = np.array([[3.0, 4.0]])                    # mean square 12.5
    np.testing.assert_allclose(ov.rmsnorm(x, np.ones(2), 0.0), x / math.sqrt(12.5), rtol=1e-15)


def test_attention_matches_sdpa_with_tree_mask():
    rng = np.random.default_rng(2)
    h, hd, p, m = 3, 16, 9, 7
    parents = np.array([-1, 0, 1, 1, 0, 4, 3])
    info = ov.tree_info(parents)
    q = rng.standard_normal((m, h, hd))
    k_ctx, v_ctx = rng.standard_normal((h, p, hd)), rng.standard_normal((h, p, hd))
    k_new, v_new = rng.standard_normal((m, h, hd)), rng.standard_normal((m, h, hd))
    mask = np.zeros((m, p + m), dtype=bool)
    mask[:, :p] = True
    for i in range(m):
        mask[i, p + info.ancestors[i]] = True
    keys = np.concatenate([k_ctx, np.transpose(k_new, (1, 0, 2))], axis=1)    # [H][P+M][hd]
    vals = np.concatenate([v_ctx, np.transpose(v_new, (1, 0, 2))], axis=1)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(np.transpose(q, (1, 0, 2))), torch.from_numpy(keys),
        torch.from_numpy(vals), attn_mask=torch.from_numpy(mask)).numpy()      # [H][M][hd]
    for i in range(m):
        a = info.ancestors[i]
        got = ov.attention_node(q[i], k_ctx, v_ctx, np.transpose(k_new[a], (1, 0, 2)),
                                np.transpose(v_new[a], (1, 0, 2)))
        np.testing.assert_allclose(got, ref[:, i], rtol=1e-12, atol=1e-13)


def test_attention_special_cases():
    rng = np.random.default_rng(3)
    h, hd = 2, 8
    q = rng.standard_normal((h, hd))
    empty = np.zeros((h, 0, hd))
    k1, v1 = rng.standard_normal((h, 1, hd)), rng.standard_normal((h, 1, hd))
    np.testing.assert_allclose(ov.attention_node(q, empty, empty, k1, v1), v1[:, 0], rtol=1e-14)
    kk = np.repeat(k1, 5, axis=1)
    vv = rng.standard_normal((h, 5, hd))
    np.testing.assert_allclose(ov.attention_node(q, kk, vv, empty, empty), vv.mean(axis=1),
                               rtol=1e-13)


# ---------------------------------------------------------------------------
# independent Llama implementation

def _hf_model(w: Weights):
    transformers = pytest.importorskip("transformers")
    cfg = w.cfg
    hcfg = transformers.LlamaConfig(
        vocab_size=cfg.vocab, hidden_size=cfg.d_model, intermediate_size=cfg.d_ffn,
        num_hidden_layers=cfg.n_layers, num_attention_heads=cfg.n_heads,
        num_key_value_heads=cfg.n_heads, head_dim=cfg.head_dim, rms_norm_eps=cfg.rms_eps,
        rope_theta=cfg.rope_base, tie_word_embeddings=False, attention_bias=False,
        mlp_bias=False, max_position_embeddings=4096, attn_implementation="eager")
    hf = transformers.LlamaForCausalLM(hcfg).double().eval()
    names = dict(wq="self_attn.q_proj", wk="self_attn.k_proj", wv="self_attn.v_proj",
                 wo="self_attn.o_proj", w_gate="mlp.gate_proj", w_up="mlp.up_proj",
                 w_down="mlp.down_proj", attn_norm="input_layernorm",
                 ffn_norm="post_attention_layernorm")
    sd = {"model.embed_tokens.weight": w.embed, "lm_head.weight": w.lm_head,
          "model.norm.weight": w.final_norm}
    for l in range(cfg.n_layers):
        for k, n in names.items():
            sd["model.layers.%d.%s.weight" % (l, n)] = w.layers[l][k]
    hf.load_state_dict({k: torch.tensor(np.asarray(v, dtype=np.float64)) for k, v in sd.items()},
                       strict=True)
    return hf


def _hf_mismatch():
    """Largest logit difference (relative to the logit scale) between the oracle
    and transformers' LlamaForCausalLM with the same weights, over a prefill
    and a tree step with a 4-D tree mask and depth-based position ids."""
    cfg = small_cfg()
    w = Weights(cfg, seed=11)
    om = w.oracle()
    hf = _hf_model(w)
    p = 12
    prompt = synth.prompt(2, p, cfg.vocab)
    with torch.no_grad():
        out = hf(input_ids=torch.tensor(prompt[None].astype(np.int64)), use_cache=True)
    kv, logits = ov.prefill(om, prompt, kv_dtype="f64")
    scale = np.abs(logits).max()
    err = np.abs(out.logits[0].numpy() - logits).max() / scale
    # committed keys (after rotation) and values
    cache = out.past_key_values
    for l in range(cfg.n_layers):
        lay = cache.layers[l]
        err = max(err, np.abs(lay.keys[0].numpy() - kv[l][0]).max() / np.abs(kv[l][0]).max())
        err = max(err, np.abs(lay.values[0].numpy() - kv[l][1]).max() / np.abs(kv[l][1]).max())

    toks, par = synth.random_tree(3, 9, 4, cfg.vocab)
    m = len(toks)
    # mask and positions from the parents array, walked here (not by the oracle)
    mask = torch.full((1, 1, m, p + m), float("-inf"), dtype=torch.float64)
    mask[..., :p] = 0.0
    pos = torch.zeros(1, m, dtype=torch.int64)
    for i in range(m):
        j, depth = i, 0
        while j >= 0:
            mask[0, 0, i, p + j] = 0.0
            j, depth = int(par[j]), depth + 1
        pos[0, i] = p + depth - 1
    with torch.no_grad():
        o2 = hf(input_ids=torch.tensor(toks[None].astype(np.int64)), position_ids=pos,
                attention_mask=mask, past_key_values=cache, use_cache=True)
    ft = ov.forward_tree(om, kv, toks, par, kv_dtype="f64")
    return max(err, np.abs(o2.logits[0].numpy() - ft["logits"]).max() / scale)


def test_forward_matches_transformers_llama():
    """transformers evaluates RMSNorm and softmax in float32 internally, so the
    agreement is ~1e-6 relative, not float64-tight."""
    assert _hf_mismatch() < 2e-5


def _rope_interleaved(x, pos, base):
    hd = x.shape[-1]
    j = np.arange(hd // 2, dtype=np.float64)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * (base ** (-2.0 * j / hd))[None, :]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    out = np.empty_like(x)
    out[..., 0::2] = x[..., 0::2] * c - x[..., 1::2] * s
    out[..., 1::2] = x[..., 1::2] * c + x[..., 0::2] * s
    return out


def _attention_unscaled(q, k_ctx, v_ctx, k_tree, v_tree):
    hd = q.shape[-1]
    return ov.__dict__["_orig_attention"](q * np.sqrt(hd), k_ctx, v_ctx, k_tree, v_tree)


def _tree_info_index_positions(parents):
    info = ov.__dict__["_orig_tree_info"](parents)
    info.depth = np.arange(1, len(info.depth) + 1)
    return info


def _tree_info_sees_siblings(parents):
    info = ov.__dict__["_orig_tree_info"](parents)
    info.ancestors = [np.arange(i + 1) for i in range(len(info.depth))]
    return info


def _layer_attn_ffn_swapped(self, l, dtype):
    w = ov.__dict__["_orig_layer"](self, l, dtype)
    w["attn_norm"], w["ffn_norm"] = w["ffn_norm"], w["attn_norm"]
    return w


def _layer_norms_of_layer0(self, l, dtype):
    w = ov.__dict__["_orig_layer"](self, l, dtype)
    w0 = ov.__dict__["_orig_layer"](self, 0, dtype)
    w["attn_norm"], w["ffn_norm"] = w0["attn_norm"], w0["ffn_norm"]
    return w


class _FinalNormTakesLastLayerGain:
    """rmsnorm whose last call of every pass (the final norm: a pass makes
    2 n_layers + 1 calls) uses the gain of the call before it (the last
    layer's FFN norm)."""

    def __init__(self, n_layers):
        self.per_pass, self.calls, self.prev = 2 * n_layers + 1, 0, None

    def __call__(self, x, g, eps):
        self.calls += 1
        if self.calls % self.per_pass == 0:
            g = self.prev
        self.prev = g
        return ov.__dict__["_orig_rmsnorm"](x, g, eps)


_MUTANTS = {
    "gain_ignored": ("rmsnorm", lambda x, g, eps: ov.__dict__["_orig_rmsnorm"](x, np.ones_like(g), eps)),
    "attn_ffn_gains_swapped": ("OracleModel.layer", _layer_attn_ffn_swapped),
    "every_layer_takes_layer0_gains": ("OracleModel.layer", _layer_norms_of_layer0),
    "final_norm_takes_last_layer_gain": ("rmsnorm", _FinalNormTakesLastLayerGain(small_cfg().n_layers)),
    "rope_interleaved": ("rope", _rope_interleaved),
    "attention_unscaled": ("attention_node", _attention_unscaled),
    "positions_by_index": ("tree_info", _tree_info_index_positions),
    "mask_sees_all_earlier_nodes": ("tree_info", _tree_info_sees_siblings),
    "silu_sign": ("silu", lambda z: z / (1.0 + np.exp(z))),
    "rmsnorm_sum_not_mean": ("rmsnorm", lambda x, g, eps: x / np.sqrt(np.sum(x * x, -1, keepdims=True) + eps) * g),
}


@pytest.mark.parametrize("name", sorted(_MUTANTS))
def test_planted_oracle_mistakes_are_caught(name, monkeypatch):
    """A plausible mistake planted in the oracle must break the pin above."""
    attr, fn = _MUTANTS[name]
    monkeypatch.setitem(ov.__dict__, "_orig_attention", ov.attention_node)
    monkeypatch.setitem(ov.__dict__, "_orig_tree_info", ov.tree_info)
    monkeypatch.setitem(ov.__dict__, "_orig_rmsnorm", ov.rmsnorm)
    monkeypatch.setitem(ov.__dict__, "_orig_layer", ov.OracleModel.layer)
    if attr == "OracleModel.layer":
        monkeypatch.setattr(ov.OracleModel, "layer", fn)
    else:
        monkeypatch.setattr(ov, attr, fn)
    assert _hf_mismatch() > 1e-3


# ---------------------------------------------------------------------------
# invariants of tree verification

def _kv_ctx(om, seed, p, kv_dtype):
    prompt = synth.prompt(seed, p, om.cfg.vocab)
    kv, _ = ov.prefill(om, prompt, kv_dtype=kv_dtype)
    return kv


@pytest.mark.parametrize("kv_dtype", ["f64", "bf16"])
def test_chain_equals_sequential(kv_dtype):
    cfg = small_cfg()
    om = Weights(cfg, 21).oracle()
    kv = _kv_ctx(om, 22, 10, kv_dtype)
    toks = synth.prompt(23, 6, cfg.vocab)
    par = np.arange(-1, 5)
    one = ov.forward_tree(om, kv, toks, par, kv_dtype=kv_dtype)
    kv_s = kv
    for i, t in enumerate(toks):
        step = ov.forward_tree(om, kv_s, [t], [-1], kv_dtype=kv_dtype)
        np.testing.assert_allclose(step["logits"][0], one["logits"][i], rtol=1e-9, atol=1e-12)
        kv_s = ov.commit(kv_s, step["new_k"], step["new_v"], [0])
    assert np.array_equal(ov.argmax_lowest(one["logits"]),
                          ov.argmax_lowest(np.stack([one["logits"][i] for i in range(6)])))


@pytest.mark.parametrize("seed", [31, 32, 33])
def test_tree_equals_per_path(seed):
    cfg = small_cfg()
    om = Weights(cfg, seed).oracle()
    kv = _kv_ctx(om, seed + 1, 7, "bf16")
    toks, par = synth.random_tree(seed + 2, 12, 5, cfg.vocab)
    full = ov.forward_tree(om, kv, toks, par)
    info = full["tree"]
    for i in range(len(toks)):
        a = info.ancestors[i]
        chain = ov.forward_tree(om, kv, toks[a], np.arange(-1, len(a) - 1))
        np.testing.assert_allclose(chain["logits"][-1], full["logits"][i], rtol=1e-9, atol=1e-12)
        for l in range(cfg.n_layers):
            np.testing.assert_array_equal(chain["new_k"][l][-1], full["new_k"][l][i])


def _brute_force_accept(om, kv, toks, par):
    """Acceptance from sequential decoding alone: node i is accepted when every
    token on its root path equals the greedy choice after the tokens before it."""
    info = ov.tree_info(par)
    m = len(toks)
    greedy_after = {}

    def greedy(prefix):
        if prefix not in greedy_after:
            kv_p, st = kv, None
            for t in prefix:
                st = ov.forward_tree(om, kv_p, [t], [-1])
                kv_p = ov.commit(kv_p, st["new_k"], st["new_v"], [0])
            greedy_after[prefix] = int(ov.argmax_lowest(st["logits"])[0])
        return greedy_after[prefix]

    ok = []
    for i in range(m):
        path = [int(toks[j]) for j in info.ancestors[i]]
        ok.append(all(path[k + 1] == greedy(tuple(path[:k + 1])) for k in range(len(path) - 1)))
    best = min((i for i in range(m) if ok[i]), key=lambda i: (-info.depth[i], i))
    return int(info.depth[best]), list(info.ancestors[best])


@pytest.mark.parametrize("vocab", [8, 16])
def test_acceptance_brute_force_exhaustive(vocab):
    cfg = small_cfg(vocab=vocab)
    om = Weights(cfg, 40 + vocab).oracle()
    kv = _kv_ctx(om, 41, 5, "bf16")
    rng = np.random.default_rng(vocab)
    n_cases = 0
    for m in range(1, 6):
        for par in all_parent_arrays(m):
            toks = rng.integers(0, vocab, m)
            got = ov.verify_step(om, kv, toks, par)
            n, path = _brute_force_accept(om, kv, toks, par)
            assert got["accept_len"] == n, (par, toks)
            assert list(got["path"]) == path
            n_cases += 1
    assert n_cases == 1 + 1 + 2 + 6 + 24


def test_greedy_accept_golden():
    for ln in _golden_lines("accept_examples.txt"):
        lhs, rhs = ln.split("->")
        par, toks, amax = [np.array([int(v) for v in s.split()]) for s in lhs.split("|")]
        n, path, bonus = [s.split() for s in rhs.split("|")]
        got = ov.greedy_accept(toks, par, amax)
        assert got[0] == int(n[0])
        assert list(got[1]) == [int(v) for v in path]
        assert got[2] == int(bonus[0])


def test_argmax_ties_lowest_id_in_fp32():
    z = np.array([[0.0, 2.0, 2.0, -1.0]])
    assert ov.argmax_lowest(z)[0] == 1
    # distinct in float64, equal once rounded to fp32
    z = np.array([[1.0, 1.0 + 2.0 ** -30, 0.5]])
    assert ov.argmax_lowest(z)[0] == 0


def _planted_tree(rng, greedy, vocab, n_nodes, depth_true):
    """Root = greedy[0]; one branch follows greedy[1:depth_true]; every other
    node is random.  Node order stays topological."""
    toks = [greedy[0]]
    par = [-1]
    prev = 0
    for k in range(1, depth_true):
        toks.append(greedy[k])
        par.append(prev)
        prev = len(toks) - 1
    while len(toks) < n_nodes:
        p = int(rng.integers(0, len(toks)))
        toks.append(int(rng.integers(0, vocab)))
        par.append(p)
    return np.array(toks), np.array(par)


def test_verify_commit_loop_is_lossless():
    """Any sequence of trees + commits emits exactly the greedy sequence."""
    cfg = small_cfg(vocab=64)
    om = Weights(cfg, 51).oracle()
    kv0 = _kv_ctx(om, 52, 6, "bf16")
    root = 7
    n_total = 24
    greedy, _ = ov.greedy_decode(om, kv0, root, n_total + 8)
    rng = np.random.default_rng(5)
    kv, emitted, pend = kv0, [], root
    while len(emitted) < n_total:
        i0 = len(emitted)
        depth_true = int(rng.integers(1, 6))
        toks, par = _planted_tree(rng, greedy[i0:], cfg.vocab, 10, depth_true)
        assert toks[0] == pend
        st = ov.verify_step(om, kv, toks, par)
        assert st["accept_len"] >= depth_true
        emitted.extend(int(toks[j]) for j in st["path"])
        kv = ov.commit(kv, st["new_k"], st["new_v"], st["path"])
        pend = st["bonus"]
    assert emitted[:n_total] == greedy[:n_total]


def test_commit_equals_prefill_of_path():
    cfg = small_cfg()
    om = Weights(cfg, 61).oracle()
    prompt = synth.prompt(62, 8, cfg.vocab)
    kv, _ = ov.prefill(om, prompt, kv_dtype="bf16")
    toks, par = synth.random_tree(63, 10, 5, cfg.vocab)
    st = ov.forward_tree(om, kv, toks, par, kv_dtype="bf16")
    info = st["tree"]
    deepest = int(np.argmax(info.depth))
    path = info.ancestors[deepest]
    kv_c = ov.commit(kv, st["new_k"], st["new_v"], path)
    kv_p, _ = ov.prefill(om, np.concatenate([prompt, toks[path]]), kv_dtype="bf16")
    for l in range(cfg.n_layers):
        np.testing.assert_allclose(kv_c[l][0], kv_p[l][0], rtol=0, atol=1e-12)
        np.testing.assert_allclose(kv_c[l][1], kv_p[l][1], rtol=0, atol=1e-12)


def test_tree_validation():
    with pytest.raises(ValueError):
        ov.tree_info([0, 0])
    with pytest.raises(ValueError):
        ov.tree_info([-1, 1])
    with pytest.raises(ValueError):
        ov.tree_info([-1, -1])
    with pytest.raises(ValueError):
        ov.tree_info([])
    info = ov.tree_info([-1, 0, 0, 2, 3])
    assert list(info.depth) == [1, 2, 2, 3, 4]
    assert list(info.ancestors[4]) == [0, 2, 3, 4]
