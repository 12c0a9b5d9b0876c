"""Pins of the draft-side oracle (DGF, draft forward, tree construction).

* DGF: a zero gate layer gives g = 1/2, so the output is the mean of the two
  projections; a gate saturated to one side returns that side's projection.
* draft forward: feeding the stack its own embedding rows through ``x0``
  reproduces the plain forward, and the logits are the lm_head of the
  RMS-normalised output features.
* tree construction against brute force: when every node of every layer is
  expanded with every token, the selection is the n - 1 most probable token
  sequences of length <= depth (enumerated directly); with width 1 the tree
  is the draft's greedy chain; structure (ancestor closure, topological
  order, scores non-increasing along paths) on random draft functions.
"""
import itertools

import numpy as np
import pytest

import synth
from oracle import draft as od
from oracle import verify as ov
from tests.helpers import Weights, small_cfg


def test_dgf_zero_gate_is_the_mean():
    rng = np.random.default_rng(0)
    f, e = rng.normal(size=(3, 8)), rng.normal(size=(3, 8))
    wh, we = rng.normal(size=(8, 8)), rng.normal(size=(8, 8))
    out = od.dgf(f, e, wh, we, np.zeros((8, 16)))
    np.testing.assert_allclose(out, 0.5 * (f @ wh.T) + 0.5 * (e @ we.T), rtol=1e-14)


@pytest.mark.parametrize("side", [1.0, -1.0])
def test_dgf_saturated_gate_picks_one_side(side):
    rng = np.random.default_rng(1)
    f, e = np.abs(rng.normal(size=(2, 4))) + 0.5, np.abs(rng.normal(size=(2, 4))) + 0.5
    wh, we = np.eye(4), 2 * np.eye(4)
    wg = np.zeros((4, 8))
    wg[:, :4] = side * 1e3 * np.eye(4)     # g = sigmoid(+-1e3 * h1) with h1 > 0
    out = od.dgf(f, e, wh, we, wg)
    np.testing.assert_allclose(out, f if side > 0 else 2 * e, rtol=1e-12)


def test_draft_forward_x0_override_and_head():
    cfg = small_cfg(n_layers=1, d_model=64, n_heads=1, head_dim=64, d_ffn=96, vocab=128, weight_dtype="f32")
    om = Weights(cfg, 3).oracle()
    kv = ov.kv_from_raw([synth.kv_layer(cfg, 4, 0, 5)])
    toks, par = synth.random_tree(5, 6, 3, cfg.vocab)
    a = ov.forward_tree(om, kv, toks, par)
    b = ov.forward_tree(om, kv, toks, par, x0=om.embed(toks, np.float64))
    np.testing.assert_array_equal(a["logits"], b["logits"])
    u = ov.rmsnorm(a["hidden"], ov._to_float(om.final_norm, np.float64), cfg.rms_eps)
    np.testing.assert_allclose(u @ ov._to_float(om.lm_head, np.float64).T, a["logits"], rtol=1e-12)


def _table_draft(V, seed):
    """A draft whose distribution depends only on the token path (hashed)."""
    def forward(tokens, parents, feat_in):
        paths = []
        for i in range(len(tokens)):
            p = [tokens[i]]
            j = parents[i]
            while j >= 0:
                p.append(tokens[j])
                j = parents[j]
            paths.append(tuple(reversed(p)))
        logits = np.stack([np.random.default_rng(hash((seed,) + pth) % (1 << 32)).normal(size=V) * 2.0
                           for pth in paths])
        return logits, np.zeros((len(tokens), 4))
    return forward


def _path_prob(forward, root, seq):
    prob, path = 1.0, [root]
    for t in seq:
        z, _ = forward(path, list(range(-1, len(path) - 1)), None)
        p = np.exp(z[-1] - z[-1].max())
        p /= p.sum()
        prob *= p[t]
        path.append(t)
    return prob


@pytest.mark.parametrize("seed", range(3))
def test_full_expansion_selects_the_most_probable_sequences(seed):
    V, depth, n_tree = 3, 3, 9
    fwd = _table_draft(V, seed)
    toks, par, sc = od.build_tree(fwd, 1, np.zeros(4), depth, width=V ** depth, n_tree=n_tree)
    got = set()
    for i in range(1, len(toks)):
        seq, j = [], i
        while j > 0:
            seq.append(int(toks[j]))
            j = par[j]
        got.add(tuple(reversed(seq)))
    allseq = [s for L in range(1, depth + 1) for s in itertools.product(range(V), repeat=L)]
    probs = {s: _path_prob(fwd, 1, s) for s in allseq}
    best = sorted(allseq, key=lambda s: -probs[s])
    assert probs[best[n_tree - 2]] > probs[best[n_tree - 1]] * (1 + 1e-9)  # no tie at the cut
    assert got == set(best[: n_tree - 1])


def test_width_one_is_the_greedy_chain():
    V = 7
    fwd = _table_draft(V, 11)
    toks, par, _ = od.build_tree(fwd, 2, np.zeros(4), depth=5, width=1, n_tree=6)
    assert list(par) == [-1, 0, 1, 2, 3, 4]
    path = [2]
    for _ in range(5):
        z, _ = fwd(path, list(range(-1, len(path) - 1)), None)
        path.append(int(np.argmax(z[-1])))
    assert list(toks) == path


@pytest.mark.parametrize("seed", range(4))
def test_tree_structure(seed):
    V = 12
    fwd = _table_draft(V, 100 + seed)
    toks, par, sc = od.build_tree(fwd, 0, np.zeros(4), depth=4, width=3, n_tree=10)
    assert len(toks) == 10 and par[0] == -1
    for i in range(1, 10):
        assert 0 <= par[i] < i
        assert sc[i] <= sc[par[i]] + 1e-15
    info = ov.tree_info(par)
    assert info.depth.max() <= 5
