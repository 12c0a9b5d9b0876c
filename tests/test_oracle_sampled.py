"""Pins of the oracle's stochastic (temperature > 0) acceptance.

The paper fixes no formula for its speculative sampling rule (Section 3.1)
beyond what it credits it with (Section 5, on verifying draft tokens): the
accepted tokens follow the target model's own distribution.  That property is
the pin: with drafts drawn from q, the tokens emitted by ``accept_sampled``
must be distributed exactly as target sampling would emit them (chi-square over
many trials).  Further pins: the greedy limit (T -> 0 gives the greedy rule)
and q = p (every first child is accepted).  A plausible mistake (residual
q - p, test against q/p, no renormalisation, bonus from the unreduced p) breaks
the Monte Carlo pin.
"""
import numpy as np
import pytest
from scipy import stats

from oracle import verify as ov


def _dist(rng, v, peak=1.0):
    x = rng.random(v) ** (1.0 + 4.0 * peak)
    return x / x.sum()


def _chi2_pvalue(counts, probs):
    n = counts.sum()
    exp = probs * n
    keep = exp > 0
    return stats.chisquare(counts[keep], exp[keep] * counts[keep].sum() / exp[keep].sum()).pvalue


def test_inverse_cdf_matches_brute_force():
    rng = np.random.default_rng(0)
    for _ in range(200):
        p = rng.random(7) * (rng.random(7) > 0.3)
        if p.sum() == 0:
            continue
        u = rng.random()
        # brute force: walk the ids until the running mass exceeds u * total
        acc, want = 0.0, None
        for v in range(7):
            acc += p[v]
            if acc > u * p.sum():
                want = v
                break
        assert ov.sample_inverse_cdf(p, u) == want


def test_first_token_follows_the_target_distribution():
    """Root with 3 children drawn i.i.d. from q: the token emitted after the
    root (accepted child or bonus) is distributed as p = softmax(z / T)."""
    rng = np.random.default_rng(1)
    V, k, T, n = 5, 3, 0.7, 20000
    z0 = rng.normal(size=V) * 1.5
    q0 = _dist(rng, V)
    p0 = ov.softmax_t(z0, T)
    parents = np.array([-1] + [0] * k)
    logits = np.zeros((k + 1, V))
    logits[0] = z0
    q = np.tile(q0, (k + 1, 1))
    counts = np.zeros(V)
    for _ in range(n):
        toks = np.concatenate([[0], rng.choice(V, size=k, p=q0)])
        n_acc, path, bonus = ov.accept_sampled(logits, toks, parents, q, T, rng.random(k + 1), rng.random(k + 1))
        counts[toks[path[1]] if n_acc > 1 else bonus] += 1
    assert _chi2_pvalue(counts, p0) > 1e-3


def test_two_tokens_follow_the_target_distribution():
    """Two levels: root -> 2 children -> 2 grandchildren each, drafts i.i.d.
    from per-node q; the target's distribution after token a is softmax(z2[a]).
    The first two emitted tokens must follow p0(a) * p_a(b) (when the step
    stops at the root, the second token is what the next step would emit)."""
    rng = np.random.default_rng(2)
    V, T, n = 4, 1.0, 30000
    z0 = rng.normal(size=V)
    z2 = rng.normal(size=(V, V)) * 1.2
    q0 = _dist(rng, V)
    q2 = np.stack([_dist(rng, V) for _ in range(V)])
    parents = np.array([-1, 0, 0, 1, 1, 2, 2])
    joint = np.outer(ov.softmax_t(z0, T), np.ones(V)) * np.stack([ov.softmax_t(z2[a], T) for a in range(V)])
    counts = np.zeros((V, V))
    for _ in range(n):
        a1, a2 = rng.choice(V, size=2, p=q0)
        g = [rng.choice(V, size=2, p=q2[a]) for a in (a1, a2)]
        toks = np.array([0, a1, a2, g[0][0], g[0][1], g[1][0], g[1][1]])
        logits = np.stack([z0, z2[a1], z2[a2], z0, z0, z0, z0])
        q = np.stack([q0, q2[a1], q2[a2], q0, q0, q0, q0])
        n_acc, path, bonus = ov.accept_sampled(logits, toks, parents, q, T, rng.random(7), rng.random(7))
        emitted = [int(toks[i]) for i in path[1:]] + [bonus]
        if len(emitted) == 1:
            # the step ended at the root; the next step's first token follows
            # the target after the bonus (the single-level pin above)
            emitted.append(int(rng.choice(V, p=ov.softmax_t(z2[bonus], T))))
        counts[emitted[0], emitted[1]] += 1
    assert _chi2_pvalue(counts.ravel(), joint.ravel()) > 1e-3


def test_mistakes_break_the_distribution_pin():
    """The residual taken the wrong way round (q - p) visibly changes the
    first-token distribution, so the Monte Carlo pin can see such a slip."""
    rng = np.random.default_rng(3)
    V, k, T, n = 5, 3, 0.7, 20000
    z0 = rng.normal(size=V) * 1.5
    q0 = _dist(rng, V)
    p0 = ov.softmax_t(z0, T)
    counts = np.zeros(V)
    for _ in range(n):
        toks = rng.choice(V, size=k, p=q0)
        p, out = p0.copy(), None
        for t in toks:
            if rng.random() * q0[t] < p[t]:
                out = t
                break
            r = np.maximum(q0 - p, 0.0)         # planted mistake
            p = r / r.sum() if r.sum() > 0 else p
        counts[out if out is not None else ov.sample_inverse_cdf(p, rng.random())] += 1
    assert _chi2_pvalue(counts, p0) < 1e-6


@pytest.mark.parametrize("seed", range(6))
def test_greedy_limit(seed):
    """T -> 0 with distinct sibling tokens: the sampled rule is the greedy rule."""
    rng = np.random.default_rng(10 + seed)
    V, m = 12, 14
    parents = [-1] + [int(rng.integers(0, i)) for i in range(1, m)]
    logits = rng.normal(size=(m, V))
    amax = ov.argmax_lowest(logits)
    toks = np.zeros(m, dtype=np.int64)
    for u in range(m):
        kids = [c for c in range(1, m) if parents[c] == u]
        ids = rng.permutation(V)[:len(kids)]
        if kids and rng.random() < 0.7:
            ids[int(rng.integers(0, len(kids)))] = amax[u]   # plant the argmax
            ids = list(dict.fromkeys(ids)) + [i for i in range(V) if i not in ids]
        for c, t in zip(kids, ids):
            toks[c] = t
    q = np.stack([_dist(rng, V) for _ in range(m)])
    n_g, path_g, bonus_g = ov.greedy_accept(toks, parents, amax)
    n_s, path_s, bonus_s = ov.accept_sampled(logits, toks, parents, q, 1e-4, rng.random(m) * 0.999,
                                             rng.random(m))
    assert (n_s, list(path_s), bonus_s) == (n_g, list(path_g), bonus_g)


def test_draft_equal_to_target_accepts_first_children():
    rng = np.random.default_rng(20)
    V, m, T = 9, 10, 0.8
    parents = np.array([-1, 0, 0, 1, 1, 3, 2, 6, 6, 7])
    logits = rng.normal(size=(m, V))
    q = np.stack([ov.softmax_t(logits[u], T) for u in range(m)])
    toks = rng.integers(0, V, size=m)
    n, path, _ = ov.accept_sampled(logits, toks, parents, q, T, rng.random(m) * 0.999, rng.random(m))
    # first child at every level: 0 -> 1 -> 3 -> 5 (a leaf)
    assert list(path) == [0, 1, 3, 5] and n == 4
