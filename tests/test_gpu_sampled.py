"""Sampled (temperature > 0) verification on the GPU vs the oracle's
``accept_sampled``, through the C ABI.

Inputs are identical bytes on both sides: float32 logits, float32 draft
distributions, float32 uniforms.  The kernel works in float32 and the oracle in
float64, so a decision whose two sides lie within rounding of each other may go
either way; every case therefore takes the oracle's decision trace and

* requires the exact same path and bonus when every decision clears its
  margin (relative 1e-4 of the compared values plus 1e-6 over the residual
  mass for an acceptance, 2e-6 of the total mass for the bonus);
* otherwise checks that the GPU result is a valid outcome: a root-to-node
  chain that leaves the oracle's path exactly at a decision inside the
  margin (the first child, in trial order, that the two walks treated
  differently), or, on the same path, a bonus whose cumulative-mass interval
  touches the target within the margin.

Outcomes that differ from the oracle's must stay rare (at most one per test),
so the comparison is not vacuous.
"""
import numpy as np
import pytest

import synth
from oracle import verify as ov
from tests.helpers import GpuCase, small_cfg

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2412_18934_amd import dv  # noqa: E402


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda:0")


def _accept(h, logits, toks, par, q, temperature, ua, ub):
    """dv_accept_sampled on host arrays (the device copies stay referenced
    until the call has returned)."""
    lg, qd = _dev(logits), _dev(q)
    return dv.dv_accept_sampled(h, lg.data_ptr(), toks, par, qd.data_ptr(), temperature, ua, ub)


def _chain_ok(path, parents):
    return path[0] == 0 and all(parents[path[k]] == path[k - 1] for k in range(1, len(path)))


def _judge(acc, n, path, bonus, trace, parents, vocab, rel=1e-4, bonus_rel=2e-6):
    """True when the GPU outcome equals the oracle's.  A different outcome is
    allowed only where the oracle's own decision lay within the margin (then
    False is returned): a different path needs an acceptance test whose two
    sides differ by at most rel (relative, plus 1e-6 over the residual mass);
    a different bonus on the same path must still be a valid inverse-CDF draw
    within bonus_rel of the total mass."""
    got_path = acc.path_list
    assert acc.accept_len == len(got_path) >= 1
    assert _chain_ok(got_path, parents), got_path
    assert 0 <= acc.bonus_token < vocab
    if got_path == list(path) and acc.bonus_token == bonus:
        return True
    if got_path != list(path):
        # the first node where the two walks part: the oracle moved to child a
        # (None: it stopped there), the GPU to child b; children are tried in
        # index order, so the first decision the two took differently is the
        # one on child min(a, b), which the oracle's walk reached
        k = 1
        while k < len(got_path) and k < len(path) and got_path[k] == path[k]:
            k += 1
        a = path[k] if k < len(path) else None
        b = got_path[k] if k < len(got_path) else None
        c = min(x for x in (a, b) if x is not None)
        ev = [e for e in trace if e[0] == "accept" and e[1] == c]
        assert len(ev) == 1, ("oracle never tried the child where the walks part", c, got_path, list(path))
        _, _, uq, pt, mass = ev[0]
        assert abs(uq - pt) <= rel * max(uq, pt) + 1e-6 / mass, \
            ("walks part at a clear decision", c, uq, pt, got_path, list(path))
        return False
    p, u = trace[-1][1], trace[-1][2]
    c = np.cumsum(p)
    target, tol = u * c[-1], bonus_rel * c[-1]
    b = acc.bonus_token
    lo = c[b - 1] if b > 0 else 0.0
    assert lo <= target + tol and c[b] >= target - tol and p[b] > 0, \
        ("bonus is not a draw within the margin", b, bonus)
    return False


def _correlated_drafts(logits, temperature, noise, rng):
    """Draft distributions that roughly agree with the target: the target's
    logits plus Gaussian noise, at the same temperature (float64, stored
    float32)."""
    z = (logits.astype(np.float64) + noise * rng.standard_normal(logits.shape)) / temperature
    z -= z.max(axis=1, keepdims=True)
    e = np.exp(z)
    return (e / e.sum(axis=1, keepdims=True)).astype(np.float32)


def _draft_tree(m, depth, q, seed, vocab):
    """Parents from the seeded tree generator; every child's token drawn from
    its parent's draft distribution (numpy's sampler)."""
    _, parents = synth.random_tree(seed, m, depth, vocab)
    rng = np.random.default_rng(seed)
    toks = np.zeros(m, dtype=np.int32)
    toks[0] = int(rng.integers(0, vocab))
    qd = q.astype(np.float64)
    for c in range(1, m):
        row = qd[parents[c]]
        toks[c] = int(rng.choice(vocab, p=row / row.sum()))
    return toks, parents


@pytest.fixture(scope="module")
def head_case():
    # only the handle's vocabulary matters for the sampling entry point
    case = GpuCase(small_cfg(n_layers=1, d_model=64, n_heads=1, head_dim=64, d_ffn=96, vocab=32000),
                   seed=5, capacity=64)
    yield case
    case.close()


@pytest.mark.parametrize("m", [1, 2, 7, 16, 33, 64])
@pytest.mark.parametrize("temperature", [0.6, 1.0, 1.7])
def test_accept_sampled_matches_oracle(head_case, m, temperature):
    V = head_case.cfg.vocab
    exact = differ = 0
    for rep in range(4):
        seed = 1000 * m + 10 * rep + int(10 * temperature)
        rng = np.random.default_rng(seed)
        logits = synth.normal(seed, 90, m * V, 2.0, "f32").reshape(m, V)
        q = _correlated_drafts(logits, temperature, (0.3, 1.0, 3.0, 0.0)[rep], rng)
        if rep == 3:
            q = synth.draft_rows(seed, m, V, sharp=16.0)   # drafts unrelated to the target
        toks, par = _draft_tree(m, 6, q, seed, V)
        ua, ub = synth.sampling_uniforms(seed, m)
        trace = []
        n, path, bonus = ov.accept_sampled(logits, toks, par, q, temperature, ua, ub, trace=trace)
        lg, qd = _dev(logits), _dev(q)
        acc = dv.dv_accept_sampled(head_case.h, lg.data_ptr(), toks, par, qd.data_ptr(), temperature, ua, ub)
        assert acc.base_len == -1 and acc.n_tree == m
        if _judge(acc, n, path, bonus, trace, par, V):
            exact += 1
        else:
            differ += 1
    assert differ <= 1, (exact, differ)


@pytest.mark.parametrize("V", [8224, 40992])
def test_accept_sampled_ragged_chunks(V):
    # 8224: threads own 12 ids each, the last busy thread 4, the rest none;
    # 40992: 44 ids each (a second load batch), the last busy thread 28
    case = GpuCase(small_cfg(n_layers=1, n_heads=1, head_dim=64, vocab=V), seed=6, capacity=64)
    try:
        exact = 0
        for seed in range(20):
            m = 1 + seed * 3
            rng = np.random.default_rng(seed)
            logits = synth.normal(seed, 91, m * V, 3.0, "f32").reshape(m, V)
            q = _correlated_drafts(logits, 0.8, 1.5, rng)
            toks, par = _draft_tree(m, 8, q, 500 + seed, V)
            ua, ub = synth.sampling_uniforms(700 + seed, m)
            trace = []
            n, path, bonus = ov.accept_sampled(logits, toks, par, q, 0.8, ua, ub, trace=trace)
            acc = _accept(case.h, logits, toks, par, q, 0.8, ua, ub)
            exact += _judge(acc, n, path, bonus, trace, par, V)
        assert exact >= 18
    finally:
        case.close()


def test_accept_sampled_degenerate_cases(head_case):
    V = head_case.cfg.vocab
    rng = np.random.default_rng(9)
    m = 9
    par = np.array([-1, 0, 0, 0, 1, 1, 4, 4, 2], dtype=np.int32)
    logits = synth.normal(9, 92, m * V, 2.0, "f32").reshape(m, V)
    toks = rng.integers(0, V, size=m).astype(np.int32)
    ua, ub = synth.sampling_uniforms(9, m)

    # draft mass 1 on every id: every residual is empty and p stays the
    # target's, so each child is accepted only when u < p(t)
    q = np.ones((m, V), dtype=np.float32)
    trace = []
    n, path, bonus = ov.accept_sampled(logits, toks, par, q, 1.0, ua, ub, trace=trace)
    acc = _accept(head_case.h, logits, toks, par, q, 1.0, ua, ub)
    _judge(acc, n, path, bonus, trace, par, V)
    assert acc.path_list == list(path)

    # a child that carries the target's top token with a tiny draft
    # probability is always accepted (u q(t) < p(t) for every u < 1)
    top = int(np.argmax(logits[0]))
    toks2 = toks.copy()
    toks2[1] = top
    q2 = synth.draft_rows(9, m, V)
    q2[0, top] = 1e-30
    acc = _accept(head_case.h, logits, toks2, par, q2, 1.0, ua, ub)
    assert acc.path_list[:2] == [0, 1]

    # root alone: the bonus is an inverse-CDF draw from softmax(z / T)
    for u in (0.0, 0.25, 0.5, 0.999):
        trace = []
        n, path, bonus = ov.accept_sampled(logits[:1], toks[:1], par[:1], q[:1], 0.7, [0.0], [u], trace=trace)
        acc = _accept(head_case.h, logits[:1], toks[:1], par[:1], q[:1], 0.7, [0.0], [u])
        assert acc.accept_len == 1
        _judge(acc, n, path, bonus, trace, par[:1], V)

    # very low temperature: the greedy rule (distinct sibling tokens)
    am = logits.argmax(axis=1)
    toks3 = toks.copy()
    toks3[1], toks3[4], toks3[6] = am[0], am[1], am[4]
    acc = _accept(head_case.h, logits, toks3, par, q2, 1e-3, ua * np.float32(0.999), ub)
    n_g, path_g, bonus_g = ov.greedy_accept(toks3, par, ov.argmax_lowest(logits))
    assert (acc.accept_len, acc.path_list, acc.bonus_token) == (n_g, list(path_g), bonus_g)

    # very high temperature with a large logit spread still gives a valid draw
    big = (logits * 40.0).astype(np.float32)
    trace = []
    n, path, bonus = ov.accept_sampled(big, toks, par, q2, 25.0, ua, ub, trace=trace)
    acc = _accept(head_case.h, big, toks, par, q2, 25.0, ua, ub)
    _judge(acc, n, path, bonus, trace, par, V)


def test_accept_sampled_is_deterministic(head_case):
    V, m = head_case.cfg.vocab, 40
    rng = np.random.default_rng(11)
    logits = synth.normal(11, 93, m * V, 2.0, "f32").reshape(m, V)
    q = _correlated_drafts(logits, 1.0, 1.0, rng)
    toks, par = _draft_tree(m, 7, q, 11, V)
    ua, ub = synth.sampling_uniforms(11, m)
    lg, qd = _dev(logits), _dev(q)
    ref = dv.dv_accept_sampled(head_case.h, lg.data_ptr(), toks, par, qd.data_ptr(), 1.0, ua, ub)
    for _ in range(5):
        acc = dv.dv_accept_sampled(head_case.h, lg.data_ptr(), toks, par, qd.data_ptr(), 1.0, ua, ub)
        assert (acc.accept_len, acc.path_list, acc.bonus_token) == (ref.accept_len, ref.path_list,
                                                                    ref.bonus_token)


def test_sampled_error_paths(head_case):
    V = head_case.cfg.vocab
    m = 3
    par = np.array([-1, 0, 0], dtype=np.int32)
    toks = np.array([1, 2, 3], dtype=np.int32)
    lg = _dev(np.zeros((m, V), dtype=np.float32))
    q = _dev(np.full((m, V), 1.0 / V, dtype=np.float32))
    ua, ub = synth.sampling_uniforms(1, m)
    h = head_case.h
    bad = [
        dict(temperature=0.0), dict(temperature=-1.0), dict(temperature=float("nan")),
        dict(temperature=float("inf")), dict(temperature=1e-45),
        dict(ua=np.array([0.0, 1.0, 0.5], dtype=np.float32)),
        dict(ub=np.array([0.5, -0.1, 0.5], dtype=np.float32)),
        dict(ua=np.array([0.0, np.nan, 0.5], dtype=np.float32)),
        dict(q=0), dict(logits=0), dict(logits=lg.data_ptr() + 4), dict(q=q.data_ptr() + 8),
        dict(par=np.array([-1, 0, 2], dtype=np.int32)), dict(toks=np.array([1, V, 3], dtype=np.int32)),
    ]
    for b in bad:
        with pytest.raises(dv.DvError) as ei:
            dv.dv_accept_sampled(h, b.get("logits", lg.data_ptr()), b.get("toks", toks), b.get("par", par),
                                 b.get("q", q.data_ptr()), b.get("temperature", 1.0), b.get("ua", ua),
                                 b.get("ub", ub))
        assert ei.value.code == dv.DV_EINVAL, b
    # u_accept[0] is not read, so any value there is accepted
    dv.dv_accept_sampled(h, lg.data_ptr(), toks, par, q.data_ptr(), 1.0,
                         np.array([7.0, 0.5, 0.5], dtype=np.float32), ub)


# ---------------------------------------------------------------------------
# the whole step: forward pass + sampling, then commit

def test_tiny_f32_sampled_step_matches_oracle_and_commits():
    cfg = small_cfg(n_layers=2, d_model=128, n_heads=2, head_dim=64, d_ffn=256, vocab=512,
                    weight_dtype="f32", init_std=0.12)
    case = GpuCase(cfg, seed=21, capacity=128)
    try:
        om = case.w.oracle()
        exact = 0
        for rep, (m, temperature) in enumerate([(1, 1.0), (6, 0.7), (16, 1.0), (23, 1.3), (40, 0.9)]):
            kv = case.new_kv()
            p = 19 + rep
            kv_o = case.synthetic_context(kv, 30 + rep, p)
            seed = 40 + rep
            _, par = synth.random_tree(seed, m, 6, cfg.vocab)
            rng = np.random.default_rng(seed)
            # the draft sees the oracle's logits of a greedy step of the same
            # tree shape, perturbed (any non-negative rows would do)
            toks0 = synth.prompt(seed, m, cfg.vocab)
            ref0 = ov.verify_step(om, kv_o, toks0, par)
            q = _correlated_drafts(ref0["logits"], temperature, 0.5, rng)
            toks = toks0.copy()
            for c in range(1, m):
                row = q[par[c]].astype(np.float64)
                toks[c] = int(rng.choice(cfg.vocab, p=row / row.sum()))
            ref = ov.verify_step(om, kv_o, toks, par)
            ua, ub = synth.sampling_uniforms(seed, m)
            trace = []
            n, path, bonus = ov.accept_sampled(ref["logits"], toks, par, q, temperature, ua, ub, trace=trace)
            out = torch.full((m, cfg.vocab), float("nan"), device="cuda:0")
            qd = _dev(q)
            acc = dv.dv_verify_step_sampled(case.h, toks, par, kv.c, qd.data_ptr(), temperature, ua, ub,
                                            out.data_ptr())
            lg = out.cpu().numpy()
            assert float(np.abs(lg - ref["logits"]).max()) <= 1e-4
            # logits differ from the oracle's by up to 1e-4: widen the margins
            same = _judge(acc, n, path, bonus, trace, par, cfg.vocab, rel=1e-3 / temperature,
                          bonus_rel=1e-3 / temperature)
            exact += same
            # the sampling rule inside the step is the stand-alone entry point
            acc2 = dv.dv_accept_sampled(case.h, out.data_ptr(), toks, par, qd.data_ptr(), temperature, ua, ub)
            assert (acc2.accept_len, acc2.path_list, acc2.bonus_token) == (acc.accept_len, acc.path_list,
                                                                           acc.bonus_token)
            if not same:
                continue
            # commit the sampled path (each side its own, equal as just
            # checked), then a greedy step over it matches the oracle on the
            # committed context
            dv.dv_kv_commit(case.h, kv.c, acc)
            kv_o = ov.commit(kv_o, ref["new_k"], ref["new_v"], path)
            assert kv.c.len == p + n
            toks_n, par_n = synth.random_tree(seed + 7, 5, 3, cfg.vocab)
            toks_n[0] = bonus
            ref_n = ov.verify_step(om, kv_o, toks_n, par_n)
            acc_n, lg_n = case.step(kv, toks_n, par_n)
            assert float(np.abs(lg_n - ref_n["logits"]).max()) <= 1e-4
        assert exact >= 4
    finally:
        case.close()


def test_bf16_sampled_step_logits_equal_greedy_step():
    cfg = small_cfg(n_layers=2, d_model=256, n_heads=2, head_dim=128, d_ffn=512, vocab=2048,
                    weight_dtype="bf16", init_std=0.09)
    case = GpuCase(cfg, seed=71, capacity=256)
    try:
        m = 17
        kv = case.new_kv()
        case.synthetic_context(kv, 72, 50)
        toks, par = synth.random_tree(75, m, 6, cfg.vocab)
        acc_g, lg_g = case.step(kv, toks, par)
        q = _dev(synth.draft_rows(3, m, cfg.vocab))
        ua, ub = synth.sampling_uniforms(3, m)
        out = torch.full((m, cfg.vocab), float("nan"), device="cuda:0")
        acc = dv.dv_verify_step_sampled(case.h, toks, par, kv.c, q.data_ptr(), 1.0, ua, ub, out.data_ptr())
        np.testing.assert_array_equal(out.cpu().numpy(), lg_g)
        assert acc.base_len == 50 and all(a == 0 for a in acc.argmax[:m])
        # no out_logits: the handle's workspace holds them; same outcome
        acc_w = dv.dv_verify_step_sampled(case.h, toks, par, kv.c, q.data_ptr(), 1.0, ua, ub, 0)
        assert (acc_w.accept_len, acc_w.path_list, acc_w.bonus_token) == (acc.accept_len, acc.path_list,
                                                                          acc.bonus_token)
        dv.dv_kv_commit(case.h, kv.c, acc_w)
        assert kv.c.len == 50 + acc.accept_len
    finally:
        case.close()
