"""GPU path vs the CPU oracle on identical seeded inputs, through the C ABI.

Bars: logits max-abs 1e-4 with fp32 weights, 2e-2 with bf16 weights (fp32
accumulation); argmax, accepted length, path and bonus bit-exact (argmax
near-ties, where the oracle's top-2 gap is within 2x the logits tolerance,
are counted and checked for validity instead); KV commit bit-exact.
"""
import numpy as np
import pytest

import synth
from oracle import verify as ov
from tests.helpers import GpuCase, compare_step, small_cfg

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2412_18934_amd import dv  # noqa: E402


def _ref(om, kv_o, toks, par):
    r = ov.verify_step(om, kv_o, toks, par)
    r["tokens"], r["parents"] = np.asarray(toks), np.asarray(par)
    return r


# ---------------------------------------------------------------------------
# the tiny fp32 workload: prefill of 64 prompt tokens + a chain of 4

def test_tiny_f32_prefill_and_chain():
    wl = synth.WORKLOADS["tiny-f32-chain4"]
    mc, sd = wl.model, wl.seeds
    case = GpuCase(mc, sd["weights"], capacity=wl.context + 64)
    try:
        om = case.w.oracle()
        kv = case.new_kv()
        prompt = synth.prompt(sd["prompt"], wl.context, mc.vocab)
        root = dv.dv_prefill(case.h, prompt, kv.c)
        assert kv.len == wl.context
        kv_o, pre = ov.prefill(om, prompt)
        assert root == int(ov.argmax_lowest(pre[-1:])[0])
        for l in range(mc.n_layers):
            k, v = kv.layer_host(l, wl.context)
            np.testing.assert_allclose(k, kv_o[l][0], rtol=0, atol=2e-5)
            np.testing.assert_allclose(v, kv_o[l][1], rtol=0, atol=2e-5)
        # chain of 4 whose tokens follow the oracle's greedy continuation
        greedy, _ = ov.greedy_decode(om, kv_o, root, wl.n_tree + 1)
        toks = np.array(greedy[:wl.n_tree])
        par = np.arange(-1, wl.n_tree - 1)
        # the oracle consumes the GPU-independent cache it built itself
        ref = _ref(om, kv_o, toks, par)
        acc, lg = case.step(kv, toks, par)
        err, near = compare_step(acc, lg, ref, 1e-4)
        assert near == 0 and acc.accept_len == wl.n_tree
        assert acc.bonus_token == greedy[wl.n_tree]
    finally:
        case.close()


# ---------------------------------------------------------------------------
# bf16 models that span several tiles with ragged tails

# init_std 0.09 gives logits of the spread a 13B-shaped model has (std ~1.4)
BF16 = dict(n_layers=2, d_model=256, n_heads=2, head_dim=128, d_ffn=512, vocab=2048,
            weight_dtype="bf16", init_std=0.09)


@pytest.fixture(scope="module")
def bf16_case():
    case = GpuCase(small_cfg(**BF16), seed=71, capacity=256)
    yield case
    case.close()


@pytest.mark.parametrize("m", [1, 2, 15, 16, 17, 33, 64])
def test_bf16_random_tree_parity(bf16_case, m):
    case = bf16_case
    om = case.w.oracle()
    p = 77
    kv = case.new_kv()
    kv_o = case.synthetic_context(kv, 72, p)
    toks, par = synth.random_tree(73 + m, m, 8, case.cfg.vocab)
    ref = _ref(om, kv_o, toks, par)
    acc, lg = case.step(kv, toks, par)
    err, near = compare_step(acc, lg, ref, 2e-2)
    assert near <= max(3, m // 3)
    # the tree's keys/values in slots [p, p+m): one bf16 rounding step (2^-7
    # relative) plus, in layer 0, the fp32 accumulation error of one length-d
    # dot product; later layers also inherit the earlier layers' differences
    for l in range(case.cfg.n_layers):
        k, v = kv.layer_host(l, p + m)
        for got, want in ((k, ref["new_k"][l]), (v, ref["new_v"][l])):
            want = np.transpose(want, (1, 0, 2))
            rms = np.sqrt(np.mean(want ** 2))
            g64 = ov.bf16_to_f64(got[:, p:])
            # observed error beyond the one-rounding-step part, in units of the RMS
            excess = float(np.max(np.abs(g64 - want) - 2 ** -7 * np.abs(want))) / rms
            print("[kv-rows] M=%d layer %d: max excess over one bf16 step %.2e of RMS" % (m, l, excess))
            np.testing.assert_allclose(g64, want, rtol=2 ** -7,
                                       atol=(1e-4 if l == 0 else 5e-3) * rms)


def test_bf16_empty_context_and_planted_acceptance(bf16_case):
    case = bf16_case
    om = case.w.oracle()
    kv = case.new_kv()
    kv_o = case.synthetic_context(kv, 74, 0)
    root = 5
    greedy, _ = ov.greedy_decode(om, kv_o, root, 6)
    rng = np.random.default_rng(3)
    toks, par = [root], [-1]
    for k in range(1, 5):                       # planted branch of depth 5
        toks.append(greedy[k])
        par.append(len(toks) - 2 if k > 1 else 0)
    while len(toks) < 12:
        par.append(int(rng.integers(0, len(toks))))
        toks.append(int(rng.integers(0, case.cfg.vocab)))
    ref = _ref(om, kv_o, np.array(toks), np.array(par))
    acc, lg = case.step(kv, np.array(toks), np.array(par))
    compare_step(acc, lg, ref, 2e-2)
    assert acc.accept_len >= 5


@pytest.mark.parametrize("m", [20, 40, 64])
def test_bf16_head_dim_64_parity(m):
    """Head size 64 with 2, 3 and 4 query tiles (the attention's multi-tile
    variants for that head size)."""
    cfg = small_cfg(n_layers=2, d_model=256, n_heads=4, head_dim=64, d_ffn=528, vocab=1056,
                    weight_dtype="bf16", init_std=0.09)
    case = GpuCase(cfg, seed=81, capacity=224)
    try:
        om = case.w.oracle()
        kv = case.new_kv()
        kv_o = case.synthetic_context(kv, 82, 45)
        toks, par = synth.random_tree(83 + m, m, 6, cfg.vocab)
        ref = _ref(om, kv_o, toks, par)
        acc, lg = case.step(kv, toks, par)
        compare_step(acc, lg, ref, 2e-2)
    finally:
        case.close()


def test_bf16_split_k_fold_parity():
    """d_model 1024 / d_ffn 2816: the O and down projections split K (2 and 5
    ways on 256 CUs) and the last split of each row group folds the partials,
    adds the residual and writes the next norm's input; bitwise repeatable."""
    cfg = small_cfg(n_layers=2, d_model=1024, n_heads=8, head_dim=128, d_ffn=2816, vocab=4096,
                    weight_dtype="bf16", init_std=0.045)
    case = GpuCase(cfg, seed=111, capacity=320)
    try:
        om = case.w.oracle()
        kv = case.new_kv()
        kv_o = case.synthetic_context(kv, 112, 200)
        for m in (16, 40):
            toks, par = synth.random_tree(113 + m, m, 6, cfg.vocab)
            ref = _ref(om, kv_o, toks, par)
            acc, lg = case.step(kv, toks, par)
            compare_step(acc, lg, ref, 2e-2)
            acc2, lg2 = case.step(kv, toks, par)
            assert np.array_equal(lg, lg2)
    finally:
        case.close()


def test_step_is_deterministic_and_ignores_stale_slots(bf16_case):
    """Same step twice -> bitwise equal; NaN in unused cache slots changes nothing."""
    case = bf16_case
    toks, par = synth.random_tree(91, 24, 6, case.cfg.vocab)
    kv = case.new_kv()
    case.synthetic_context(kv, 92, 50)
    a1, l1 = case.step(kv, toks, par)
    a2, l2 = case.step(kv, toks, par)
    assert np.array_equal(l1, l2)
    assert a1.path_list == a2.path_list and list(a1.argmax_array()) == list(a2.argmax_array())
    kvn = case.new_kv(fill=float("nan"))
    case.synthetic_context(kvn, 92, 50)
    a3, l3 = case.step(kvn, toks, par)
    assert np.array_equal(l1, l3)
    assert a3.path_list == a1.path_list


# ---------------------------------------------------------------------------
# commit

def test_commit_overlapping_path_moves_rows_exactly(bf16_case):
    """Path 0-2-3: slot p+1 <- p+2 and p+2 <- p+3 (a destination is another
    move's source); every other slot keeps its bytes."""
    case = bf16_case
    p = 40
    kv = case.new_kv()
    case.synthetic_context(kv, 93, p)
    toks = np.array([3, 4, 5, 6, 7, 8])
    par = np.array([-1, 0, 0, 2, 3, 1])
    acc, _ = case.step(kv, toks, par, want_logits=False)
    before = [kv.layer_host(l, p + 6) for l in range(case.cfg.n_layers)]
    acc.accept_len = 3
    acc.path[0], acc.path[1], acc.path[2] = 0, 2, 3
    dv.dv_kv_commit(case.h, kv.c, acc)
    torch.cuda.synchronize()
    assert kv.len == p + 3
    for l in range(case.cfg.n_layers):
        after = kv.layer_host(l, p + 6)
        for which in range(2):
            b, a = before[l][which], after[which]
            assert np.array_equal(a[:, :p], b[:, :p])
            assert np.array_equal(a[:, p + 0], b[:, p + 0])
            assert np.array_equal(a[:, p + 1], b[:, p + 2])
            assert np.array_equal(a[:, p + 2], b[:, p + 3])
            assert np.array_equal(a[:, p + 3:], b[:, p + 3:])


def test_commit_then_step_equals_oracle(bf16_case):
    """The committed cache feeds the next step exactly as the oracle's commit."""
    case = bf16_case
    om = case.w.oracle()
    kv = case.new_kv()
    kv_o = case.synthetic_context(kv, 94, 30)
    toks, par = synth.random_tree(95, 10, 4, case.cfg.vocab)
    acc, _ = case.step(kv, toks, par, want_logits=False)
    # commit the deepest node's path whatever was accepted
    info = ov.tree_info(par)
    deepest = int(np.argmax(info.depth))
    path = list(info.ancestors[deepest])
    acc.accept_len = len(path)
    for k, node in enumerate(path):
        acc.path[k] = node
    dv.dv_kv_commit(case.h, kv.c, acc)
    st = ov.forward_tree(om, kv_o, toks, par)
    kv_o2 = ov.commit(kv_o, st["new_k"], st["new_v"], path)
    # next step on both sides from their own caches
    toks2, par2 = synth.random_tree(96, 9, 4, case.cfg.vocab)
    ref = _ref(om, kv_o2, toks2, par2)
    acc2, lg2 = case.step(kv, toks2, par2)
    compare_step(acc2, lg2, ref, 2e-2)


def test_verify_commit_loop_is_lossless():
    """fp32 model: verify + commit over planted trees emits the oracle's greedy sequence."""
    cfg = small_cfg(n_layers=2, d_model=128, n_heads=2, head_dim=64, d_ffn=256, vocab=256,
                    weight_dtype="f32", init_std=0.05)
    case = GpuCase(cfg, seed=101, capacity=256)
    try:
        om = case.w.oracle()
        kv = case.new_kv()
        prompt = synth.prompt(102, 20, cfg.vocab)
        root = dv.dv_prefill(case.h, prompt, kv.c)
        kv_o, pre = ov.prefill(om, prompt)
        assert root == int(ov.argmax_lowest(pre[-1:])[0])
        n_total = 40
        greedy, _ = ov.greedy_decode(om, kv_o, root, n_total + 8)
        rng = np.random.default_rng(7)
        emitted, pend = [], root
        while len(emitted) < n_total:
            i0 = len(emitted)
            depth_true = int(rng.integers(1, 7))
            toks, par = [greedy[i0]], [-1]
            for k in range(1, depth_true):
                toks.append(greedy[i0 + k])
                par.append(len(toks) - 2)
            while len(toks) < 12:
                par.append(int(rng.integers(0, len(toks))))
                toks.append(int(rng.integers(0, cfg.vocab)))
            assert toks[0] == pend
            acc, _ = case.step(kv, np.array(toks), np.array(par), want_logits=False)
            assert acc.accept_len >= depth_true
            emitted.extend(toks[j] for j in acc.path_list)
            dv.dv_kv_commit(case.h, kv.c, acc)
            pend = acc.bonus_token
        assert emitted[:n_total] == greedy[:n_total]
    finally:
        case.close()


# ---------------------------------------------------------------------------
# error paths on a live handle: codes returned, nothing changed, handle usable

def test_error_paths_leave_state_untouched(bf16_case):
    case = bf16_case
    kv = case.new_kv()
    case.synthetic_context(kv, 97, 20)
    toks, par = synth.random_tree(98, 8, 4, case.cfg.vocab)

    def code(fn, *a):
        with pytest.raises(dv.DvError) as e:
            fn(*a)
        return e.value.code

    assert code(dv.dv_kv_commit, case.h, kv.c, dv.dv_accept()) == dv.DV_ESTATE
    bad = toks.copy()
    bad[3] = case.cfg.vocab
    assert code(case.step, kv, bad, par) == dv.DV_EINVAL
    assert code(case.step, kv, toks, np.array([0] + list(par[1:]))) == dv.DV_EINVAL
    kv.c.len = case.capacity - 4
    assert code(case.step, kv, toks, par) == dv.DV_ECAPACITY
    kv.c.len = 20
    acc, _ = case.step(kv, toks, par)
    wrong = dv.dv_accept.from_buffer_copy(acc)
    wrong.base_len = 21
    assert code(dv.dv_kv_commit, case.h, kv.c, wrong) == dv.DV_ESTATE
    wrong = dv.dv_accept.from_buffer_copy(acc)
    wrong.accept_len = 2
    wrong.path[1] = 7 if par[7] != 0 else 6
    if par[wrong.path[1]] != 0:
        assert code(dv.dv_kv_commit, case.h, kv.c, wrong) == dv.DV_EINVAL
    assert kv.len == 20
    dv.dv_kv_commit(case.h, kv.c, acc)
    assert kv.len == 20 + acc.accept_len
    assert code(dv.dv_kv_commit, case.h, kv.c, acc) == dv.DV_ESTATE
    acc2, _ = case.step(kv, toks, par)          # still usable
    assert acc2.base_len == kv.len
