"""Weight-only int8 verification on the GPU vs the oracle's exactly
dequantised model, through the C ABI (identical int8 codes, row scales,
bf16 embeddings/gains and cache bytes on both sides).

Bars as for bf16 weights: logits max-abs <= 2e-2 (the int8 codes are exact in
the bf16 MFMA operand; activations enter as bf16 hi + lo, accumulation fp32,
the row scale multiplies the fp32 sums), argmax / accept / path / bonus
bit-exact outside near-ties, KV rows within the bf16 rounding bound.
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


I8 = dict(n_layers=2, d_model=256, n_heads=2, head_dim=128, d_ffn=512, vocab=2048,
          weight_dtype="i8", init_std=0.09)


@pytest.fixture(scope="module")
def i8_case():
    case = GpuCase(small_cfg(**I8), seed=171, capacity=256)
    yield case
    case.close()


@pytest.mark.parametrize("m", [1, 2, 16, 17, 40, 64])
def test_int8_random_tree_parity(i8_case, m):
    case = i8_case
    om = case.w.oracle()
    p = 77
    kv = case.new_kv()
    kv_o = case.synthetic_context(kv, 172, p)
    toks, par = synth.random_tree(173 + m, m, 8, case.cfg.vocab)
    ref = _ref(om, kv_o, toks, par)
    acc, lg = case.step(kv, toks, par)
    err, near = compare_step(acc, lg, ref, 2e-2)
    assert near <= max(3, m // 3)
    for l in range(case.cfg.n_layers):
        k, v = kv.layer_host(l, p + m)
        for got, want in ((k, ref["new_k"][l]), (v, ref["new_v"][l])):
            want = np.transpose(want, (1, 0, 2))
            rms = np.sqrt(np.mean(want ** 2))
            np.testing.assert_allclose(ov.bf16_to_f64(got[:, p:]), want, rtol=2 ** -7,
                                       atol=(1e-4 if l == 0 else 5e-3) * rms)


def test_int8_planted_acceptance_and_commit(i8_case):
    case = i8_case
    om = case.w.oracle()
    kv = case.new_kv()
    kv_o = case.synthetic_context(kv, 174, 20)
    root = 11
    greedy, _ = ov.greedy_decode(om, kv_o, root, 6)
    toks, par = [root], [-1]
    for k in range(1, 5):
        toks.append(greedy[k])
        par.append(len(toks) - 2 if k > 1 else 0)
    rng = np.random.default_rng(4)
    while len(toks) < 12:
        par.append(int(rng.integers(0, len(toks))))
        toks.append(int(rng.integers(0, case.cfg.vocab)))
    toks, par = np.array(toks), np.array(par)
    ref = _ref(om, kv_o, toks, par)
    acc, lg = case.step(kv, toks, par)
    compare_step(acc, lg, ref, 2e-2)
    assert acc.accept_len >= 5
    assert acc.path_list == list(ref["path"]) and acc.bonus_token == ref["bonus"]
    # each side commits its own result (equal, as just checked)
    dv.dv_kv_commit(case.h, kv.c, acc)
    kv_o2 = ov.commit(kv_o, ref["new_k"], ref["new_v"], ref["path"])
    toks2, par2 = synth.random_tree(175, 9, 4, case.cfg.vocab)
    toks2[0] = ref["bonus"]
    ref2 = _ref(om, kv_o2, toks2, par2)
    acc2, lg2 = case.step(kv, toks2, par2)
    compare_step(acc2, lg2, ref2, 2e-2)


def test_int8_split_k_fold_and_two_block_head():
    """d_model 1024 / d_ffn 2816: split-K O and down with the fold; vocab 2080
    gives the lm_head 2-block row groups; bitwise repeatable."""
    cfg = small_cfg(n_layers=2, d_model=1024, n_heads=8, head_dim=128, d_ffn=2816, vocab=2080,
                    weight_dtype="i8", init_std=0.045)
    case = GpuCase(cfg, seed=181, capacity=320)
    try:
        om = case.w.oracle()
        kv = case.new_kv()
        kv_o = case.synthetic_context(kv, 182, 200)
        for m in (16, 40):
            toks, par = synth.random_tree(183 + m, m, 6, cfg.vocab)
            ref = _ref(om, kv_o, toks, par)
            acc, lg = case.step(kv, toks, par)
            compare_step(acc, lg, ref, 2e-2)
            acc2, lg2 = case.step(kv, toks, par)
            assert np.array_equal(lg, lg2)
    finally:
        case.close()


def test_int8_prefill_and_sampled_step(i8_case):
    """GPU prefill of a 40-token prompt (chunks through the same kernels), then
    a sampled step whose logits equal the greedy step's bitwise."""
    case = i8_case
    om = case.w.oracle()
    kv = case.new_kv()
    prompt = synth.prompt(176, 40, case.cfg.vocab)
    nxt = dv.dv_prefill(case.h, prompt, kv.c)
    ref_kv, pre = ov.prefill(om, prompt)
    want = int(ov.argmax_lowest(pre[-1:])[0])
    assert kv.c.len == 40 and nxt == want
    toks, par = synth.random_tree(177, 10, 4, case.cfg.vocab)
    toks[0] = want
    ref = _ref(om, ref_kv, toks, par)
    acc, lg = case.step(kv, toks, par)
    compare_step(acc, lg, ref, 2e-2)
    q = torch.from_numpy(synth.draft_rows(5, 10, case.cfg.vocab)).to("cuda:0")
    ua, ub = synth.sampling_uniforms(5, 10)
    out = torch.empty((10, case.cfg.vocab), device="cuda:0")
    dv.dv_verify_step_sampled(case.h, toks, par, kv.c, q.data_ptr(), 1.0, ua, ub, out.data_ptr())
    np.testing.assert_array_equal(out.cpu().numpy(), lg)
