"""Parity at the full Llama-7B/13B shapes, in the launch configuration the
benchmark times (same workload definitions, seeds, tree generator and KV
capacity rule as bench.py), against the float64 oracle on the same bytes.

Every node's logits of the step are computed by the oracle (a 13B pass takes
a few minutes of host time), so these are the slowest GPU tests.
"""
import os
import time

import numpy as np
import pytest

import synth
from oracle import verify as ov
from tests.helpers import compare_step

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2412_18934_amd import device as D  # noqa: E402
from paper_2412_18934_amd import dv  # noqa: E402


def _say(msg):
    print("[fullsize] " + msg, flush=True)


class _Model:
    """One set of full-size weights on the GPU and on the host (bf16 bits, or
    int8 codes with row scales)."""

    def __init__(self, mc, seed):
        t0 = time.time()
        self.mc = mc
        self.layers = [synth.layer_weights(mc, seed, l) for l in range(mc.n_layers)]
        self.embed = synth.embed(mc, seed)
        self.lm = synth.lm_head(mc, seed)
        self.lm_s = synth.lm_head_scale(mc, seed)
        self.fn = synth.final_norm(mc, seed)
        self.dev = D.DeviceWeights(mc.n_layers, lambda l: self.layers[l], self.embed, self.lm, self.fn,
                                   lm_head_scale=self.lm_s)
        self.om = ov.OracleModel(mc, lambda l: self.layers[l], lambda ids: self.embed[ids],
                                 self.lm, self.fn, lm_head_scale=self.lm_s)
        _say("weights ready in %.0f s" % (time.time() - t0))

    def run(self, wl, m=None):
        mc, sd = wl.model, wl.seeds
        m = m or wl.n_tree
        p = wl.context
        cap = p + 64                       # as bench.py
        kv = D.DeviceKV(mc.n_layers, mc.n_heads, mc.head_dim, cap, mc.weight_dtype)
        raw = []
        for l in range(mc.n_layers):
            k, v = synth.kv_layer(mc, sd["kv"], l, p)
            kv.set_layer(l, k, v)
            raw.append((k, v))
        kv.c.len = p
        toks, par = synth.random_tree(sd["tree"], m, wl.depth, mc.vocab, chain=wl.chain)
        cfg = D.make_config(mc.n_layers, mc.d_model, mc.n_heads, mc.head_dim, mc.d_ffn, mc.vocab,
                            mc.rms_eps, mc.rope_base, mc.weight_dtype, cap, 64)
        h = dv.dv_verify_init(cfg, self.dev.c, torch.cuda.current_stream().cuda_stream)
        try:
            logits = torch.empty((m, mc.vocab), dtype=torch.float32, device="cuda:0")
            acc = dv.dv_verify_step(h, toks, par, kv.c, logits.data_ptr())
            torch.cuda.synchronize()
            gl = logits.cpu().numpy()
        finally:
            dv.dv_verify_free(h)
        del kv
        t0 = time.time()
        ref = ov.verify_step(self.om, ov.kv_from_raw(raw), toks, par)
        ref["tokens"], ref["parents"] = toks, par
        _say("%s M=%d: oracle %.0f s" % (wl.name, m, time.time() - t0))
        err, near = compare_step(acc, gl, ref, 2e-2)
        _say("%s M=%d: logits max-abs err %.3g, near-ties %d, accept_len %d"
             % (wl.name, m, err, near, acc.accept_len))
        return err, near


@pytest.fixture(scope="module")
def llama13b():
    wl = synth.WORKLOADS["llama13b-bf16-m16-ctx1024"]
    model = _Model(wl.model, wl.seeds["weights"])
    yield model
    del model
    torch.cuda.empty_cache()


def test_llama13b_m16_ctx1024(llama13b):
    llama13b.run(synth.WORKLOADS["llama13b-bf16-m16-ctx1024"])


@pytest.mark.parametrize("m", [1, 2, 4, 8, 32, 64])
def test_llama13b_sweep_extremes(llama13b, m):
    wl = synth.sweep_workload(m)
    assert wl.model == llama13b.mc
    llama13b.run(wl)


def test_llama13b_ctx8192(llama13b):
    llama13b.run(synth.WORKLOADS["llama13b-bf16-ctx8192"])


def test_llama13b_prefill_1024(llama13b):
    """Large-M prefill of a 1024-token prompt at the 13B shape (the prompt
    bench.py times): layer-0 keys and values of sampled tokens against the
    oracle computed token by token, and the split property (600 + 424 tokens
    in two calls write the cache one call writes) on the first, a middle and
    the last layer."""
    m = llama13b
    mc = m.mc
    n = 1024
    cap = n + 64
    prompt = synth.prompt(303, n, mc.vocab)
    cfg = D.make_config(mc.n_layers, mc.d_model, mc.n_heads, mc.head_dim, mc.d_ffn, mc.vocab,
                        mc.rms_eps, mc.rope_base, mc.weight_dtype, cap, 64)
    h = dv.dv_verify_init(cfg, m.dev.c, torch.cuda.current_stream().cuda_stream)
    try:
        kv = D.DeviceKV(mc.n_layers, mc.n_heads, mc.head_dim, cap, mc.weight_dtype)
        dv.dv_prefill(h, prompt, kv.c)
        kv2 = D.DeviceKV(mc.n_layers, mc.n_heads, mc.head_dim, cap, mc.weight_dtype)
        dv.dv_prefill(h, prompt[:600], kv2.c)
        dv.dv_prefill(h, prompt[600:], kv2.c)
        assert kv.c.len == kv2.c.len == n
        w0 = m.om.layer(0, np.float64)
        idx = np.array([0, 1, 17, 511, 600, 1023])
        u = ov.rmsnorm(ov.bf16_to_f64(m.embed[prompt[idx]]), w0["attn_norm"], mc.rms_eps)
        hh, hd = mc.n_heads, mc.head_dim
        k_ref = ov.round_cache(ov.rope((u @ w0["wk"].T).reshape(len(idx), hh, hd), idx, mc.rope_base), "bf16")
        v_ref = ov.round_cache((u @ w0["wv"].T).reshape(len(idx), hh, hd), "bf16")
        k, v = kv.layer_host(0, n)
        for got, want in ((k, k_ref), (v, v_ref)):
            got = ov.bf16_to_f64(got[:, idx])                  # [H][len(idx)][hd]
            want = np.transpose(want, (1, 0, 2))
            rms = np.sqrt(np.mean(want ** 2))
            np.testing.assert_allclose(got, want, rtol=2 ** -7, atol=1e-4 * rms)
        # the two calls run other GEMM shapes (other summation orders), so
        # entries near a bf16 rounding midpoint can round apart; the first
        # layers keep the row bar, deep layers (where those one-step
        # differences have passed through many attention layers) a
        # statistical one: median and tail of |difference| / RMS
        for l in (0, 1, 2, 20, mc.n_layers - 1):
            a, b = kv.layer_host(l, n), kv2.layer_host(l, n)
            for x, y in zip(a, b):
                x, y = ov.bf16_to_f64(x), ov.bf16_to_f64(y)
                rms = np.sqrt(np.mean(x ** 2))
                if l <= 2:
                    np.testing.assert_allclose(x, y, rtol=2 ** -6, atol=(1e-4 if l == 0 else 1e-2) * rms)
                else:
                    dif = np.abs(x - y) / rms
                    assert np.median(dif) <= 1e-3 and dif.max() <= 5e-2, (l, np.median(dif), dif.max())
        _say("prefill 1024 at 13B: sampled layer-0 rows and the split property hold")
    finally:
        dv.dv_verify_free(h)


def test_llama13b_int8_m16_ctx1024():
    """The weight-only int8 13B workload bench.py times beside the headline."""
    wl = synth.WORKLOADS["llama13b-i8-m16-ctx1024"]
    model = _Model(wl.model, wl.seeds["weights"])
    model.run(wl)
    del model
    torch.cuda.empty_cache()


@pytest.mark.parametrize("m", [16, 11])
def test_llama7b_width_two_layers(m):
    """Two layers at the 7B widths with one full or ragged 16-token tile (the
    8-node workload below runs the half-layout tile): 8-block gate/up groups
    (172 of them, fewer than the CUs) and 4-block QKV groups (192)."""
    mc = synth.shrink(synth.LLAMA7B, n_layers=2)
    wl = synth.Workload("llama7b-2l-bf16-ctx512", mc, context=512, n_tree=m, depth=6, seed_base=250,
                        weight_seed=251)
    model = _Model(wl.model, wl.seeds["weights"])
    model.run(wl)
    del model
    torch.cuda.empty_cache()


def test_llama7b_m8_ctx512():
    wl = synth.WORKLOADS["llama7b-bf16-m8-ctx512"]
    model = _Model(wl.model, wl.seeds["weights"])
    model.run(wl)
