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
        self.fn = synth.final_norm(mc)
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


@pytest.mark.parametrize("m", [1, 64])
def test_llama13b_sweep_extremes(llama13b, m):
    wl = synth.sweep_workload(m)
    assert wl.model == llama13b.mc
    llama13b.run(wl)


def test_llama13b_ctx8192(llama13b):
    llama13b.run(synth.WORKLOADS["llama13b-bf16-ctx8192"])


def test_llama13b_int8_m16_ctx1024():
    """The weight-only int8 13B workload bench.py times beside the headline."""
    wl = synth.WORKLOADS["llama13b-i8-m16-ctx1024"]
    model = _Model(wl.model, wl.seeds["weights"])
    model.run(wl)
    del model
    torch.cuda.empty_cache()


def test_llama7b_m8_ctx512():
    wl = synth.WORKLOADS["llama7b-bf16-m8-ctx512"]
    model = _Model(wl.model, wl.seeds["weights"])
    model.run(wl)
