"""Draft side on the GPU vs the oracle (oracle/draft.py), through the C ABI:
the DGF + block-stack pass (dv_draft_forward) and the tree construction
(dv_draft_tree).

Bars: draft logits max-abs <= 2e-2 and output features within 5e-3 of their
RMS (bf16 weights, fp32 arithmetic, as the verify step); the constructed tree
(tokens, parents) equal to the oracle's wherever every ranking decision of the
oracle clears a relative margin of 1e-2 (the GPU ranks fp32 probabilities
from its own logits); otherwise it must still be a valid tree of the right
size, and at most one case per test may differ.
"""
import numpy as np
import pytest

import synth
from oracle import draft as od
from oracle import verify as ov
from tests.helpers import GpuCase, Weights, compare_step, small_cfg

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2412_18934_amd import device as D  # noqa: E402
from paper_2412_18934_amd import dv  # noqa: E402

TARGET = dict(n_layers=2, d_model=256, n_heads=2, head_dim=128, d_ffn=512, vocab=2048,
              weight_dtype="bf16", init_std=0.09)


class DraftCase:
    """A draft of n_blocks blocks sharing the target's embedding and lm_head."""

    def __init__(self, n_blocks, seed, capacity=128, target=TARGET):
        tcfg = small_cfg(**target)
        self.cfg = synth.draft_cfg(tcfg, n_blocks)
        tw = Weights(tcfg, seed)                 # the target's embedding / lm_head
        self.w = Weights(self.cfg, seed + 1)     # the draft's blocks
        self.w.embed, self.w.lm_head = tw.embed, tw.lm_head
        self.dgf = synth.dgf_weights(self.cfg, seed + 2)
        self.dev = D.DeviceWeights(self.cfg.n_layers, lambda l: self.w.layers[l], self.w.embed, self.w.lm_head,
                                   self.w.final_norm)
        self.dgf_dev = {k: D.to_device(v, "cuda:0") for k, v in self.dgf.items()}
        self.dgf_c = dv.dv_dgf_weights(*(self.dgf_dev[k].data_ptr() for k in ("w_hidden", "w_embed", "w_gate")))
        c = self.cfg
        self.ccfg = D.make_config(c.n_layers, c.d_model, c.n_heads, c.head_dim, c.d_ffn, c.vocab, c.rms_eps,
                                  c.rope_base, c.weight_dtype, capacity, 64)
        self.capacity = capacity
        self.h = dv.dv_draft_init(self.ccfg, self.dev.c, self.dgf_c)
        self.om = od.DraftModel(self.w.oracle(), self.dgf["w_hidden"], self.dgf["w_embed"], self.dgf["w_gate"])

    def kv(self, seed, p):
        c = self.cfg
        kv = D.DeviceKV(c.n_layers, c.n_heads, c.head_dim, self.capacity, c.weight_dtype)
        raw = [synth.kv_layer(c, seed, l, p) for l in range(c.n_layers)]
        for l, (k, v) in enumerate(raw):
            if p:
                kv.set_layer(l, k, v)
        kv.c.len = p
        return kv, ov.kv_from_raw(raw)

    def close(self):
        dv.dv_verify_free(self.h)


@pytest.fixture(scope="module")
def draft2():
    c = DraftCase(2, 301)
    yield c
    c.close()


@pytest.mark.parametrize("m", [1, 7, 20])
def test_draft_forward_matches_oracle(draft2, m):
    c = draft2
    kv, kv_o = c.kv(302, 40)
    toks, par = synth.random_tree(303 + m, m, 5, c.cfg.vocab)
    feat = synth.features(304 + m, m, c.cfg.d_model)
    f_in = torch.from_numpy(feat).to("cuda:0")
    f_out = torch.full((m, c.cfg.d_model), float("nan"), device="cuda:0")
    lg = torch.full((m, c.cfg.vocab), float("nan"), device="cuda:0")
    dv.dv_draft_forward(c.h, toks, par, kv.c, f_in.data_ptr(), f_out.data_ptr(), lg.data_ptr())
    logits, hidden = c.om.forward(kv_o, toks, par, feat)
    assert float(np.abs(lg.cpu().numpy() - logits).max()) <= 2e-2
    fo = f_out.cpu().numpy()
    rms = np.sqrt(np.mean(hidden ** 2))
    assert float(np.abs(fo - hidden).max()) <= 5e-3 * rms


def test_draft_forward_split_k_fusion():
    """d_model 1024: the gated fusion's projections split K (2 splits for W_h and
    W_e, 4 for W_g) and the last split of each row group folds them."""
    wide = dict(n_layers=2, d_model=1024, n_heads=8, head_dim=128, d_ffn=2816, vocab=4096,
                weight_dtype="bf16", init_std=0.05)
    c = DraftCase(1, 305, target=wide)
    try:
        kv, kv_o = c.kv(306, 33)
        for m in (5, 19):
            toks, par = synth.random_tree(307 + m, m, 4, c.cfg.vocab)
            feat = synth.features(308 + m, m, c.cfg.d_model)
            f_in = torch.from_numpy(feat).to("cuda:0")
            f_out = torch.full((m, c.cfg.d_model), float("nan"), device="cuda:0")
            lg = torch.full((m, c.cfg.vocab), float("nan"), device="cuda:0")
            dv.dv_draft_forward(c.h, toks, par, kv.c, f_in.data_ptr(), f_out.data_ptr(), lg.data_ptr())
            logits, hidden = c.om.forward(kv_o, toks, par, feat)
            assert float(np.abs(lg.cpu().numpy() - logits).max()) <= 2e-2
            rms = np.sqrt(np.mean(hidden ** 2))
            assert float(np.abs(f_out.cpu().numpy() - hidden).max()) <= 5e-3 * rms
            # the same pass again: bitwise reproducible
            f2 = torch.full_like(f_out, float("nan"))
            dv.dv_draft_forward(c.h, toks, par, kv.c, f_in.data_ptr(), f2.data_ptr(), lg.data_ptr())
            assert torch.equal(f_out, f2)
    finally:
        c.close()


def _clear(trace, rel=1e-2):
    return all(ev[1] > ev[2] * (1 + rel) for ev in trace)


def _valid(tok, par, n, V):
    assert len(tok) == n and par[0] == -1
    assert all(0 <= par[i] < i for i in range(1, n))
    assert all(0 <= t < V for t in tok)


@pytest.mark.parametrize("depth,width,n_tree", [(1, 3, 4), (3, 4, 10), (7, 10, 16), (4, 10, 7), (5, 16, 40)])
def test_draft_tree_matches_oracle(draft2, depth, width, n_tree):
    c = draft2
    differ = 0
    for rep in range(2):
        kv, kv_o = c.kv(310 + rep, 30)
        root = int(synth.prompt(311 + rep, 1, c.cfg.vocab)[0])
        feat = synth.features(312 + rep, 1, c.cfg.d_model)[0]
        rf = torch.from_numpy(feat).to("cuda:0")
        tok, par, sc = dv.dv_draft_tree(c.h, root, rf.data_ptr(), kv.c, depth, width, n_tree)
        trace = []
        otok, opar, osc = od.build_tree(lambda t, p, f: c.om.forward(kv_o, t, p, f), root, feat, depth, width,
                                        n_tree, trace=trace)
        _valid(tok, par, len(otok), c.cfg.vocab)
        same = list(tok) == list(otok) and list(par) == list(opar)
        if same:
            np.testing.assert_allclose(sc, osc, rtol=1e-2)
        else:
            assert not _clear(trace), "trees differ although every ranking decision was clear"
            differ += 1
    assert differ <= 1


def test_draft_tree_feeds_a_verify_step(draft2):
    """The constructed tree is a valid input of the target's verify step (the
    target here is the draft's own target-shaped model), and construction is
    deterministic."""
    c = draft2
    kv, _ = c.kv(320, 25)
    root = 17
    rf = torch.from_numpy(synth.features(321, 1, c.cfg.d_model)[0]).to("cuda:0")
    t1 = dv.dv_draft_tree(c.h, root, rf.data_ptr(), kv.c, 6, 8, 16)
    t2 = dv.dv_draft_tree(c.h, root, rf.data_ptr(), kv.c, 6, 8, 16)
    assert all(np.array_equal(a, b) for a, b in zip(t1, t2))
    tcfg = small_cfg(**TARGET)
    tgt = GpuCase(tcfg, seed=301, capacity=128)
    try:
        tkv = tgt.new_kv()
        kv_o = tgt.synthetic_context(tkv, 322, 25)
        toks, par = t1[0], t1[1]
        ref = ov.verify_step(tgt.w.oracle(), kv_o, toks, par)
        ref["tokens"], ref["parents"] = toks, par
        acc, lg = tgt.step(tkv, toks, par)
        compare_step(acc, lg, ref, 2e-2)
    finally:
        tgt.close()


def test_draft_error_paths(draft2):
    c = draft2
    kv, _ = c.kv(330, 10)
    rf = torch.zeros(c.cfg.d_model, device="cuda:0")
    for args in [(5, 17, 10), (5, 4, 65), (0, 4, 10), (3, 0, 10)]:
        with pytest.raises(dv.DvError) as e:
            dv.dv_draft_tree(c.h, 1, rf.data_ptr(), kv.c, *args)
        assert e.value.code == dv.DV_EINVAL
    with pytest.raises(dv.DvError) as e:
        dv.dv_draft_tree(c.h, c.cfg.vocab, rf.data_ptr(), kv.c, 3, 4, 10)
    assert e.value.code == dv.DV_EINVAL
    tgt = GpuCase(small_cfg(**TARGET), seed=1, capacity=64)
    try:
        with pytest.raises(dv.DvError) as e:
            dv.dv_draft_tree(tgt.h, 1, rf.data_ptr(), kv.c, 3, 4, 10)
        assert e.value.code == dv.DV_ESTATE
    finally:
        tgt.close()
    kv_small, _ = c.kv(331, 120)
    with pytest.raises(dv.DvError) as e:
        dv.dv_draft_tree(c.h, 1, rf.data_ptr(), kv_small.c, 3, 4, 10)
    assert e.value.code == dv.DV_ECAPACITY
