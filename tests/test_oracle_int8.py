"""Pins of the oracle's weight-only int8 model (the int8 target of Section 4,
read as one fp32 scale per output row: W[r][c] = scale[r] * q[r][c]).

* dequantisation against values worked out by hand from that definition;
* wiring: an int8 model whose scales are powers of two equals, bit for bit in
  float64, the dense fp32 model whose weights are those exact products (built
  with ``np.ldexp``), for the logits of a tree step and the cached keys; a
  scale applied per column instead of per row breaks it;
* the seeded int8 generator: codes in [-127, 127] with the Gaussian profile it
  states, scales within their stated band.
"""
import numpy as np
import pytest

import synth
from oracle import verify as ov


def test_dequantize_rows_by_hand():
    q = np.array([[1, -2, 127], [-127, 0, 3]], dtype=np.int8)
    s = np.array([0.5, 2.0], dtype=np.float32)
    want = np.array([[0.5, -1.0, 63.5], [-254.0, 0.0, 6.0]])
    got = ov.dequantize_rows(q, s)
    assert got.dtype == np.float64
    np.testing.assert_array_equal(got, want)


def _pow2_model(cfg, seed, transpose_scale=False):
    """int8 layers with power-of-two row scales, and the dense fp32 twin."""
    q_layers, d_layers = [], []
    rng = np.random.default_rng(seed)
    for l in range(cfg.n_layers):
        raw = synth.layer_weights(cfg, seed, l)
        ql, dl = {}, {}
        for k, v in raw.items():
            if k.endswith("_scale"):
                continue
            if k + "_scale" in raw:
                e = rng.integers(6, 10, size=v.shape[0])          # scale 2^-e per row
                ql[k] = v
                ql[k + "_scale"] = np.ldexp(np.float32(1.0), -e).astype(np.float32)
                ee = e if not transpose_scale else np.resize(e, v.shape[1])
                dl[k] = (np.ldexp(v.astype(np.float32), -ee[:, None]) if not transpose_scale
                         else np.ldexp(v.astype(np.float32), -ee[None, :])).astype(np.float32)
            else:
                ql[k] = v
                dl[k] = synth.bf16_bits_to_f32(v)
        q_layers.append(ql)
        d_layers.append(dl)
    lm = synth.lm_head(cfg, seed)
    e = rng.integers(6, 10, size=lm.shape[0])
    lm_s = np.ldexp(np.float32(1.0), -e).astype(np.float32)
    lm_d = np.ldexp(lm.astype(np.float32), -e[:, None]).astype(np.float32)
    emb = synth.embed(cfg, seed)
    fn = synth.final_norm(cfg, seed)
    om_q = ov.OracleModel(cfg, lambda l: q_layers[l], lambda ids: emb[ids], lm, fn, lm_head_scale=lm_s)
    om_d = ov.OracleModel(cfg, lambda l: d_layers[l], lambda ids: synth.bf16_bits_to_f32(emb[ids]), lm_d,
                          synth.bf16_bits_to_f32(fn))
    return om_q, om_d


def test_int8_model_equals_its_dense_twin():
    cfg = synth.ModelCfg(n_layers=2, d_model=128, n_heads=2, head_dim=64, d_ffn=256, vocab=384,
                         weight_dtype="i8", init_std=0.1)
    om_q, om_d = _pow2_model(cfg, 7)
    kv = [(k, v) for k, v in (synth.kv_layer(cfg, 8, l, 9) for l in range(cfg.n_layers))]
    toks, par = synth.random_tree(9, 7, 4, cfg.vocab)
    rq = ov.verify_step(om_q, ov.kv_from_raw(kv), toks, par)
    rd = ov.verify_step(om_d, ov.kv_from_raw(kv), toks, par)
    np.testing.assert_array_equal(rq["logits"], rd["logits"])
    for l in range(cfg.n_layers):
        np.testing.assert_array_equal(rq["new_k"][l], rd["new_k"][l])


def test_scale_per_column_breaks_the_twin():
    cfg = synth.ModelCfg(n_layers=1, d_model=128, n_heads=2, head_dim=64, d_ffn=256, vocab=384,
                         weight_dtype="i8", init_std=0.1)
    om_q, om_bad = _pow2_model(cfg, 7, transpose_scale=True)
    toks, par = synth.random_tree(9, 5, 3, cfg.vocab)
    rq = ov.verify_step(om_q, ov.kv_from_raw([synth.kv_layer(cfg, 8, 0, 9)]), toks, par)
    rb = ov.verify_step(om_bad, ov.kv_from_raw([synth.kv_layer(cfg, 8, 0, 9)]), toks, par)
    assert np.abs(rq["logits"] - rb["logits"]).max() > 1e-3


def test_int8_generator_profile():
    cfg = synth.ModelCfg(n_layers=1, d_model=256, n_heads=2, head_dim=128, d_ffn=512, vocab=256,
                         weight_dtype="i8", init_std=0.02)
    w = synth.layer_weights(cfg, 3, 0)
    q = w["w_gate"].astype(np.float64)
    assert w["w_gate"].dtype == np.int8 and q.min() >= -127 and q.max() <= 127
    # rint(31.75 z) clipped at 4 sigma: std within 1% of 31.75, ~0.006% clipped
    assert abs(q.std() / synth.I8_CODE_SIGMA - 1) < 0.01
    assert abs(q.mean()) < 0.1
    s = w["w_gate_scale"]
    band = cfg.init_std / synth.I8_CODE_SIGMA
    assert s.dtype == np.float32 and s.shape == (512,)
    assert s.min() >= 0.75 * band * (1 - 1e-6) and s.max() <= 1.25 * band
    assert w["attn_norm"].dtype == np.uint16 and synth.embed(cfg, 3).dtype == np.uint16
    assert cfg.kv_dtype == "bf16"


@pytest.mark.parametrize("dtype", [np.float64, np.float32])
def test_dequantize_rows_dtype(dtype):
    q = np.array([[3, -4]], dtype=np.int8)
    s = np.array([0.25], dtype=np.float32)
    got = ov.dequantize_rows(q, s, dtype)
    assert got.dtype == dtype
    np.testing.assert_array_equal(got, np.array([[0.75, -1.0]], dtype=dtype))
