"""Shared test helpers: small models built from the seeded generator."""
import numpy as np

import synth
from oracle.verify import OracleModel


def small_cfg(**kw):
    base = dict(n_layers=2, d_model=64, n_heads=4, head_dim=16, d_ffn=96, vocab=128,
                weight_dtype="f32", init_std=0.1)
    base.update(kw)
    return synth.ModelCfg(**base)


class Weights:
    """All weights of a model generated once, kept as stored arrays."""

    def __init__(self, cfg, seed):
        self.cfg = cfg
        self.seed = seed
        self.layers = [synth.layer_weights(cfg, seed, l) for l in range(cfg.n_layers)]
        self.embed = synth.embed(cfg, seed)
        self.lm_head = synth.lm_head(cfg, seed)
        self.final_norm = synth.final_norm(cfg)

    def oracle(self):
        return OracleModel(self.cfg, lambda l: self.layers[l], lambda ids: self.embed[ids],
                           self.lm_head, self.final_norm)


def all_parent_arrays(m):
    """Every valid parents array of an m-node tree (parents[i] in [0, i))."""
    out = [[-1]]
    for i in range(1, m):
        out = [p + [j] for p in out for j in range(i)]
    return [np.array(p, dtype=np.int32) for p in out]
