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
        self.lm_head_scale = synth.lm_head_scale(cfg, seed)
        self.final_norm = synth.final_norm(cfg, seed)

    def oracle(self):
        return OracleModel(self.cfg, lambda l: self.layers[l], lambda ids: self.embed[ids],
                           self.lm_head, self.final_norm, lm_head_scale=self.lm_head_scale)


def all_parent_arrays(m):
    """Every valid parents array of an m-node tree (parents[i] in [0, i))."""
    out = [[-1]]
    for i in range(1, m):
        out = [p + [j] for p in out for j in range(i)]
    return [np.array(p, dtype=np.int32) for p in out]


# ---------------------------------------------------------------------------
# GPU-side case: the same seeded arrays uploaded for the C ABI and handed to
# the oracle.

class GpuCase:
    def __init__(self, cfg, seed, capacity, max_tree=64, max_ctx=None, weights=None):
        import torch  # noqa: F401
        from paper_2412_18934_amd import device as D
        from paper_2412_18934_amd import dv
        self.cfg = cfg
        self.w = weights or Weights(cfg, seed)
        self.capacity = capacity
        self.dev = D.DeviceWeights(cfg.n_layers, lambda l: self.w.layers[l], self.w.embed,
                                   self.w.lm_head, self.w.final_norm, lm_head_scale=self.w.lm_head_scale)
        self.ccfg = D.make_config(cfg.n_layers, cfg.d_model, cfg.n_heads, cfg.head_dim, cfg.d_ffn,
                                  cfg.vocab, cfg.rms_eps, cfg.rope_base, cfg.weight_dtype,
                                  max_ctx or capacity, max_tree)
        self.h = dv.dv_verify_init(self.ccfg, self.dev.c)

    def new_kv(self, fill=None):
        from paper_2412_18934_amd import device as D
        c = self.cfg
        return D.DeviceKV(c.n_layers, c.n_heads, c.head_dim, self.capacity, c.weight_dtype,
                          fill=fill)

    def synthetic_context(self, kv, seed, p):
        """Fill kv with p seeded entries; returns the oracle's float64 view."""
        import synth
        from oracle.verify import kv_from_raw
        raw = [synth.kv_layer(self.cfg, seed, l, p) for l in range(self.cfg.n_layers)]
        for l, (k, v) in enumerate(raw):
            if p:
                kv.set_layer(l, k, v)
        kv.c.len = p
        return kv_from_raw(raw)

    def step(self, kv, tokens, parents, want_logits=True):
        import torch
        from paper_2412_18934_amd import dv
        logits = None
        ptr = 0
        if want_logits:
            logits = torch.full((len(tokens), self.cfg.vocab), float("nan"), dtype=torch.float32,
                                device="cuda:0")
            ptr = logits.data_ptr()
        acc = dv.dv_verify_step(self.h, tokens, parents, kv.c, ptr)
        torch.cuda.synchronize()
        return acc, (logits.cpu().numpy() if logits is not None else None)

    def close(self):
        from paper_2412_18934_amd import dv
        dv.dv_verify_free(self.h)
        self.h = None


def top2_gap(logits_row):
    z = np.sort(np.asarray(logits_row, dtype=np.float64))
    return float(z[-1] - z[-2])


def compare_step(acc, gpu_logits, ref, tol, tie_margin=None):
    """Element-wise logits within tol; argmax equal wherever the oracle's top-2
    gap exceeds tie_margin (default 2 tol), and otherwise a valid maximiser;
    acceptance equal to the greedy rule applied to the GPU's argmax.
    Returns (max abs error, number of near-tie nodes)."""
    from oracle.verify import greedy_accept
    tie_margin = 2 * tol if tie_margin is None else tie_margin
    err = float(np.abs(gpu_logits - ref["logits"]).max())
    assert np.all(np.isfinite(gpu_logits))
    assert err <= tol, "logits max-abs error %g > %g" % (err, tol)
    g_am = acc.argmax_array()
    near = 0
    for i, row in enumerate(ref["logits"]):
        if top2_gap(row) > tie_margin:
            assert g_am[i] == ref["argmax"][i], (i, g_am[i], ref["argmax"][i])
        else:
            near += 1
            assert row[g_am[i]] >= row.max() - tie_margin
    n, path, bonus = greedy_accept(ref["tokens"], ref["parents"], g_am)
    assert acc.accept_len == n and acc.path_list == list(path) and acc.bonus_token == bonus
    if near == 0:
        assert acc.accept_len == ref["accept_len"] and acc.path_list == list(ref["path"])
    return err, near
