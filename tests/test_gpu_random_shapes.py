"""GPU path vs the CPU oracle over a seeded sweep of model and tree shapes.

Each case draws head size, head count, FFN width (multiples of 16, so some
down projections take the VALU kernel; 64 for int8 weights), vocabulary,
weight type (fp32, bf16, and int8 with per-row scales), layer count,
cache capacity, committed length P (including 0), tree size M in [1, 64] and
depth.  One verify step is compared with the oracle to the same bars as the
fixed parity cases; then a random root-to-node path is committed and the
moved cache rows are checked byte for byte against the rows the step wrote.
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

N_CASES = 32   # cases 20.. use int8 weights


def _draw(i):
    rng = np.random.default_rng(9000 + i)
    hd = int(rng.choice([64, 128]))
    heads = [h for h in (1, 2, 3, 4, 5, 6, 8) if h * hd <= 1024]
    H = int(rng.choice(heads))
    d = H * hd
    F = 16 * int(rng.integers(d // 16, 3 * d // 16 + 1))
    V = 32 * int(rng.integers(32, 129))
    dtype = "f32" if rng.random() < 0.2 else "bf16"
    layers = int(rng.integers(1, 3))
    cap = 32 * int(rng.integers(3, 13))
    m = int(rng.integers(1, min(64, cap) + 1))
    p = int(rng.integers(0, cap - m + 1))
    depth = int(rng.integers(2, 10)) if m > 1 else 1
    if i % 10 == 4:
        p = 0                  # empty context
    if i % 10 == 7:
        m, depth = 1, 1        # the root alone
    if i >= 20:                # int8 weights with per-row scales
        dtype, F = "i8", 64 * max(1, F // 64)
    cfg = small_cfg(n_layers=layers, d_model=d, n_heads=H, head_dim=hd, d_ffn=F, vocab=V,
                    weight_dtype=dtype, init_std=0.09 * np.sqrt(256.0 / d))
    return cfg, cap, m, p, depth


def _random_path(parents, rng):
    """A root-to-node path (increasing node indices) ending at a random node."""
    node = int(rng.integers(0, len(parents)))
    path = []
    while node >= 0:
        path.append(node)
        node = int(parents[node])
    return path[::-1]


@pytest.mark.parametrize("i", range(N_CASES))
def test_random_shape_step_and_commit(i):
    cfg, cap, m, p, depth = _draw(i)
    print("case %d: L%d d%d H%d hd%d F%d V%d %s cap%d P%d M%d depth%d" %
          (i, cfg.n_layers, cfg.d_model, cfg.n_heads, cfg.head_dim, cfg.d_ffn, cfg.vocab,
           cfg.weight_dtype, cap, p, m, depth), flush=True)
    tol = 1e-4 if cfg.weight_dtype == "f32" else 2e-2
    case = GpuCase(cfg, seed=9100 + i, capacity=cap)
    try:
        om = case.w.oracle()
        kv = case.new_kv()
        kv_o = case.synthetic_context(kv, 9200 + i, p)
        toks, par = synth.random_tree(9300 + i, m, depth, cfg.vocab)
        ref = ov.verify_step(om, kv_o, toks, par)
        ref["tokens"], ref["parents"] = np.asarray(toks), np.asarray(par)
        acc, lg = case.step(kv, toks, par)
        _, near = compare_step(acc, lg, ref, tol)
        assert near <= max(3, m // 3)

        # commit a random path: slot p + k <- slot p + path[k], all else unchanged
        before = [kv.layer_host(l, p + m) for l in range(cfg.n_layers)]
        path = _random_path(par, np.random.default_rng(9400 + i))
        acc.accept_len = len(path)
        for k, node in enumerate(path):
            acc.path[k] = node
        dv.dv_kv_commit(case.h, kv.c, acc)
        torch.cuda.synchronize()
        assert kv.len == p + len(path)
        for l in range(cfg.n_layers):
            after = kv.layer_host(l, p + len(path))
            for which in range(2):
                b, a = before[l][which], after[which]
                assert np.array_equal(a[:, :p], b[:, :p])
                for k, node in enumerate(path):
                    assert np.array_equal(a[:, p + k], b[:, p + node])
    finally:
        case.close()
