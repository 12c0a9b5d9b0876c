"""The allocation-free sampling entry point (dv_accept_sampled_noalloc, its
workspace a fixed per-GPU array of the library) against the handle-based
dv_accept_sampled on the same device inputs, through the C ABI.

Both run the same kernel, so path, accept length and bonus must be equal.
The allocation-free calls come two in a row, the second with a smaller tree
and vocabulary, so the second runs on a workspace that still holds the first
call's rows."""
import numpy as np
import pytest

import synth
from tests.helpers import GpuCase, small_cfg

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2412_18934_amd import dv  # noqa: E402


def _inputs(seed, m, V):
    """Target logits, draft rows, a seeded tree whose child tokens are drawn
    from their parent's draft row, and the walk's uniforms."""
    logits = synth.normal(seed, 90, m * V, 2.0, "f32").reshape(m, V)
    q = synth.draft_rows(seed, m, V, sharp=4.0)
    _, par = synth.random_tree(seed, m, 6, V)
    rng = np.random.default_rng(seed)
    toks = np.zeros(m, dtype=np.int32)
    toks[0] = int(rng.integers(0, V))
    for c in range(1, m):
        row = q[par[c]].astype(np.float64)
        toks[c] = int(rng.choice(V, p=row / row.sum()))
    ua, ub = synth.sampling_uniforms(seed, m)
    return logits, q, toks, par, ua, ub


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda:0")


def test_noalloc_equals_handle_entry_point_on_two_calls():
    cases = [(71, 33, 32000, 1.0), (72, 7, 8224, 0.7)]      # the second call is smaller
    ins, refs = [], []
    for seed, m, V, T in cases:
        case = GpuCase(small_cfg(n_layers=1, d_model=64, n_heads=1, head_dim=64, d_ffn=96, vocab=V),
                       seed=5, capacity=64)
        try:
            logits, q, toks, par, ua, ub = _inputs(seed, m, V)
            lg, qd = _dev(logits), _dev(q)
            refs.append(dv.dv_accept_sampled(case.h, lg.data_ptr(), toks, par, qd.data_ptr(), T, ua, ub))
            ins.append((lg, qd, toks, par, V, T, ua, ub))
        finally:
            case.close()
    stream = torch.cuda.current_stream().cuda_stream
    got = [dv.dv_accept_sampled_noalloc(lg.data_ptr(), toks, par, V, qd.data_ptr(), T, ua, ub, stream)
           for lg, qd, toks, par, V, T, ua, ub in ins]
    for (seed, m, V, T), r, g in zip(cases, refs, got):
        print("[noalloc] seed %d M=%d V=%d: path %s bonus %d (handle: %s %d)"
              % (seed, m, V, g.path_list, g.bonus_token, r.path_list, r.bonus_token), flush=True)
        assert g.accept_len == r.accept_len and g.path_list == r.path_list
        assert g.bonus_token == r.bonus_token
        assert g.n_tree == m and g.base_len == -1
    # not every case may stop at the root, or the comparison says little
    assert max(r.accept_len for r in refs) > 1


def test_noalloc_rejects_vocab_beyond_its_workspace():
    V = dv.DV_NOALLOC_MAX_VOCAB + 4
    lg = torch.zeros((1, V), dtype=torch.float32, device="cuda:0")
    with pytest.raises(dv.DvError) as e:
        dv.dv_accept_sampled_noalloc(lg.data_ptr(), [0], [-1], V, lg.data_ptr(), 1.0, [0.5], [0.5])
    assert e.value.code == dv.DV_EINVAL and "limit" in str(e.value)
