"""C-ABI checks that need no GPU: the library loads, exports what include/dv.h
declares, validates configs, trees and handles before touching the device,
and its host tree preprocessing agrees with the oracle's definition."""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import verify as ov
from paper_2412_18934_amd import dv
from tests.helpers import all_parent_arrays

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "dv.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(dv_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    lib = dv.lib()
    names = _declared()
    assert set(names) == set(dv.EXPORTS), names
    for n in names:
        assert hasattr(lib, n), n


def test_tree_prepare_matches_oracle_definition():
    rng = np.random.default_rng(0)
    cases = [p for m in range(1, 6) for p in all_parent_arrays(m)]
    for m in (16, 33, 64):
        par = [-1] + [int(rng.integers(0, i)) for i in range(1, m)]
        cases.append(np.array(par))
    for par in cases:
        base = int(rng.integers(0, 1000))
        pos, depth, anc = dv.dv_tree_prepare(par, base)
        info = ov.tree_info(par)
        assert list(depth) == list(info.depth)
        assert list(pos) == list(base + info.depth - 1)
        for i in range(len(par)):
            bits = [j for j in range(len(par)) if (int(anc[i]) >> j) & 1]
            assert bits == list(info.ancestors[i])


@pytest.mark.parametrize("par", [[0], [-1, 1], [-1, -1], [-1, 0, 3], [-1, 0, -2], [], list(range(-1, 64))])
def test_tree_prepare_rejects_bad_trees(par):
    with pytest.raises(dv.DvError) as e:
        dv.dv_tree_prepare(par, 0)
    assert e.value.code == dv.DV_EINVAL


def test_tree_prepare_accepts_64_node_chain():
    pos, depth, anc = dv.dv_tree_prepare(list(range(-1, 63)), 5)
    assert depth[-1] == 64 and pos[-1] == 68 and int(anc[-1]) == (1 << 64) - 1


def _good_cfg(**kw):
    c = dict(n_layers=2, d_model=256, n_heads=4, head_dim=64, d_ffn=688, vocab=1024,
             rms_eps=1e-6, rope_base=10000.0, weight_dtype=dv.DV_F32, max_ctx=128, max_tree=64)
    c.update(kw)
    return dv.dv_config(**c)


def _fake_weights(n_layers=2):
    # non-null dummy addresses: validation must reject configs before any use
    tab = (ctypes.c_void_p * n_layers)(*([0x1000] * n_layers))
    pp = ctypes.cast(tab, ctypes.POINTER(ctypes.c_void_p))
    w = dv.dv_weights(0x1000, 0x1000, 0x1000, pp, pp, pp, pp, pp, pp, pp, pp, pp)
    return w, tab


@pytest.mark.parametrize("bad", [
    dict(head_dim=96), dict(n_heads=3), dict(d_model=250, n_heads=5, head_dim=50),
    dict(vocab=1000), dict(d_ffn=680), dict(d_model=8448, n_heads=66, head_dim=128), dict(max_tree=65), dict(max_tree=0),
    dict(max_ctx=10), dict(weight_dtype=7), dict(rope_base=0.0), dict(rms_eps=-1.0),
    dict(n_layers=0),
])
def test_init_rejects_bad_config_before_device_use(bad):
    w, tab = _fake_weights()
    with pytest.raises(dv.DvError) as e:
        dv.dv_verify_init(_good_cfg(**bad), w)
    assert e.value.code == dv.DV_EINVAL
    assert dv.dv_last_error(None)


def test_init_rejects_null_weight_pointer():
    w, tab = _fake_weights()
    tab[1] = None
    with pytest.raises(dv.DvError) as e:
        dv.dv_verify_init(_good_cfg(), w)
    assert e.value.code == dv.DV_EINVAL and "layer 1" in str(e.value)


def _header_fields(name):
    src = open(os.path.join(ROOT, "include", "dv.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    body = re.search(r"typedef struct %s \{(.*?)\} %s;" % (name, name), src, flags=re.S).group(1)
    return re.findall(r"(\w+)\s*(?:\[[^\]]*\])?\s*;", body)


@pytest.mark.parametrize("name", ["dv_config", "dv_weights", "dv_kv", "dv_accept"])
def test_binding_structs_follow_the_header(name):
    assert [f[0] for f in getattr(dv, name)._fields_] == _header_fields(name)


def test_int8_config_needs_64_multiples_and_scales():
    w, tab = _fake_weights()
    with pytest.raises(dv.DvError) as e:   # d_ffn 688 is not a multiple of 64
        dv.dv_verify_init(_good_cfg(weight_dtype=dv.DV_I8), w)
    assert e.value.code == dv.DV_EINVAL and "64" in str(e.value)
    with pytest.raises(dv.DvError) as e:   # no scale tables
        dv.dv_verify_init(_good_cfg(weight_dtype=dv.DV_I8, d_ffn=704), w)
    assert e.value.code == dv.DV_EINVAL and "scale" in str(e.value)
    pp = ctypes.cast(tab, ctypes.POINTER(ctypes.c_void_p))
    w.lm_head_scale = 0x1000
    for f in ("wq_scale", "wk_scale", "wv_scale", "wo_scale", "w_gate_scale", "w_up_scale"):
        setattr(w, f, pp)
    with pytest.raises(dv.DvError) as e:   # w_down_scale still missing
        dv.dv_verify_init(_good_cfg(weight_dtype=dv.DV_I8, d_ffn=704), w)
    assert e.value.code == dv.DV_EINVAL and "scale" in str(e.value)


def test_calls_on_null_handle_fail_cleanly():
    L = dv.lib()
    kv = dv.dv_kv(0, 0, 0, 0)
    acc = dv.dv_accept()
    t = np.zeros(1, np.int32)
    p = np.array([-1], np.int32)
    assert L.dv_verify_step(None, dv._ptr(t), dv._ptr(p), 1, ctypes.byref(kv), None,
                            ctypes.byref(acc)) == dv.DV_EINVAL
    assert L.dv_kv_commit(None, ctypes.byref(kv), ctypes.byref(acc)) == dv.DV_EINVAL
    assert L.dv_prefill(None, dv._ptr(t), 1, ctypes.byref(kv), None) == dv.DV_EINVAL
    assert L.dv_profile_enable(None, 1) == dv.DV_EINVAL
    u = np.zeros(1, np.float32)
    assert L.dv_verify_step_sampled(None, dv._ptr(t), dv._ptr(p), 1, ctypes.byref(kv), None, 1.0,
                                    dv._fptr(u), dv._fptr(u), None, ctypes.byref(acc)) == dv.DV_EINVAL
    assert L.dv_accept_sampled(None, None, dv._ptr(t), dv._ptr(p), 1, None, 1.0, dv._fptr(u), dv._fptr(u),
                               ctypes.byref(acc)) == dv.DV_EINVAL
    L.dv_verify_free(None)


def test_noalloc_sampling_validates_before_device_use():
    """dv_accept_sampled_noalloc checks its arguments before any HIP call, so
    these run without a GPU."""
    L = dv.lib()
    acc = dv.dv_accept()
    t = np.zeros(1, np.int32)
    p = np.array([-1], np.int32)
    u = np.full(1, 0.5, np.float32)
    fake = ctypes.c_void_p(1 << 20)   # aligned, never dereferenced on these paths
    for vocab in (dv.DV_NOALLOC_MAX_VOCAB + 4, 6, 0):
        assert L.dv_accept_sampled_noalloc(fake, dv._ptr(t), dv._ptr(p), 1, vocab, fake, 1.0, dv._fptr(u),
                                           dv._fptr(u), None, ctypes.byref(acc)) == dv.DV_EINVAL
    assert "limit" not in dv.dv_last_error(None)
    assert L.dv_accept_sampled_noalloc(fake, dv._ptr(t), dv._ptr(p), 1, dv.DV_NOALLOC_MAX_VOCAB + 4, fake, 1.0,
                                       dv._fptr(u), dv._fptr(u), None, ctypes.byref(acc)) == dv.DV_EINVAL
    assert "limit" in dv.dv_last_error(None)
    assert L.dv_accept_sampled_noalloc(None, dv._ptr(t), dv._ptr(p), 1, 1024, fake, 1.0, dv._fptr(u),
                                       dv._fptr(u), None, ctypes.byref(acc)) == dv.DV_EINVAL
