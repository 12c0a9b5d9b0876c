"""ctypes binding of libdv.so (include/dv.h), same names as the C ABI.

Argument marshalling only: device buffers are passed as raw addresses
(``tensor.data_ptr()``), host arrays as numpy int32 arrays.  Every step of the
verification runs in the HIP kernels of libdv.so; if the library is missing
this module raises instead of falling back to anything else.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libdv.so")

DV_OK, DV_EINVAL, DV_ECAPACITY, DV_ESTATE, DV_EHIP, DV_ENOMEM = 0, -1, -2, -3, -4, -5
DV_F32, DV_BF16, DV_I8 = 0, 1, 2
DV_MAX_TREE = 64
DV_NOALLOC_MAX_VOCAB = 262144
DV_K_GEMM, DV_K_ATTN, DV_K_NORM, DV_K_OTHER = 0, 1, 2, 3

# every symbol include/dv.h declares
EXPORTS = ("dv_verify_init", "dv_verify_step", "dv_verify_step_sampled", "dv_accept_sampled",
           "dv_accept_sampled_noalloc",
           "dv_draft_init", "dv_draft_forward", "dv_draft_tree",
           "dv_kv_commit", "dv_prefill", "dv_verify_free", "dv_last_error", "dv_tree_prepare",
           "dv_profile_enable", "dv_profile_read")


class DvError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__("%s (code %d)" % (msg, code))
        self.code = code


class dv_config(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32),
                ("n_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("d_ffn", ctypes.c_int32), ("vocab", ctypes.c_int32),
                ("rms_eps", ctypes.c_float), ("rope_base", ctypes.c_float),
                ("weight_dtype", ctypes.c_int32), ("max_ctx", ctypes.c_int32),
                ("max_tree", ctypes.c_int32)]


_PP = ctypes.POINTER(ctypes.c_void_p)


class dv_weights(ctypes.Structure):
    _fields_ = [("embed", ctypes.c_void_p), ("final_norm", ctypes.c_void_p),
                ("lm_head", ctypes.c_void_p), ("attn_norm", _PP), ("wq", _PP), ("wk", _PP),
                ("wv", _PP), ("wo", _PP), ("ffn_norm", _PP), ("w_gate", _PP), ("w_up", _PP),
                ("w_down", _PP), ("lm_head_scale", ctypes.c_void_p), ("wq_scale", _PP),
                ("wk_scale", _PP), ("wv_scale", _PP), ("wo_scale", _PP), ("w_gate_scale", _PP),
                ("w_up_scale", _PP), ("w_down_scale", _PP)]


class dv_dgf_weights(ctypes.Structure):
    _fields_ = [("w_hidden", ctypes.c_void_p), ("w_embed", ctypes.c_void_p), ("w_gate", ctypes.c_void_p)]


class dv_kv(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p),
                ("capacity", ctypes.c_int32), ("len", ctypes.c_int32)]


class dv_accept(ctypes.Structure):
    _fields_ = [("accept_len", ctypes.c_int32), ("path", ctypes.c_int32 * DV_MAX_TREE),
                ("bonus_token", ctypes.c_int32), ("n_tree", ctypes.c_int32),
                ("base_len", ctypes.c_int32), ("argmax", ctypes.c_int32 * DV_MAX_TREE)]

    @property
    def path_list(self):
        return [int(self.path[i]) for i in range(self.accept_len)]

    def argmax_array(self):
        return np.array(self.argmax[: self.n_tree], dtype=np.int64)


_lib = None


def lib():
    """Load libdv.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError("libdv.so not built: run __graft_entry__.build() "
                               "(expected at %s)" % _LIB_PATH)
        L = ctypes.CDLL(_LIB_PATH)
        vp, i32, i32p = ctypes.c_void_p, ctypes.c_int32, ctypes.POINTER(ctypes.c_int32)
        L.dv_verify_init.argtypes = [ctypes.POINTER(dv_config), ctypes.POINTER(dv_weights), vp,
                                     ctypes.POINTER(vp)]
        L.dv_verify_init.restype = ctypes.c_int
        L.dv_verify_step.argtypes = [vp, i32p, i32p, i32, ctypes.POINTER(dv_kv), vp,
                                     ctypes.POINTER(dv_accept)]
        L.dv_verify_step.restype = ctypes.c_int
        f32p = ctypes.POINTER(ctypes.c_float)
        L.dv_verify_step_sampled.argtypes = [vp, i32p, i32p, i32, ctypes.POINTER(dv_kv), vp, ctypes.c_float,
                                             f32p, f32p, vp, ctypes.POINTER(dv_accept)]
        L.dv_verify_step_sampled.restype = ctypes.c_int
        L.dv_accept_sampled.argtypes = [vp, vp, i32p, i32p, i32, vp, ctypes.c_float, f32p, f32p,
                                        ctypes.POINTER(dv_accept)]
        L.dv_accept_sampled.restype = ctypes.c_int
        L.dv_accept_sampled_noalloc.argtypes = [vp, i32p, i32p, i32, i32, vp, ctypes.c_float, f32p, f32p, vp,
                                                ctypes.POINTER(dv_accept)]
        L.dv_accept_sampled_noalloc.restype = ctypes.c_int
        L.dv_draft_init.argtypes = [ctypes.POINTER(dv_config), ctypes.POINTER(dv_weights),
                                    ctypes.POINTER(dv_dgf_weights), vp, ctypes.POINTER(vp)]
        L.dv_draft_init.restype = ctypes.c_int
        L.dv_draft_forward.argtypes = [vp, i32p, i32p, i32, ctypes.POINTER(dv_kv), vp, vp, vp]
        L.dv_draft_forward.restype = ctypes.c_int
        L.dv_draft_tree.argtypes = [vp, i32, vp, ctypes.POINTER(dv_kv), i32, i32, i32, i32p, i32p, f32p]
        L.dv_draft_tree.restype = ctypes.c_int
        L.dv_kv_commit.argtypes = [vp, ctypes.POINTER(dv_kv), ctypes.POINTER(dv_accept)]
        L.dv_kv_commit.restype = ctypes.c_int
        L.dv_prefill.argtypes = [vp, i32p, i32, ctypes.POINTER(dv_kv), i32p]
        L.dv_prefill.restype = ctypes.c_int
        L.dv_verify_free.argtypes = [vp]
        L.dv_verify_free.restype = None
        L.dv_last_error.argtypes = [vp]
        L.dv_last_error.restype = ctypes.c_char_p
        L.dv_tree_prepare.argtypes = [i32p, i32, i32, i32p, i32p, ctypes.POINTER(ctypes.c_uint64)]
        L.dv_tree_prepare.restype = ctypes.c_int
        L.dv_profile_enable.argtypes = [vp, i32]
        L.dv_profile_enable.restype = ctypes.c_int
        L.dv_profile_read.argtypes = [vp, i32, ctypes.POINTER(ctypes.c_double),
                                      ctypes.POINTER(ctypes.c_int64), i32]
        L.dv_profile_read.restype = ctypes.c_int
        _lib = L
    return _lib


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def dv_last_error(h) -> str:
    msg = lib().dv_last_error(h)
    return msg.decode() if msg else ""


def _check(rc: int, h):
    if rc != DV_OK:
        raise DvError(rc, dv_last_error(h))


def dv_verify_init(cfg: dv_config, weights: dv_weights, stream: int = 0):
    h = ctypes.c_void_p()
    rc = lib().dv_verify_init(ctypes.byref(cfg), ctypes.byref(weights), ctypes.c_void_p(stream or None),
                              ctypes.byref(h))
    _check(rc, None)
    return h


def dv_verify_step(h, tokens, tree_parents, kv: dv_kv, out_logits: int = 0) -> dv_accept:
    t, p = _i32(tokens), _i32(tree_parents)
    acc = dv_accept()
    rc = lib().dv_verify_step(h, _ptr(t), _ptr(p), len(t), ctypes.byref(kv),
                              ctypes.c_void_p(out_logits or None), ctypes.byref(acc))
    _check(rc, h)
    return acc


def _f32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float32))


def _fptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_float))


def dv_verify_step_sampled(h, tokens, tree_parents, kv: dv_kv, draft_probs: int, temperature: float,
                           u_accept, u_bonus, out_logits: int = 0) -> dv_accept:
    """draft_probs / out_logits: device addresses; u_accept / u_bonus: host arrays."""
    t, p = _i32(tokens), _i32(tree_parents)
    ua, ub = _f32(u_accept), _f32(u_bonus)
    if len(ua) < len(t) or len(ub) < len(t):
        raise ValueError("u_accept and u_bonus need one entry per tree node")
    acc = dv_accept()
    rc = lib().dv_verify_step_sampled(h, _ptr(t), _ptr(p), len(t), ctypes.byref(kv),
                                      ctypes.c_void_p(draft_probs or None), float(temperature), _fptr(ua),
                                      _fptr(ub), ctypes.c_void_p(out_logits or None), ctypes.byref(acc))
    _check(rc, h)
    return acc


def dv_accept_sampled(h, logits: int, tokens, tree_parents, draft_probs: int, temperature: float,
                      u_accept, u_bonus) -> dv_accept:
    """logits / draft_probs: device addresses; u_accept / u_bonus: host arrays."""
    t, p = _i32(tokens), _i32(tree_parents)
    ua, ub = _f32(u_accept), _f32(u_bonus)
    if len(ua) < len(t) or len(ub) < len(t):
        raise ValueError("u_accept and u_bonus need one entry per tree node")
    acc = dv_accept()
    rc = lib().dv_accept_sampled(h, ctypes.c_void_p(logits or None), _ptr(t), _ptr(p), len(t),
                                 ctypes.c_void_p(draft_probs or None), float(temperature), _fptr(ua), _fptr(ub),
                                 ctypes.byref(acc))
    _check(rc, h)
    return acc


def dv_accept_sampled_noalloc(logits: int, tokens, tree_parents, vocab: int, draft_probs: int,
                              temperature: float, u_accept, u_bonus, stream: int = 0) -> dv_accept:
    """Handle-free, allocation-free sampling rule (workspace: the library's
    fixed per-GPU array).  logits / draft_probs: device addresses."""
    t, p = _i32(tokens), _i32(tree_parents)
    ua, ub = _f32(u_accept), _f32(u_bonus)
    if len(ua) < len(t) or len(ub) < len(t):
        raise ValueError("u_accept and u_bonus need one entry per tree node")
    acc = dv_accept()
    rc = lib().dv_accept_sampled_noalloc(ctypes.c_void_p(logits or None), _ptr(t), _ptr(p), len(t), int(vocab),
                                         ctypes.c_void_p(draft_probs or None), float(temperature), _fptr(ua),
                                         _fptr(ub), ctypes.c_void_p(stream or None), ctypes.byref(acc))
    _check(rc, None)
    return acc


def dv_draft_init(cfg: dv_config, weights: dv_weights, dgf: dv_dgf_weights, stream: int = 0):
    h = ctypes.c_void_p()
    rc = lib().dv_draft_init(ctypes.byref(cfg), ctypes.byref(weights), ctypes.byref(dgf),
                             ctypes.c_void_p(stream or None), ctypes.byref(h))
    _check(rc, None)
    return h


def dv_draft_forward(h, tokens, tree_parents, kv: dv_kv, feat_in: int, feat_out: int, out_logits: int):
    """feat_in / feat_out / out_logits: device addresses."""
    t, p = _i32(tokens), _i32(tree_parents)
    rc = lib().dv_draft_forward(h, _ptr(t), _ptr(p), len(t), ctypes.byref(kv), ctypes.c_void_p(feat_in or None),
                                ctypes.c_void_p(feat_out or None), ctypes.c_void_p(out_logits or None))
    _check(rc, h)


def dv_draft_tree(h, root_token: int, root_feature: int, kv: dv_kv, depth: int, width: int, n_tree: int):
    """Returns (tokens, parents, scores) of the constructed tree (numpy)."""
    tok = np.full(n_tree, -1, dtype=np.int32)
    par = np.full(n_tree, -1, dtype=np.int32)
    sc = np.zeros(n_tree, dtype=np.float32)
    rc = lib().dv_draft_tree(h, int(root_token), ctypes.c_void_p(root_feature or None), ctypes.byref(kv), depth,
                             width, n_tree, _ptr(tok), _ptr(par), _fptr(sc))
    if rc < 0:
        _check(rc, h)
    return tok[:rc], par[:rc], sc[:rc]


def dv_kv_commit(h, kv: dv_kv, accept: dv_accept):
    _check(lib().dv_kv_commit(h, ctypes.byref(kv), ctypes.byref(accept)), h)


def dv_prefill(h, tokens, kv: dv_kv) -> int:
    t = _i32(tokens)
    nxt = ctypes.c_int32(-1)
    _check(lib().dv_prefill(h, _ptr(t), len(t), ctypes.byref(kv), ctypes.byref(nxt)), h)
    return int(nxt.value)


def dv_verify_free(h):
    if h:
        lib().dv_verify_free(h)


def dv_tree_prepare(tree_parents, base_len: int):
    p = _i32(tree_parents)
    n = len(p)
    pos = np.zeros(max(n, 1), dtype=np.int32)
    depth = np.zeros(max(n, 1), dtype=np.int32)
    anc = np.zeros(max(n, 1), dtype=np.uint64)
    rc = lib().dv_tree_prepare(_ptr(p) if n else None, n, base_len, _ptr(pos), _ptr(depth),
                               anc.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64)))
    if rc != DV_OK:
        raise DvError(rc, "invalid tree")
    return pos[:n], depth[:n], anc[:n]


def dv_profile_enable(h, class_mask: int):
    """Bit c of class_mask times kernel class c (DV_K_*); 0 turns timing off."""
    _check(lib().dv_profile_enable(h, class_mask), h)


def dv_profile_read(h, kernel_class: int, reset: bool = False):
    ms = ctypes.c_double()
    n = ctypes.c_int64()
    _check(lib().dv_profile_read(h, kernel_class, ctypes.byref(ms), ctypes.byref(n), 1 if reset else 0), h)
    return float(ms.value), int(n.value)
