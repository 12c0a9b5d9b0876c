"""Seeded synthetic inputs for the tree-verification workloads.

Holds the workload definitions (Llama-style shapes, context length, tree size)
and generators for weights, KV-cache contents, prompts and draft trees.  It
contains none of the verification arithmetic: every number comes from the
counter-based splitmix64 stream in ``gen.c`` (Box-Muller for normals) and is
rounded to its storage dtype.  Tests and the benchmark hand the same bytes to
the GPU library and to the CPU oracle.

Weight matrices are stored ``[out][in]`` row-major, the layout the GPU library
takes.  bf16 tensors are returned as ``uint16`` bit patterns.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass, field, replace

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "libdvsynth.so")
_SRC = os.path.join(_HERE, "gen.c")


def build_lib(force: bool = True) -> str:
    """Compile the host generator with gcc (OpenMP)."""
    if force or not os.path.exists(_SO):
        tmp = _SO + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC",
                               "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _SO)
    return _SO


_lib = None


def _L():
    global _lib
    if _lib is None:
        if not os.path.exists(_SO):
            build_lib(force=False)
        lib = ctypes.CDLL(_SO)
        u64, p = ctypes.c_uint64, ctypes.c_void_p
        lib.dvs_key.argtypes = [u64, u64]
        lib.dvs_key.restype = u64
        lib.dvs_normal_bf16.argtypes = [u64, u64, u64, u64, ctypes.c_double, p]
        lib.dvs_normal_f32.argtypes = [u64, u64, u64, u64, ctypes.c_double, p]
        lib.dvs_normal_i8.argtypes = [u64, u64, u64, u64, ctypes.c_double, p]
        lib.dvs_gain_bf16.argtypes = [u64, u64, u64, u64, ctypes.c_double, p]
        lib.dvs_gain_f32.argtypes = [u64, u64, u64, u64, ctypes.c_double, p]
        lib.dvs_u64.argtypes = [u64, u64, u64, u64, p]
        lib.dvs_uniform_int.argtypes = [u64, u64, u64, u64, ctypes.c_uint32, p]
        _lib = lib
    return _lib


# ---------------------------------------------------------------------------
# raw streams

def normal(seed: int, tensor: int, n: int, sigma: float, dtype: str, start: int = 0) -> np.ndarray:
    """``n`` draws of N(0, sigma^2) stored as ``dtype`` ('bf16' -> uint16 bits, 'f32',
    'i8' -> int8 codes rint(sigma z) clipped to [-127, 127])."""
    if dtype == "i8":
        out = np.empty(n, dtype=np.int8)
        _L().dvs_normal_i8(seed, tensor, start, n, sigma, out.ctypes.data)
    elif dtype == "bf16":
        out = np.empty(n, dtype=np.uint16)
        _L().dvs_normal_bf16(seed, tensor, start, n, sigma, out.ctypes.data)
    elif dtype == "f32":
        out = np.empty(n, dtype=np.float32)
        _L().dvs_normal_f32(seed, tensor, start, n, sigma, out.ctypes.data)
    else:
        raise ValueError(dtype)
    return out


def gain(seed: int, tensor: int, n: int, sigma: float, dtype: str) -> np.ndarray:
    """``n`` norm gains 1 + N(0, sigma^2) stored as ``dtype`` ('bf16' -> uint16
    bits, 'f32')."""
    if dtype == "bf16":
        out = np.empty(n, dtype=np.uint16)
        _L().dvs_gain_bf16(seed, tensor, 0, n, sigma, out.ctypes.data)
    elif dtype == "f32":
        out = np.empty(n, dtype=np.float32)
        _L().dvs_gain_f32(seed, tensor, 0, n, sigma, out.ctypes.data)
    else:
        raise ValueError(dtype)
    return out


def u64(seed: int, tensor: int, n: int, start: int = 0) -> np.ndarray:
    out = np.empty(n, dtype=np.uint64)
    _L().dvs_u64(seed, tensor, start, n, out.ctypes.data)
    return out


def uniform_int(seed: int, tensor: int, n: int, hi: int, start: int = 0) -> np.ndarray:
    out = np.empty(n, dtype=np.int32)
    _L().dvs_uniform_int(seed, tensor, start, n, hi, out.ctypes.data)
    return out


# Pure-numpy restatement of the stream, used only to check the C build.
_GOLDEN = 0x9E3779B97F4A7C15
_MASK = (1 << 64) - 1


def _mix64_py(z: int) -> int:
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK
    return z ^ (z >> 31)


def u64_py(seed: int, tensor: int, i: int) -> int:
    key = _mix64_py(_mix64_py((seed + _GOLDEN) & _MASK) ^ ((tensor * _GOLDEN) & _MASK))
    return _mix64_py((key + (i + 1) * _GOLDEN) & _MASK)


# ---------------------------------------------------------------------------
# model shapes and workloads

@dataclass(frozen=True)
class ModelCfg:
    n_layers: int
    d_model: int
    n_heads: int
    head_dim: int
    d_ffn: int
    vocab: int
    rms_eps: float = 1e-6
    rope_base: float = 10000.0
    weight_dtype: str = "bf16"   # 'bf16', 'f32' or 'i8'; the KV cache uses the same dtype (bf16 for 'i8')
    init_std: float = 0.02

    @property
    def kv_dtype(self) -> str:
        return "bf16" if self.weight_dtype == "i8" else self.weight_dtype

    @property
    def dense_dtype(self) -> str:
        """dtype of the embedding and the norm gains"""
        return "bf16" if self.weight_dtype == "i8" else self.weight_dtype

    def layer_params(self) -> int:
        d, f = self.d_model, self.d_ffn
        return 4 * d * d + 3 * d * f + 2 * d


@dataclass(frozen=True)
class Workload:
    name: str
    model: ModelCfg
    context: int        # committed KV length P before the step
    n_tree: int         # draft tokens M in the step (root included)
    depth: int          # maximum tree depth (root depth 1)
    chain: bool = False  # tree is a chain of n_tree tokens
    prefill: bool = False  # KV built by prefilling uniform-random prompt ids
    seed_base: int = 0
    weight_seed: int = 0  # shared by every workload of one model

    @property
    def seeds(self):
        b = self.seed_base
        return dict(weights=self.weight_seed or 1 + b, prompt=2 + b, tree=3 + b, kv=4 + b)


TINY = ModelCfg(n_layers=2, d_model=256, n_heads=4, head_dim=64, d_ffn=688, vocab=1024,
                weight_dtype="f32")
LLAMA7B = ModelCfg(n_layers=32, d_model=4096, n_heads=32, head_dim=128, d_ffn=11008,
                   vocab=32000)
LLAMA13B = ModelCfg(n_layers=40, d_model=5120, n_heads=40, head_dim=128, d_ffn=13824,
                    vocab=32000)
LLAMA13B_I8 = replace(LLAMA13B, weight_dtype="i8")

WORKLOADS = {
    "tiny-f32-chain4": Workload("tiny-f32-chain4", TINY, context=64, n_tree=4, depth=4,
                                chain=True, prefill=True, seed_base=100),
    "llama7b-bf16-m8-ctx512": Workload("llama7b-bf16-m8-ctx512", LLAMA7B, context=512,
                                       n_tree=8, depth=5, seed_base=200, weight_seed=201),
    "llama13b-bf16-m16-ctx1024": Workload("llama13b-bf16-m16-ctx1024", LLAMA13B,
                                          context=1024, n_tree=16, depth=6, seed_base=300,
                                          weight_seed=301),
    "llama13b-bf16-ctx8192": Workload("llama13b-bf16-ctx8192", LLAMA13B, context=8192,
                                      n_tree=16, depth=6, seed_base=500, weight_seed=301),
    # weight-only int8 variant of the 13B workload (same context, tree and seeds)
    "llama13b-i8-m16-ctx1024": Workload("llama13b-i8-m16-ctx1024", LLAMA13B_I8,
                                        context=1024, n_tree=16, depth=6, seed_base=300,
                                        weight_seed=301),
}
SWEEP_M = (1, 2, 4, 8, 16, 32, 64)


def sweep_workload(m: int) -> Workload:
    return Workload("llama13b-bf16-m%d-ctx1024" % m, LLAMA13B, context=1024, n_tree=m,
                    depth=8, seed_base=400 + m, weight_seed=301)


def shrink(model: ModelCfg, **kw) -> ModelCfg:
    return replace(model, **kw)


# ---------------------------------------------------------------------------
# tensor ids inside one seed

T_EMBED, T_LMHEAD, T_PROMPT, T_TREE_PARENT, T_TREE_TOKEN = 1, 2, 3, 4, 5
T_UNIFORM, T_DRAFT = 6, 7
T_FINAL_NORM = 8
T_SCALE_OFFSET = 1 << 40   # row scales of the matrix with tensor id t use id t + T_SCALE_OFFSET
LAYER_NAMES = ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")


def _t_layer(l: int, name: str) -> int:
    return 1000 + 16 * l + LAYER_NAMES.index(name)


def _t_norm(l: int, which: int) -> int:
    """attention norm (which 0) and FFN norm (which 1) of layer l"""
    return 1000 + 16 * l + len(LAYER_NAMES) + which


def _t_kv(l: int, which: int) -> int:
    return 500000 + 2 * l + which


# Norm gains: 1 + N(0, GAIN_SIGMA^2) per element, a distinct stream per layer
# and norm, so that a gain applied in the wrong place changes the result.
GAIN_SIGMA = 0.1


I8_CODE_SIGMA = 127.0 / 4.0   # int8 codes: the clip sits at 4 standard deviations


def row_scales(cfg: ModelCfg, seed: int, tensor: int, rows: int) -> np.ndarray:
    """Per-row scales of an int8 matrix: init_std / I8_CODE_SIGMA, varied by
    up to +-25% per row (uniform), float32."""
    u = uniform01(seed, tensor, rows).astype(np.float64)
    return (cfg.init_std / I8_CODE_SIGMA * (0.75 + 0.5 * u)).astype(np.float32)


def _matrix(cfg: ModelCfg, seed: int, tensor: int, rows: int, cols: int, out: dict, key: str):
    if cfg.weight_dtype == "i8":
        out[key] = normal(seed, tensor, rows * cols, I8_CODE_SIGMA, "i8").reshape(rows, cols)
        out[key + "_scale"] = row_scales(cfg, seed, tensor + T_SCALE_OFFSET, rows)
    else:
        out[key] = normal(seed, tensor, rows * cols, cfg.init_std, cfg.weight_dtype).reshape(rows, cols)


def layer_weights(cfg: ModelCfg, seed: int, l: int) -> dict:
    """Weights of layer ``l``: matrices ``[out][in]`` and the two norm gains
    (1 + N(0, GAIN_SIGMA^2) each).  For 'i8' each matrix comes with
    ``<name>_scale`` (float32 per row)."""
    d, f = cfg.d_model, cfg.d_ffn
    shapes = dict(wq=(d, d), wk=(d, d), wv=(d, d), wo=(d, d),
                  w_gate=(f, d), w_up=(f, d), w_down=(d, f))
    out = {}
    for k, (a, b) in shapes.items():
        _matrix(cfg, seed, _t_layer(l, k), a, b, out, k)
    out["attn_norm"] = gain(seed, _t_norm(l, 0), d, GAIN_SIGMA, cfg.dense_dtype)
    out["ffn_norm"] = gain(seed, _t_norm(l, 1), d, GAIN_SIGMA, cfg.dense_dtype)
    return out


def embed(cfg: ModelCfg, seed: int) -> np.ndarray:
    return normal(seed, T_EMBED, cfg.vocab * cfg.d_model, cfg.init_std,
                  cfg.dense_dtype).reshape(cfg.vocab, cfg.d_model)


def embed_rows(cfg: ModelCfg, seed: int, ids) -> np.ndarray:
    rows = [normal(seed, T_EMBED, cfg.d_model, cfg.init_std, cfg.dense_dtype,
                   start=int(t) * cfg.d_model) for t in ids]
    return np.stack(rows)


def lm_head(cfg: ModelCfg, seed: int) -> np.ndarray:
    """The lm_head matrix (for 'i8' the int8 codes; see lm_head_scale)."""
    out = {}
    _matrix(cfg, seed, T_LMHEAD, cfg.vocab, cfg.d_model, out, "w")
    return out["w"]


def lm_head_scale(cfg: ModelCfg, seed: int):
    """Row scales of an 'i8' lm_head (None otherwise)."""
    if cfg.weight_dtype != "i8":
        return None
    return row_scales(cfg, seed, T_LMHEAD + T_SCALE_OFFSET, cfg.vocab)


def final_norm(cfg: ModelCfg, seed: int) -> np.ndarray:
    """Gains of the final norm (1 + N(0, GAIN_SIGMA^2))."""
    return gain(seed, T_FINAL_NORM, cfg.d_model, GAIN_SIGMA, cfg.dense_dtype)


def kv_sigma(cfg: ModelCfg) -> float:
    """Scale of synthetic cached keys/values: what W u gives for unit-RMS u."""
    return cfg.init_std * float(np.sqrt(cfg.d_model))


def kv_layer(cfg: ModelCfg, seed: int, l: int, n_ctx: int):
    """Synthetic committed K and V of layer ``l``: ``[H][n_ctx][hd]`` each."""
    h, hd = cfg.n_heads, cfg.head_dim
    s = kv_sigma(cfg)
    k = normal(seed, _t_kv(l, 0), h * n_ctx * hd, s, cfg.kv_dtype).reshape(h, n_ctx, hd)
    v = normal(seed, _t_kv(l, 1), h * n_ctx * hd, s, cfg.kv_dtype).reshape(h, n_ctx, hd)
    return k, v


def prompt(seed: int, n: int, vocab: int) -> np.ndarray:
    return uniform_int(seed, T_PROMPT, n, vocab)


def random_tree(seed: int, n: int, depth: int, vocab: int, chain: bool = False,
                stream: int = 0):
    """Draft tree: node 0 is the root (parent -1); node i >= 1 picks its parent
    uniformly among earlier nodes whose depth is below ``depth``.  Token ids are
    uniform in [0, vocab).  Returns (tokens int32[n], parents int32[n])."""
    if n < 1:
        raise ValueError("tree needs at least its root")
    toks = uniform_int(seed, T_TREE_TOKEN + 16 * stream, n, vocab)
    draws = u64(seed, T_TREE_PARENT + 16 * stream, n)
    parents = np.full(n, -1, dtype=np.int32)
    dep = np.ones(n, dtype=np.int64)
    for i in range(1, n):
        if chain:
            p = i - 1
        else:
            cand = [j for j in range(i) if dep[j] < depth]
            if not cand:
                raise ValueError("depth bound leaves no parent for node %d" % i)
            p = cand[int(draws[i] % np.uint64(len(cand)))]
        parents[i] = p
        dep[i] = dep[p] + 1
    return toks, parents


def uniform01(seed: int, tensor: int, n: int, start: int = 0) -> np.ndarray:
    """``n`` float32 uniforms in [0, 1): the top 24 bits of the stream, so
    every value is exact in float32 and strictly below 1."""
    return (u64(seed, tensor, n, start) >> np.uint64(40)).astype(np.float32) * np.float32(2.0 ** -24)


def sampling_uniforms(seed: int, n: int, stream: int = 0):
    """The random numbers of one sampled acceptance over an n-node tree:
    (u_accept float32[n], u_bonus float32[n])."""
    u = uniform01(seed, T_UNIFORM + 16 * stream, 2 * n)
    return u[:n].copy(), u[n:].copy()


def draft_rows(seed: int, m: int, vocab: int, sharp: float = 8.0, stream: int = 0) -> np.ndarray:
    """m draft distributions over the vocabulary, float32 [m][vocab]: uniforms
    raised to ``sharp`` (a few ids carry most of the mass), each row divided
    by its float64 total."""
    w = uniform01(seed, T_DRAFT + 16 * stream, m * vocab).astype(np.float64).reshape(m, vocab) ** sharp
    return (w / w.sum(axis=1, keepdims=True)).astype(np.float32)


T_DGF = 900000             # DGF weights of a draft: ids T_DGF + 0, 1, 2
T_FEATURE = 900010         # hidden states handed to a draft


def draft_cfg(target: ModelCfg, n_blocks: int) -> ModelCfg:
    """The draft's block stack: n_blocks Llama blocks of the target's width."""
    return replace(target, n_layers=n_blocks)


def dgf_weights(cfg: ModelCfg, seed: int) -> dict:
    """DGF weights (bf16 bits): w_hidden, w_embed [d][d], w_gate [d][2d]."""
    d, s = cfg.d_model, cfg.init_std
    return {"w_hidden": normal(seed, T_DGF, d * d, s, "bf16").reshape(d, d),
            "w_embed": normal(seed, T_DGF + 1, d * d, s, "bf16").reshape(d, d),
            "w_gate": normal(seed, T_DGF + 2, 2 * d * d, s, "bf16").reshape(d, 2 * d)}


def features(seed: int, n: int, d: int, sigma: float = 1.0, stream: int = 0) -> np.ndarray:
    """n hidden-state rows [n][d] float32, N(0, sigma^2)."""
    return normal(seed, T_FEATURE + stream, n * d, sigma, "f32").reshape(n, d)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Storage conversion for uploading/reading bf16 buffers (exact)."""
    return (bits.astype(np.uint32) << 16).view(np.float32)
