"""Device memory for the C ABI: weights, KV cache and outputs as torch tensors.

PyTorch is used only to allocate HIP device memory and copy host arrays into
it; the tensors' raw addresses are handed to libdv.so.  Host arrays are numpy:
bf16 data as uint16 bit patterns, fp32 as float32; matrices [out][in].
"""
from __future__ import annotations

import ctypes

import numpy as np
import torch

from . import dv

LAYER_KEYS = ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down")
MATRIX_KEYS = ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")


def to_device(a: np.ndarray, device) -> torch.Tensor:
    """Copy a host array (uint16 bf16 bits, float32 or int8) to a device tensor."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).to(device).view(torch.bfloat16)
    if a.dtype in (np.float32, np.int8):
        return torch.from_numpy(a).to(device)
    raise TypeError("unsupported host dtype %s" % a.dtype)


def make_config(n_layers, d_model, n_heads, head_dim, d_ffn, vocab, rms_eps, rope_base,
                weight_dtype, max_ctx, max_tree) -> dv.dv_config:
    wd = {"bf16": dv.DV_BF16, "f32": dv.DV_F32, "i8": dv.DV_I8}[weight_dtype]
    return dv.dv_config(n_layers, d_model, n_heads, head_dim, d_ffn, vocab, rms_eps, rope_base,
                        wd, max_ctx, max_tree)


class DeviceWeights:
    """Uploads weights and builds the dv_weights pointer tables.

    layer_fn(l) -> dict with the LAYER_KEYS arrays of layer l (int8 weights:
    also ``<matrix>_scale``, float32 per row; lm_head_scale for the head)."""

    def __init__(self, n_layers, layer_fn, embed, lm_head, final_norm, device="cuda:0", lm_head_scale=None):
        self.device = torch.device(device)
        self.embed = to_device(embed, self.device)
        self.lm_head = to_device(lm_head, self.device)
        self.final_norm = to_device(final_norm, self.device)
        self.lm_head_scale = None if lm_head_scale is None else to_device(lm_head_scale, self.device)
        self.layers = []
        for l in range(n_layers):
            src = layer_fn(l)
            keys = LAYER_KEYS + tuple(k + "_scale" for k in MATRIX_KEYS if k + "_scale" in src)
            self.layers.append({k: to_device(src[k], self.device) for k in keys})
            del src
        self.quantized = "wq_scale" in self.layers[0] if self.layers else False
        self._tables = {}
        keys = LAYER_KEYS + (tuple(k + "_scale" for k in MATRIX_KEYS) if self.quantized else ())
        for k in keys:
            arr = (ctypes.c_void_p * n_layers)(*[t[k].data_ptr() for t in self.layers])
            self._tables[k] = arr
        pp = ctypes.POINTER(ctypes.c_void_p)
        scale_tables = [ctypes.cast(self._tables[k + "_scale"], pp) if self.quantized else None
                        for k in MATRIX_KEYS]
        self.c = dv.dv_weights(
            self.embed.data_ptr(), self.final_norm.data_ptr(), self.lm_head.data_ptr(),
            *[ctypes.cast(self._tables[k], pp) for k in LAYER_KEYS],
            self.lm_head_scale.data_ptr() if self.lm_head_scale is not None else None,
            *scale_tables)

    def nbytes(self) -> int:
        n = self.embed.nbytes + self.lm_head.nbytes + self.final_norm.nbytes
        if self.lm_head_scale is not None:
            n += self.lm_head_scale.nbytes
        return n + sum(t.nbytes for lay in self.layers for t in lay.values())


class DeviceKV:
    """KV cache: K [L][H][capacity][hd], V [L][H][capacity/32][hd][32] (32-slot
    tiles, dim-major within a tile), weight dtype.  capacity must be a
    multiple of 32."""

    def __init__(self, n_layers, n_heads, head_dim, capacity, weight_dtype, device="cuda:0",
                 fill=None):
        dt = torch.float32 if weight_dtype == "f32" else torch.bfloat16  # int8 models keep a bf16 cache
        kshape = (n_layers, n_heads, capacity, head_dim)
        vshape = (n_layers, n_heads, capacity // 32, head_dim, 32)
        if fill is None:
            self.k = torch.zeros(kshape, dtype=dt, device=device)
            self.v = torch.zeros(vshape, dtype=dt, device=device)
        else:
            self.k = torch.full(kshape, fill, dtype=dt, device=device)
            self.v = torch.full(vshape, fill, dtype=dt, device=device)
        self.c = dv.dv_kv(self.k.data_ptr(), self.v.data_ptr(), capacity, 0)

    @property
    def len(self) -> int:
        return int(self.c.len)

    def set_layer(self, l: int, k: np.ndarray, v: np.ndarray):
        """Write committed entries [0, n) of layer l from host arrays [H][n][hd]."""
        n = k.shape[1]
        self.k[l, :, :n].copy_(to_device(k, self.k.device))
        slots = self._v_slots(l).clone()           # [H][capacity][hd]
        slots[:, :n] = to_device(v, self.v.device)
        h, cap, hd = slots.shape
        self.v[l].copy_(slots.reshape(h, cap // 32, 32, hd).transpose(2, 3))

    def _v_slots(self, l: int) -> torch.Tensor:
        """V of layer l viewed slot-major, [H][capacity][hd] (a copy)."""
        v = self.v[l]
        h, nt, hd, _ = v.shape
        return v.transpose(2, 3).reshape(h, nt * 32, hd)

    def layer_host(self, l: int, n: int):
        """Entries [0, n) of layer l as host arrays [H][n][hd] in the stored format."""
        def host(t):
            t = t.contiguous().cpu()
            if t.dtype == torch.bfloat16:
                return t.view(torch.int16).numpy().view(np.uint16)
            return t.numpy()
        return host(self.k[l, :, :n]), host(self._v_slots(l)[:, :n])
