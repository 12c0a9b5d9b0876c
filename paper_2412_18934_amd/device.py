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


def to_device(a: np.ndarray, device) -> torch.Tensor:
    """Copy a host array (uint16 bf16 bits or float32) to a device tensor."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).to(device).view(torch.bfloat16)
    if a.dtype == np.float32:
        return torch.from_numpy(a).to(device)
    raise TypeError("unsupported host dtype %s" % a.dtype)


def make_config(n_layers, d_model, n_heads, head_dim, d_ffn, vocab, rms_eps, rope_base,
                weight_dtype, max_ctx, max_tree) -> dv.dv_config:
    return dv.dv_config(n_layers, d_model, n_heads, head_dim, d_ffn, vocab, rms_eps, rope_base,
                        dv.DV_BF16 if weight_dtype == "bf16" else dv.DV_F32, max_ctx, max_tree)


class DeviceWeights:
    """Uploads weights and builds the dv_weights pointer tables.

    layer_fn(l) -> dict with the LAYER_KEYS arrays of layer l."""

    def __init__(self, n_layers, layer_fn, embed, lm_head, final_norm, device="cuda:0"):
        self.device = torch.device(device)
        self.embed = to_device(embed, self.device)
        self.lm_head = to_device(lm_head, self.device)
        self.final_norm = to_device(final_norm, self.device)
        self.layers = []
        for l in range(n_layers):
            src = layer_fn(l)
            self.layers.append({k: to_device(src[k], self.device) for k in LAYER_KEYS})
            del src
        self._tables = {}
        for k in LAYER_KEYS:
            arr = (ctypes.c_void_p * n_layers)(*[t[k].data_ptr() for t in self.layers])
            self._tables[k] = arr
        pp = ctypes.POINTER(ctypes.c_void_p)
        self.c = dv.dv_weights(
            self.embed.data_ptr(), self.final_norm.data_ptr(), self.lm_head.data_ptr(),
            *[ctypes.cast(self._tables[k], pp) for k in LAYER_KEYS])

    def nbytes(self) -> int:
        n = self.embed.nbytes + self.lm_head.nbytes + self.final_norm.nbytes
        return n + sum(t.nbytes for lay in self.layers for t in lay.values())


class DeviceKV:
    """KV cache: K [L][H][capacity][hd], V [L][H][hd][capacity] (dim-major),
    weight dtype.  capacity must be a multiple of 32."""

    def __init__(self, n_layers, n_heads, head_dim, capacity, weight_dtype, device="cuda:0",
                 fill=None):
        dt = torch.bfloat16 if weight_dtype == "bf16" else torch.float32
        kshape = (n_layers, n_heads, capacity, head_dim)
        vshape = (n_layers, n_heads, head_dim, capacity)
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
        self.v[l, :, :, :n].copy_(to_device(v, self.v.device).transpose(1, 2))

    def layer_host(self, l: int, n: int):
        """Entries [0, n) of layer l as host arrays [H][n][hd] in the stored format."""
        def host(t):
            t = t.contiguous().cpu()
            if t.dtype == torch.bfloat16:
                return t.view(torch.int16).numpy().view(np.uint16)
            return t.numpy()
        return host(self.k[l, :, :n]), host(self.v[l, :, :, :n].transpose(1, 2))
