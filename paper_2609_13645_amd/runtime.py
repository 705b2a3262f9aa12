"""Device-buffer plumbing around the C ABI (PyTorch used for memory and streams).

Nothing here computes: it allocates caller-owned device buffers with torch,
fills the C structs and calls libforge. The arithmetic of every step is in
the HIP kernels.
"""
from __future__ import annotations

import numpy as np

from . import _lib

LAYER_WEIGHTS = ("attn_norm", "w_qkv", "w_o", "ffn_norm", "w_gate_up", "w_down")
GRAD_NAMES = {n: "d_" + n for n in LAYER_WEIGHTS}


def _torch():
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("libforge needs a ROCm GPU (torch.cuda.is_available() is False)")
    return torch


def to_device_bf16(bits: np.ndarray, device="cuda"):
    """uint16 bf16 bit patterns (host) -> torch.bfloat16 device tensor."""
    torch = _torch()
    arr = np.ascontiguousarray(bits, dtype=np.uint16).view(np.int16)
    return torch.from_numpy(arr.copy()).view(torch.bfloat16).to(device)


def to_host_bits(t) -> np.ndarray:
    """torch.bfloat16 tensor -> uint16 bit patterns on the host."""
    torch = _torch()
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def to_device(arr: np.ndarray, device="cuda"):
    torch = _torch()
    return torch.from_numpy(np.ascontiguousarray(arr).copy()).to(device)


def layer_shapes(cfg: dict) -> dict:
    """Shapes of one dense layer's weights."""
    h, d = cfg["hidden"], cfg["head_dim"]
    hq, hkv, f = cfg["n_heads"] * d, cfg["n_kv_heads"] * d, cfg["ffn"]
    return {"attn_norm": (h,), "w_qkv": (hq + 2 * hkv, h), "w_o": (h, hq),
            "ffn_norm": (h,), "w_gate_up": (2 * f, h), "w_down": (h, f)}


def empty_bytes(n: int, device="cuda"):
    torch = _torch()
    return torch.empty(max(int(n), 1), dtype=torch.uint8, device=device)


class FlatParams:
    """Flat optimizer buffers for a set of named tensors.

    One bf16 parameter buffer and fp32 master / grad / m / v buffers, with
    every tensor a view at a 64-element-aligned offset, so a single
    forge_adamw_step call updates them all (gaps stay zero).
    """

    def __init__(self, shapes: dict, device="cuda"):
        torch = _torch()
        self.offsets, off = {}, 0
        for name, shape in shapes.items():
            self.offsets[name] = (off, tuple(shape))
            off += (int(np.prod(shape)) + 63) // 64 * 64
        self.n = off
        self.param = torch.zeros(off, dtype=torch.bfloat16, device=device)
        self.master = torch.zeros(off, dtype=torch.float32, device=device)
        self.grad = torch.zeros(off, dtype=torch.float32, device=device)
        self.m = torch.zeros(off, dtype=torch.float32, device=device)
        self.v = torch.zeros(off, dtype=torch.float32, device=device)

    def view(self, buf, name):
        off, shape = self.offsets[name]
        return buf[off:off + int(np.prod(shape))].view(shape)

    def load_bits(self, name, bits):
        """Set a parameter from bf16 bits; the master copy is its exact fp32 value."""
        p = self.view(self.param, name)
        p.copy_(to_device_bf16(bits, p.device))
        self.view(self.master, name).copy_(p.float())


class Layer:
    """One decoder layer's device state: weights, RoPE tables, grads, buffers.

    With `flat`, the weights and their gradients are views into a FlatParams.
    """

    def __init__(self, cfg: dict, weights_bits: dict, device="cuda", stream=None,
                 flat: FlatParams | None = None):
        torch = _torch()
        self.cfg = dict(cfg)
        self.c = _lib.layer_cfg(cfg)
        self.stream = stream
        if flat is None:
            self.w = {n: to_device_bf16(weights_bits[n], device) for n in LAYER_WEIGHTS}
        else:
            for n in LAYER_WEIGHTS:
                flat.load_bits(n, weights_bits[n])
            self.w = {n: flat.view(flat.param, n) for n in LAYER_WEIGHTS}
        half = cfg["head_dim"] // 2
        self.w["rope_cos"] = torch.empty((cfg["seq"], half), dtype=torch.float32, device=device)
        self.w["rope_sin"] = torch.empty((cfg["seq"], half), dtype=torch.float32, device=device)
        _lib.forge_rope_table(cfg["seq"], cfg["head_dim"], cfg["rope_base"],
                              self.w["rope_cos"], self.w["rope_sin"], stream)
        self.weights = _lib.layer_weights(self.w)
        if flat is None:
            self.g = {GRAD_NAMES[n]: torch.zeros(self.w[n].shape, dtype=torch.float32,
                                                 device=device) for n in LAYER_WEIGHTS}
        else:
            self.g = {GRAD_NAMES[n]: flat.view(flat.grad, n) for n in LAYER_WEIGHTS}
        self.grads = _lib.layer_grads(self.g)
        self.saved = empty_bytes(_lib.forge_layer_saved_bytes(self.c), device)
        self.workspace = empty_bytes(_lib.forge_layer_workspace_bytes(self.c), device)

    def zero_grads(self):
        for t in self.g.values():
            t.zero_()

    def fwd(self, x_in, x_out, saved=None, workspace=None):
        _lib.forge_layer_fwd(self.c, self.weights, x_in, x_out,
                             self.saved if saved is None else saved,
                             self.workspace if workspace is None else workspace,
                             None, self.stream)

    def bwd(self, x_in, d_out, d_in, saved=None, workspace=None):
        _lib.forge_layer_bwd(self.c, self.weights, self.saved if saved is None else saved,
                             x_in, d_out, d_in, self.grads,
                             self.workspace if workspace is None else workspace, self.stream)
