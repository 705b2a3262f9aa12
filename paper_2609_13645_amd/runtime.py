"""Device-buffer plumbing around the C ABI (PyTorch used for memory and streams).

Nothing here computes: it allocates caller-owned device buffers with torch,
fills the C structs and calls libforge. The arithmetic of every step is in
the HIP kernels.
"""
from __future__ import annotations

import numpy as np

from . import _lib

LAYER_WEIGHTS = ("attn_norm", "w_qkv", "w_o", "ffn_norm", "w_gate_up", "w_down")


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


def layer_weight_names(cfg: dict):
    return tuple(layer_shapes(cfg))


def layer_shapes(cfg: dict) -> dict:
    """Shapes of one layer's weights (dense or MoE, with the variants the
    configuration turns on: QK-Norm gains, shared expert)."""
    h, d = cfg["hidden"], cfg["head_dim"]
    hq, hkv = cfg["n_heads"] * d, cfg["n_kv_heads"] * d
    out = {"attn_norm": (h,), "w_qkv": (hq + 2 * hkv, h), "w_o": (h, hq), "ffn_norm": (h,)}
    if cfg.get("n_experts", 0):
        E, fe = cfg["n_experts"], cfg["expert_ffn"]
        out.update({"w_router": (E, h), "w_gate_up_e": (E, 2 * fe, h), "w_down_e": (E, h, fe)})
        fs = cfg.get("shared_ffn", 0)
        if fs:
            out.update({"w_gate_up_s": (2 * fs, h), "w_down_s": (h, fs)})
    else:
        f = cfg["ffn"]
        out.update({"w_gate_up": (2 * f, h), "w_down": (h, f)})
    if cfg.get("qk_norm", 0):
        out.update({"q_norm": (d,), "k_norm": (d,)})
    return out


def model_layer_cfg(cfg: dict, i: int) -> dict:
    """Configuration of layer i of a model: the first dense_first_layers
    layers of a MoE model use the dense FFN of width ffn (App. B, the sparse
    model's dense layer 0)."""
    if cfg.get("n_experts", 0) and i < cfg.get("dense_first_layers", 0):
        return dict(cfg, n_experts=0, top_k=0, expert_ffn=0, shared_ffn=0)
    return cfg


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
        names = layer_weight_names(cfg)
        self.names = names
        if flat is None:
            self.w = {n: to_device_bf16(weights_bits[n], device) for n in names}
        else:
            for n in names:
                flat.load_bits(n, weights_bits[n])
            self.w = {n: flat.view(flat.param, n) for n in names}
        half = cfg["head_dim"] // 2
        self.w["rope_cos"] = torch.empty((cfg["seq"], half), dtype=torch.float32, device=device)
        self.w["rope_sin"] = torch.empty((cfg["seq"], half), dtype=torch.float32, device=device)
        if cfg.get("positions") is not None:    # document-aware RoPE positions [T]
            self.w["positions"] = torch.from_numpy(
                np.ascontiguousarray(cfg["positions"], dtype=np.int32)).to(device)
        _lib.forge_rope_table(cfg["seq"], cfg["head_dim"], cfg["rope_base"],
                              self.w["rope_cos"], self.w["rope_sin"], stream)
        self.weights = _lib.layer_weights(self.w)
        if flat is None:
            self.g = {"d_" + n: torch.zeros(self.w[n].shape, dtype=torch.float32,
                                            device=device) for n in names}
        else:
            self.g = {"d_" + n: flat.view(flat.grad, n) for n in names}
        self.aux = torch.zeros(1, dtype=torch.float32, device=device)
        self.grads = _lib.layer_grads(self.g)
        self.saved = empty_bytes(_lib.forge_layer_saved_bytes(self.c), device)
        self.workspace = empty_bytes(_lib.forge_layer_workspace_bytes(self.c), device)

    def zero_grads(self):
        for t in self.g.values():
            t.zero_()

    def fwd(self, x_in, x_out, saved=None, workspace=None, aux=None):
        """Forward; for a MoE layer the load-balance loss is added to `aux`
        (a device fp32 scalar; self.aux when None)."""
        _lib.forge_layer_fwd(self.c, self.weights, x_in, x_out,
                             self.saved if saved is None else saved,
                             self.workspace if workspace is None else workspace,
                             (self.aux if aux is None else aux) if self.cfg.get("n_experts", 0)
                             else None, self.stream)

    def bwd(self, x_in, d_out, d_in, saved=None, workspace=None, overwrite=False):
        """Backward; weight gradients are accumulated (+=) into self.g, or
        written (=) with overwrite (no zeroing needed beforehand)."""
        self.grads.overwrite = int(overwrite)
        _lib.forge_layer_bwd(self.c, self.weights, self.saved if saved is None else saved,
                             x_in, d_out, d_in, self.grads,
                             self.workspace if workspace is None else workspace, self.stream)

    def bwd_adamw(self, x_in, d_out, d_in, flat: "FlatParams", hparams, dev_scalars,
                  overwrite=True):
        """Backward plus the AdamW update of every weight of this layer (its
        weights must be views into `flat`), each update overlapping the rest
        of the backward; dev_scalars = device fp32 {lr, bc1, bc2, clip}."""
        self.grads.overwrite = int(overwrite)
        opt = _lib.layer_optim({n: {k: flat.view(getattr(flat, k), n)
                                    for k in ("master", "param", "m", "v")}
                                for n in self.names})
        _lib.forge_layer_bwd_adamw(self.c, self.weights, self.saved, x_in, d_out, d_in,
                                   self.grads, opt, hparams, dev_scalars, self.workspace,
                                   self.stream)


class Model:
    """A whole decoder stack's training step through the C ABI.

    Embedding -> n_layers decoder layers -> final RMSNorm + LM head + CE
    (tied to the embedding when w_lm is None) -> backward -> embedding
    backward -> one fused AdamW over every parameter (flat buffers).
    Every step of the computation runs in libforge's kernels; this class only
    owns the buffers and issues the calls in order on one stream.
    """

    def __init__(self, cfg: dict, inputs: dict, device="cuda", stream=None):
        torch = _torch()
        self.cfg = dict(cfg)
        self.stream = stream
        L, V, h = cfg["n_layers"], cfg["vocab"], cfg["hidden"]
        self.T = cfg["batch"] * cfg["seq"]
        self.tied = inputs["w_lm"] is None
        shapes = {"embedding": (V, h), "final_norm": (h,)}
        if not self.tied:
            shapes["w_lm"] = (V, h)
        for i in range(L):
            for n, s in layer_shapes(model_layer_cfg(cfg, i)).items():
                shapes[f"{i}.{n}"] = s
        self.flat = FlatParams(shapes, device)
        # the embedding / head tensors come first in the flat buffers
        self.head_grad_elems = max(self.flat.offsets[n][0] + int(np.prod(shapes[n]))
                                   for n in shapes if "." not in n)
        self.flat.load_bits("embedding", inputs["embedding"])
        self.flat.load_bits("final_norm", inputs["final_norm"])
        if not self.tied:
            self.flat.load_bits("w_lm", inputs["w_lm"])
        self.layers, self.layer_flats = [], []
        for i in range(L):
            view = _PrefixedFlat(self.flat, f"{i}.")
            self.layer_flats.append(view)
            self.layers.append(Layer(model_layer_cfg(cfg, i), inputs["layers"][i], device, stream,
                                     flat=view))
        ws = max(max(_lib.forge_layer_workspace_bytes(ly.c) for ly in self.layers), 1)
        self.workspace = empty_bytes(ws, device)
        for ly in self.layers:               # one shared scratch buffer
            ly.workspace = self.workspace
        self.head = _lib.HeadCfg(self.T, h, V, cfg["rms_eps"], cfg.get("logit_scale", 0.0))
        self.embed_scale = cfg.get("embed_scale", 0.0) or 1.0
        # ce_chunk: the streaming head (chunk x V logits at a time), else T x V
        self.ce_chunk = int(cfg.get("ce_chunk", 0))
        self.head_ws = empty_bytes(
            _lib.forge_loss_chunked_workspace_bytes(self.head, self.ce_chunk) if self.ce_chunk
            else _lib.forge_loss_workspace_bytes(self.head), device)
        self.ids = torch.from_numpy(inputs["ids"].astype(np.int32)).to(device)
        self.targets = torch.from_numpy(inputs["targets"].astype(np.int32)).to(device)
        self.acts = [torch.empty((self.T, h), dtype=torch.bfloat16, device=device)
                     for _ in range(L + 1)]
        self.grad_a = torch.empty((self.T, h), dtype=torch.bfloat16, device=device)
        self.grad_b = torch.empty((self.T, h), dtype=torch.bfloat16, device=device)
        self.loss = torch.zeros(1, dtype=torch.float32, device=device)
        # MoE layers add their load-balance losses here (their gradients are
        # part of each layer's backward); the reported loss is the CE alone
        self.aux = torch.zeros(1, dtype=torch.float32, device=device)
        self.scalars = torch.zeros(4, dtype=torch.float32, device=device)
        self.hp = _lib.AdamwHparams(cfg["beta1"], cfg["beta2"], cfg["adam_eps"],
                                    cfg["weight_decay"])
        self.step_count = 0
        self.dev_step = torch.zeros(1, dtype=torch.int32, device=device)
        # global gradient norm for clipping, summed on the device
        self.norm_sq = torch.zeros(1, dtype=torch.float32, device=device)
        self.norm_ws = torch.empty(_lib.GRAD_NORM_WORKSPACE_FLOATS, dtype=torch.float32,
                                   device=device)

    def w_lm(self, buf):
        return self.flat.view(buf, "embedding" if self.tied else "w_lm")

    def _forward_and_head(self, accumulate):
        """Embedding, layers, then the loss head's forward and backward: the
        loss, the head gradients and the gradient at the last layer's output
        (self.grad_a)."""
        c, s = self.cfg, self.stream
        if not accumulate:
            self.flat.grad[:self.head_grad_elems].zero_()
        T, h, V = self.T, c["hidden"], c["vocab"]
        emb = self.flat.view(self.flat.param, "embedding")
        _lib.forge_embed_fwd(self.ids, emb, self.acts[0], T, h, V, self.embed_scale, s)
        if any(ly.cfg.get("n_experts", 0) for ly in self.layers):
            self.aux.zero_()
        for i, ly in enumerate(self.layers):
            ly.fwd(self.acts[i], self.acts[i + 1], aux=self.aux)
        head_args = (self.acts[-1], self.flat.view(self.flat.param, "final_norm"),
                     self.w_lm(self.flat.param), self.targets, self.loss, self.grad_a,
                     self.flat.view(self.flat.grad, "final_norm"), self.w_lm(self.flat.grad),
                     self.head_ws, s)
        if self.ce_chunk:
            _lib.forge_loss_fwd_bwd_chunked(self.head, self.ce_chunk, *head_args)
        else:
            _lib.forge_loss_fwd_bwd(self.head, *head_args)

    def forward_backward(self, accumulate=True):
        """Cross-entropy loss (device scalar) and every gradient accumulated
        into flat.grad; for MoE layers self.aux holds the summed aux losses.
        With accumulate=False the gradients are this step's alone: the layers
        write theirs and only the head / embedding gradients are zeroed."""
        c, s = self.cfg, self.stream
        self._forward_and_head(accumulate)
        g_in, g_out = self.grad_a, self.grad_b
        for i in reversed(range(len(self.layers))):
            self.layers[i].bwd(self.acts[i], g_in, g_out, overwrite=not accumulate)
            g_in, g_out = g_out, g_in
        _lib.forge_embed_bwd(self.ids, g_in, self.flat.view(self.flat.grad, "embedding"),
                             self.T, c["hidden"], c["vocab"], self.embed_scale, s)
        return self.loss

    def train_step_overlapped(self, lr=None, clip=1.0):
        """The step of train_step() with each layer's AdamW update issued
        inside its backward (forge_layer_bwd_adamw), where it overlaps the
        backward of the layers below; the embedding / LM-head and final-norm
        updates follow the embedding backward. The clip coefficient must be
        known before the backward (no norm clipping here). Gives the same
        bits as train_step() for every layer weight."""
        c, s = self.cfg, self.stream
        lr = c["lr"] if lr is None else lr
        self.step_count += 1
        self._forward_and_head(accumulate=False)
        self.scalars[3:4].fill_(clip)
        _lib.forge_adamw_advance(self.scalars, self.dev_step, lr, c["beta1"], c["beta2"], s)
        g_in, g_out = self.grad_a, self.grad_b
        for i in reversed(range(len(self.layers))):
            self.layers[i].bwd_adamw(self.acts[i], g_in, g_out, self.layer_flats[i], self.hp,
                                     self.scalars, overwrite=True)
            g_in, g_out = g_out, g_in
        _lib.forge_embed_bwd(self.ids, g_in, self.flat.view(self.flat.grad, "embedding"),
                             self.T, c["hidden"], c["vocab"], self.embed_scale, s)
        f, n = self.flat, self.head_grad_elems
        _lib.forge_adamw_step(f.master[:n], f.param[:n], f.grad[:n], f.m[:n], f.v[:n], n,
                              self.hp, self.scalars, s)
        return self.loss

    def optimizer_step(self, lr=None, clip=1.0, max_norm=None):
        """One fused AdamW over all parameters. The step count and bias
        corrections advance on the device (no host write: capturable).
        Gradients are scaled by `clip`, or, with `max_norm`, by
        min(1, max_norm / (||g|| + 1e-6)) over the whole flat gradient,
        computed on the device (App. F: norm, clip coefficient and step
        scalars never visit the host)."""
        self.step_count += 1
        c = self.cfg
        lr = c["lr"] if lr is None else lr
        f = self.flat
        if max_norm is None:
            self.scalars[3:4].fill_(clip)
        else:
            self.norm_sq.zero_()
            _lib.forge_grad_norm_sq(f.grad, f.n, self.norm_sq, self.norm_ws, self.stream)
            _lib.forge_clip_coeff(self.norm_sq, max_norm, 1e-6, self.scalars, self.stream)
        _lib.forge_adamw_advance(self.scalars, self.dev_step, lr, c["beta1"], c["beta2"],
                                 self.stream)
        _lib.forge_adamw_step(f.master, f.param, f.grad, f.m, f.v, f.n, self.hp,
                              self.scalars, self.stream)

    def train_step(self, max_norm=None):
        loss = self.forward_backward(accumulate=False)
        self.optimizer_step(max_norm=max_norm)
        return loss


def uses_side_streams(cfg: dict) -> bool:
    """Whether libforge runs a layer's weight gradients and updates on its
    own streams: from 2^20 token x hidden elements (below, the event
    hand-offs cost more than the overlap gains, and one AdamW launch over
    all parameters beats one per weight)."""
    return cfg["batch"] * cfg["seq"] * cfg["hidden"] >= (1 << 20)


class _PrefixedFlat:
    """View of a FlatParams under a name prefix (one layer's tensors)."""

    def __init__(self, flat: FlatParams, prefix: str):
        self._f, self._p = flat, prefix
        self.param, self.grad = flat.param, flat.grad
        self.master, self.m, self.v = flat.master, flat.m, flat.v

    def view(self, buf, name):
        return self._f.view(buf, self._p + name)

    def load_bits(self, name, bits):
        self._f.load_bits(self._p + name, bits)
