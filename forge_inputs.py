"""Seeded synthetic inputs for the decoder training step.

This module is shared by the tests, the bench and the oracle's callers. It
holds the workload shapes and the random draws, and nothing of the method's
arithmetic: no normalisation, attention, loss or optimizer math lives here.
Every array is drawn from NumPy's PCG64 generator from a fixed seed, in fp32,
then rounded once to bfloat16 (round to nearest, ties to even) where the
workload is bf16.

bf16 tensors are carried as ``uint16`` bit patterns (the upper half of an
fp32), so that the exact same bits reach the GPU and the oracle.

Workloads (the paper trains decoder-only GQA / SwiGLU / RMSNorm / RoPE models,
App. B "Model Architectures"; the shapes below are synthetic stand-ins at
Llama-like and MoE-like sizes, since the paper's data and weights are not
available):

* ``tiny``      one layer B1 S128 h256, 4/2 heads of 64, f688, V1024, untied head.
* ``llama8b_layer``  one layer B1 S4096 h4096, 32/8 heads of 128, f14336.
* ``dense1b``   16 layers B4 S2048 h2048, 32/8 heads of 64, f8192, V32000 tied.
* ``llama8b_layer_16k``  as ``llama8b_layer`` at S16384, attention recomputed in bwd.
* ``moe_layer`` one layer B2 S4096 h2048, 16/4 heads of 128, 64 experts top-8, fe1408.
"""
from __future__ import annotations

import copy
import numpy as np

# --------------------------------------------------------------------------
# Workload table
# --------------------------------------------------------------------------

_BASE = dict(
    batch=1, seq=128, hidden=256, n_heads=4, n_kv_heads=2, head_dim=64,
    ffn=688, rope_base=10000.0, rms_eps=1e-5,
    n_experts=0, top_k=0, expert_ffn=0, aux_coef=0.0, recompute_attn=0,
    vocab=0, n_layers=1, tied=False,
    lr=1e-3, beta1=0.9, beta2=0.95, adam_eps=1e-8, weight_decay=0.1,
    init_std=0.02, x_std=1.0, dy_std=1e-2, seed=1,
)


def _cfg(**kw):
    c = dict(_BASE)
    c.update(kw)
    return c


CONFIGS = {
    # tiny layer + untied LM head + CE + AdamW
    "tiny": _cfg(vocab=1024, seed=1),
    # one Llama-8B-shape layer, fwd+bwd
    "llama8b_layer": _cfg(seq=4096, hidden=4096, n_heads=32, n_kv_heads=8,
                          head_dim=128, ffn=14336, rope_base=500000.0, seed=2),
    # 16-layer dense model, tied LM head
    "dense1b": _cfg(batch=4, seq=2048, hidden=2048, n_heads=32, n_kv_heads=8,
                    head_dim=64, ffn=8192, vocab=32000, n_layers=16, tied=True,
                    seed=3),
    # the same model with the streaming cross-entropy head (2048 x 32000
    # logits at a time instead of 8192 x 32000)
    "dense1b_streaming_ce": _cfg(batch=4, seq=2048, hidden=2048, n_heads=32, n_kv_heads=8,
                                 head_dim=64, ffn=8192, vocab=32000, n_layers=16, tied=True,
                                 ce_chunk=2048, seed=3),
    # long-context 8B-shape layer with attention recompute in bwd
    "llama8b_layer_16k": _cfg(seq=16384, hidden=4096, n_heads=32, n_kv_heads=8,
                              head_dim=128, ffn=14336, rope_base=500000.0,
                              recompute_attn=1, seed=4),
    # MoE layer: 64 experts, top-8, expert FFN 1408
    "moe_layer": _cfg(batch=2, seq=4096, hidden=2048, n_heads=16, n_kv_heads=4,
                      head_dim=128, ffn=0, n_experts=64, top_k=8,
                      expert_ffn=1408, aux_coef=1e-2, seed=5),
}


def config(name: str, **overrides) -> dict:
    """A copy of a named workload, with optional overrides (e.g. a shorter seq)."""
    c = copy.deepcopy(CONFIGS[name])
    c.update(overrides)
    c["name"] = name
    return c


def tokens(cfg: dict) -> int:
    return cfg["batch"] * cfg["seq"]


# --------------------------------------------------------------------------
# bf16 bit handling (input preparation only)
# --------------------------------------------------------------------------

def to_bf16_bits(x) -> np.ndarray:
    """fp32 -> bf16 bit pattern, round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> 16) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> 16).astype(np.uint16)


def bf16_bits_to_f32(bits) -> np.ndarray:
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def bf16_bits_to_f64(bits) -> np.ndarray:
    return bf16_bits_to_f32(bits).astype(np.float64)


# --------------------------------------------------------------------------
# Draws
# --------------------------------------------------------------------------

def _normal_bf16(rng, shape, std):
    return to_bf16_bits(rng.standard_normal(shape, dtype=np.float32) * np.float32(std))


def layer_weights(cfg: dict, rng) -> dict:
    """One decoder layer's bf16 weights (nn.Linear convention, [out, in]).

    w_qkv rows are [q heads; k heads; v heads], head-major with the head dim
    contiguous; w_gate_up rows are [gate; up]. Norm gains are 1.
    """
    h, d = cfg["hidden"], cfg["head_dim"]
    hq, hkv = cfg["n_heads"] * d, cfg["n_kv_heads"] * d
    std = cfg["init_std"]
    one = to_bf16_bits(np.ones(h, np.float32))
    w = {
        "attn_norm": one.copy(),
        "w_qkv": _normal_bf16(rng, (hq + 2 * hkv, h), std),
        "w_o": _normal_bf16(rng, (h, hq), std),
        "ffn_norm": one.copy(),
    }
    if cfg["n_experts"] == 0:
        f = cfg["ffn"]
        w["w_gate_up"] = _normal_bf16(rng, (2 * f, h), std)
        w["w_down"] = _normal_bf16(rng, (h, f), std)
    else:
        E, fe = cfg["n_experts"], cfg["expert_ffn"]
        w["w_router"] = _normal_bf16(rng, (E, h), std)
        w["w_gate_up_e"] = _normal_bf16(rng, (E, 2 * fe, h), std)
        w["w_down_e"] = _normal_bf16(rng, (E, h, fe), std)
    return w


def layer_inputs(cfg: dict, seed: int | None = None) -> dict:
    """Weights, input activations x ~ N(0, x_std) and upstream grad dy."""
    rng = np.random.default_rng(cfg["seed"] if seed is None else seed)
    T, h = tokens(cfg), cfg["hidden"]
    w = layer_weights(cfg, rng)
    x = _normal_bf16(rng, (T, h), cfg["x_std"])
    dy = _normal_bf16(rng, (T, h), cfg["dy_std"])
    return {"weights": w, "x": x, "dy": dy}


def model_inputs(cfg: dict, seed: int | None = None) -> dict:
    """Embedding, layers, final norm, LM head (absent when tied), ids, targets."""
    rng = np.random.default_rng(cfg["seed"] if seed is None else seed)
    T, h, V = tokens(cfg), cfg["hidden"], cfg["vocab"]
    emb = _normal_bf16(rng, (V, h), cfg["init_std"])
    layers = [layer_weights(cfg, rng) for _ in range(cfg["n_layers"])]
    final_norm = to_bf16_bits(np.ones(h, np.float32))
    w_lm = None if cfg["tied"] else _normal_bf16(rng, (V, h), cfg["init_std"])
    ids = rng.integers(0, V, size=T, dtype=np.int32)
    targets = rng.integers(0, V, size=T, dtype=np.int32)
    return {"embedding": emb, "layers": layers, "final_norm": final_norm,
            "w_lm": w_lm, "ids": ids, "targets": targets}


def router_logits(T: int, E: int, seed: int) -> np.ndarray:
    """fp32 router logits ~ N(0, 1) for the routing test."""
    rng = np.random.default_rng(seed)
    return rng.standard_normal((T, E), dtype=np.float32)


def optimizer_inputs(n: int, seed: int, grad_std: float = 1e-2,
                     step: int = 1) -> dict:
    """fp32 master / grad / moments for an optimizer-only test.

    At step 1 the moments are zero; for later steps they hold plausible
    running averages (m ~ N(0, grad_std), v ~ grad_std^2 * U(0.5, 1.5)).
    """
    rng = np.random.default_rng(seed)
    master = bf16_bits_to_f32(_normal_bf16(rng, n, 0.02))
    grad = (rng.standard_normal(n, dtype=np.float32) * np.float32(grad_std))
    if step == 1:
        m = np.zeros(n, np.float32)
        v = np.zeros(n, np.float32)
    else:
        m = rng.standard_normal(n, dtype=np.float32) * np.float32(grad_std)
        v = (rng.uniform(0.5, 1.5, n).astype(np.float32)
             * np.float32(grad_std) ** 2)
    return {"master": master, "grad": grad.astype(np.float32), "m": m, "v": v}
