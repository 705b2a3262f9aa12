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

Model variants of App. B (shapes of the paper's own models, one layer each):

* ``qwen3_layer``  Qwen3-0.6B-shape layer with per-head QK-Norm: B4 S4096 h1024,
  16/8 heads of 128, f3072, RoPE base 1e6, RMSNorm eps 1e-6.
* ``minicpm5_moe_layer``  MiniCPM5-16B-A3B-shape MoE layer: B4 S4096 h2048,
  32/2 heads of 128, 160 routed experts top-16 of width 512 plus a 512-wide
  shared expert, eps 1e-6, muP branch scale 1.4 / sqrt(28).
* ``packed_docs_layer``  the 8B-shape layer over rows packed with documents
  of random lengths, RoPE positions restarting at each document.
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
    qk_norm=0, branch_scale=0.0, shared_ffn=0, dense_first_layers=0,
    embed_scale=0.0, logit_scale=0.0, packed_docs=0,
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
    # Qwen3-0.6B-shape layer, per-head QK-Norm
    "qwen3_layer": _cfg(batch=4, seq=4096, hidden=1024, n_heads=16, n_kv_heads=8,
                        head_dim=128, ffn=3072, rope_base=1e6, rms_eps=1e-6, qk_norm=1,
                        seed=6),
    # MiniCPM5-16B-A3B-shape MoE layer: 160 experts top-16, shared expert,
    # muP branch scale scale_depth / sqrt(n_layers) = 1.4 / sqrt(28)
    "minicpm5_moe_layer": _cfg(batch=4, seq=4096, hidden=2048, n_heads=32, n_kv_heads=2,
                               head_dim=128, ffn=0, n_experts=160, top_k=16,
                               expert_ffn=512, shared_ffn=512, aux_coef=1e-2, rms_eps=1e-6,
                               branch_scale=1.4 / 28 ** 0.5, seed=7),
    # the 8B-shape layer over packed documents (document-aware RoPE)
    "packed_docs_layer": _cfg(seq=4096, hidden=4096, n_heads=32, n_kv_heads=8,
                              head_dim=128, ffn=14336, rope_base=500000.0, packed_docs=512,
                              seed=8),
}


def config(name: str, **overrides) -> dict:
    """A copy of a named workload, with optional overrides (e.g. a shorter seq).

    A workload with packed_docs = L gets RoPE positions (key "positions") of
    rows packed with documents of mean length L (doc_positions)."""
    c = copy.deepcopy(CONFIGS[name])
    c.update(overrides)
    c["name"] = name
    if c.get("packed_docs") and "positions" not in overrides:
        c["positions"] = doc_positions(c["batch"], c["seq"], c["packed_docs"], c["seed"])
    return c


def doc_positions(batch: int, seq: int, mean_len: int, seed: int) -> np.ndarray:
    """RoPE positions of rows packed with documents: each batch row is cut
    into documents of lengths 1 + Geometric(1 / mean_len) (the last one cut
    at the row end), and a token's position is its offset in its document.
    int32 [batch * seq]."""
    rng = np.random.default_rng(seed + 1000)
    pos = np.empty(batch * seq, np.int32)
    for b in range(batch):
        t = 0
        while t < seq:
            n = min(int(rng.geometric(1.0 / mean_len)), seq - t)
            pos[b * seq + t:b * seq + t + n] = np.arange(n, dtype=np.int32)
            t += n
    return pos


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
        fs = cfg.get("shared_ffn", 0)
        if fs:
            w["w_gate_up_s"] = _normal_bf16(rng, (2 * fs, h), std)
            w["w_down_s"] = _normal_bf16(rng, (h, fs), std)
    if cfg.get("qk_norm", 0):
        w["q_norm"] = to_bf16_bits(np.ones(d, np.float32))
        w["k_norm"] = to_bf16_bits(np.ones(d, np.float32))
    return w


def model_layer_cfg(cfg: dict, i: int) -> dict:
    """Layer i's configuration: the first dense_first_layers layers of a MoE
    model are dense (FFN width ffn)."""
    if cfg.get("n_experts", 0) and i < cfg.get("dense_first_layers", 0):
        return dict(cfg, n_experts=0, top_k=0, expert_ffn=0, shared_ffn=0)
    return cfg


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
    layers = [layer_weights(model_layer_cfg(cfg, i), rng) for i in range(cfg["n_layers"])]
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
