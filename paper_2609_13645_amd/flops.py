"""Model-FLOP count used for MFU (App. C, "Model-FLOPs Utilization").

A multiply-accumulate counts two FLOPs. Forward FLOPs per token:

  attention projections  2 h (hq + 2 hkv) + 2 hq h
  FFN (SwiGLU)           2 (2 h f) + 2 f h
  attention core         2 n_h s d       (causal factor 1/2 folded in)
  output head            2 h V

Each per-layer term is tripled (one forward, two backward) and summed over
the layers; the head is counted once at the same 1:2 ratio. Recomputation is
not model FLOPs (it counts toward hardware FLOPs only).

MoE extension (the paper's formula is dense only): the FFN term becomes
top_k * 6 h fe (each token runs k SwiGLU experts) plus the router 2 h E,
plus 6 h fs for a shared expert of width fs; routing, permutation and
combine are not counted. The first dense_first_layers layers of a MoE model
count as dense layers. QK-Norm and the muP scalars add no model FLOPs.
"""
from __future__ import annotations


def per_token_fwd(hidden, n_heads, n_kv_heads, head_dim, seq, ffn=0, vocab=0,
                  n_experts=0, top_k=0, expert_ffn=0, shared_ffn=0):
    """Forward FLOPs per token by operator class, for one layer (+ head)."""
    h, d = hidden, head_dim
    hq, hkv = n_heads * d, n_kv_heads * d
    out = {
        "attn_proj": 2 * h * (hq + 2 * hkv) + 2 * hq * h,
        "attn_core": 2 * n_heads * seq * d,
        "head": 2 * h * vocab,
    }
    if n_experts:
        out["ffn"] = top_k * 6 * h * expert_ffn + 2 * h * n_experts + 6 * h * shared_ffn
    else:
        out["ffn"] = 2 * (2 * h * ffn) + 2 * ffn * h
    return out


def per_token(cfg: dict, with_head: bool | None = None) -> dict:
    """fwd+bwd FLOPs per token by class for a workload dict (n_layers layers).

    with_head defaults to vocab > 0.
    """
    L = cfg.get("n_layers", 1)
    if with_head is None:
        with_head = cfg.get("vocab", 0) > 0
    res = {"attn_proj": 0, "attn_core": 0, "ffn": 0, "head": 0}
    for i in range(L):
        dense = not cfg.get("n_experts", 0) or i < cfg.get("dense_first_layers", 0)
        f = per_token_fwd(cfg["hidden"], cfg["n_heads"], cfg["n_kv_heads"],
                          cfg["head_dim"], cfg["seq"], cfg.get("ffn", 0),
                          cfg.get("vocab", 0), 0 if dense else cfg["n_experts"],
                          0 if dense else cfg.get("top_k", 0),
                          0 if dense else cfg.get("expert_ffn", 0),
                          0 if dense else cfg.get("shared_ffn", 0))
        for k in ("attn_proj", "attn_core", "ffn"):
            res[k] += 3 * f[k]
    if with_head:
        res["head"] = 3 * 2 * cfg["hidden"] * cfg.get("vocab", 0)
    res["total"] = sum(res.values())
    return res


def step_flops(cfg: dict, with_head: bool | None = None) -> float:
    """Model FLOPs of one fwd+bwd step over batch * seq tokens."""
    return per_token(cfg, with_head)["total"] * cfg["batch"] * cfg["seq"]


def recompute_flops(cfg: dict) -> float:
    """Extra hardware FLOPs of re-running the attention core forward in bwd."""
    if not cfg.get("recompute_attn"):
        return 0.0
    f = per_token_fwd(cfg["hidden"], cfg["n_heads"], cfg["n_kv_heads"],
                      cfg["head_dim"], cfg["seq"])
    return f["attn_core"] * cfg.get("n_layers", 1) * cfg["batch"] * cfg["seq"]
