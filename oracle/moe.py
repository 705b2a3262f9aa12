"""Oracle: top-k softmax-routed mixture-of-experts FFN, fp64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper's sparse model replaces the dense SwiGLU FFN by routed experts
(App. B, Table "H100 architecture configurations": MiniCPM5 16B-A3B, routed
experts with top-k selection). The workload here is dropless (no capacity),
with a softmax router and a load-balance auxiliary loss.

Readings where the paper is silent:
  * p = softmax(l) over all E experts; gate of a chosen expert = its p, with
    no renormalisation over the top k.
  * The top-k set and its order: descending logit, ties to the lower expert
    id. The decision is taken on the logits rounded to fp32, the precision in
    which the GPU path holds them, so that both sides decide in one precision.
  * Canonical permutation: expert-major, tokens ascending within an expert,
    then slot ascending; entries are flat (token * k + slot) indices.
  * Aux loss (Switch style): alpha * E * sum_e f_e P_e with f_e = count_e / (T k)
    (no gradient) and P_e = mean_t p_te.
  * Shared expert (MiniCPM5 16B-A3B's 512-wide shared expert, App. B): with
    cfg["shared_ffn"] = fs > 0, every token also goes through one SwiGLU FFN
    of width fs (w_gate_up_s [2fs, h], w_down_s [h, fs]) with weight 1, added
    to the routed experts' sum; the router does not see it.
  * branch_scale (muP): the whole FFN branch (routed + shared) is multiplied
    by it; the aux loss is not.
"""
from __future__ import annotations

import numpy as np

from .dense import rmsnorm_fwd, rmsnorm_bwd, swiglu_fwd, swiglu_bwd, \
    attention_block_fwd, attention_block_bwd


def softmax(l):
    m = np.max(l, axis=-1, keepdims=True)
    e = np.exp(l - m)
    return e / np.sum(e, axis=-1, keepdims=True)


def topk(l32, k):
    """Indices of the k largest entries per row, descending, ties to lower id."""
    order = np.argsort(-np.asarray(l32, dtype=np.float64), axis=1, kind="stable")
    return order[:, :k].astype(np.int32)


def topk_margin(l32, k):
    """Per row, how far the k-th largest logit lies above the (k+1)-th (fp64
    difference of the fp32 values). A perturbation of the logits smaller than
    half of it in every entry cannot change the top-k set; when k equals the
    number of experts the set is fixed and the margin is infinite.
    """
    v = -np.sort(-np.asarray(l32, dtype=np.float32).astype(np.float64), axis=1)
    if k >= v.shape[1]:
        return np.full(v.shape[0], np.inf)
    return v[:, k - 1] - v[:, k]


def route(l, k, idx=None):
    """Routing decision for logits l [T, E].

    Returns idx [T, k] int32, gates [T, k], p [T, E], counts [E] int32,
    offsets [E + 1] int32 (exclusive scan of counts), perm [T k] int32.

    With `idx` given, that choice of experts is taken instead of the top-k of
    l (k distinct experts per token, in [0, E)): for a token whose k-th and
    (k+1)-th logits lie within rounding of each other, either choice is a
    correct top-k, and the caller may follow the one another implementation
    made. Everything downstream (gates, counts, order) follows from it.
    """
    T, E = l.shape
    if idx is None:
        idx = topk(np.asarray(l, dtype=np.float32), k)
    else:
        idx = np.asarray(idx, dtype=np.int32)
        assert idx.shape == (T, k) and idx.min() >= 0 and idx.max() < E
        assert all(len(set(r)) == k for r in idx.tolist()), "experts repeat in a row"
    p = softmax(np.asarray(l, dtype=np.float64))
    gates = np.take_along_axis(p, idx, axis=1)
    counts = np.bincount(idx.reshape(-1), minlength=E).astype(np.int32)
    offsets = np.zeros(E + 1, np.int32)
    offsets[1:] = np.cumsum(counts)
    flat = idx.reshape(-1)
    # canonical order: expert, then flat (token, slot) index ascending
    perm = np.lexsort((np.arange(T * k), flat)).astype(np.int32)
    return idx, gates, p, counts, offsets, perm


def aux_loss(p, counts, k, alpha):
    """alpha * E * sum_e f_e P_e."""
    T, E = p.shape
    f = counts.astype(np.float64) / (T * k)
    P = np.mean(p, axis=0)
    return alpha * E * np.sum(f * P)


def expert_ffn(xe, wgu, wd, fe):
    """SwiGLU expert on rows xe: (silu(xe Wg^T) * (xe Wu^T)) Wd^T."""
    gu = xe @ wgu.T
    G, U = gu[:, :fe], gu[:, fe:]
    A = swiglu_fwd(G, U)
    return A @ wd.T, (G, U, A)


def moe_fwd(b, W, cfg, idx=None):
    """y_t = sum_{e in topk(t)} p_te * FFN_e(b_t); also returns the aux loss.

    Grouped form: rows gathered per expert in canonical order, one dense
    product per expert, scattered back weighted by the gate. `idx` forces the
    choice of experts (see route).
    """
    T, h = b.shape
    E, k, fe = cfg["n_experts"], cfg["top_k"], cfg["expert_ffn"]
    l = b @ W["w_router"].T
    idx, gates, p, counts, offsets, perm = route(l, k, idx)
    y = np.zeros_like(b)
    per_expert = []
    for e in range(E):
        rows = perm[offsets[e]:offsets[e + 1]]
        tok, slot = rows // k, rows % k
        ye, acts = expert_ffn(b[tok], W["w_gate_up_e"][e], W["w_down_e"][e], fe)
        np.add.at(y, tok, gates[tok, slot][:, None] * ye)
        per_expert.append((tok, slot, ye, acts))
    aux = aux_loss(p, counts, k, cfg["aux_coef"])
    cache = dict(b=b, l=l, idx=idx, gates=gates, p=p, counts=counts,
                 offsets=offsets, perm=perm, per_expert=per_expert)
    return y, aux, cache


def moe_bwd(c, W, cfg, dy):
    """Backward of moe_fwd for the objective <y, dy> + aux.

      dgate_tj = dy_t . FFN_e(b_t)
      dp_te = dgate (chosen e) + alpha E f_e / T (aux, every e)
      dl = p (dp - sum_e p_e dp_e)
    """
    b, p = c["b"], c["p"]
    T, h = b.shape
    E, k, fe = cfg["n_experts"], cfg["top_k"], cfg["expert_ffn"]
    g = {"w_gate_up_e": np.zeros_like(W["w_gate_up_e"]),
         "w_down_e": np.zeros_like(W["w_down_e"])}
    db = np.zeros_like(b)
    dp = np.zeros_like(p)
    for e in range(E):
        tok, slot, ye, (G, U, A) = c["per_expert"][e]
        gate = c["gates"][tok, slot][:, None]
        np.add.at(dp, (tok, np.full(tok.shape, e)), np.sum(dy[tok] * ye, axis=1))
        dye = gate * dy[tok]
        g["w_down_e"][e] = dye.T @ A
        dA = dye @ W["w_down_e"][e]
        dG, dU = swiglu_bwd(G, U, dA)
        dgu = np.concatenate([dG, dU], axis=1)
        g["w_gate_up_e"][e] = dgu.T @ b[tok]
        np.add.at(db, tok, dgu @ W["w_gate_up_e"][e])
    f = c["counts"].astype(np.float64) / (T * k)
    dp += cfg["aux_coef"] * E * f[None, :] / T
    dl = p * (dp - np.sum(p * dp, axis=1, keepdims=True))
    g["w_router"] = dl.T @ b
    db += dl @ W["w_router"]
    return db, g


def moe_fwd_per_token(b, W, cfg):
    """Brute-force reference: each token through its chosen experts one by one."""
    T, h = b.shape
    k, fe = cfg["top_k"], cfg["expert_ffn"]
    l = b @ W["w_router"].T
    p = softmax(l)
    idx = topk(np.asarray(l, np.float32), k)
    y = np.zeros_like(b)
    for t in range(T):
        for j in range(k):
            e = idx[t, j]
            ye, _ = expert_ffn(b[t:t + 1], W["w_gate_up_e"][e], W["w_down_e"][e], fe)
            y[t] += p[t, e] * ye[0]
    return y


def shared_fwd(b, W, cfg):
    """The shared expert on every token: (silu(b Wg^T) * (b Wu^T)) Wd^T."""
    return expert_ffn(b, W["w_gate_up_s"], W["w_down_s"], cfg["shared_ffn"])


def layer_fwd(x, W, cfg, idx=None):
    """MoE decoder layer: attention block, then h1 + s (MoE + shared)(RMSNorm(h1)).

    Returns (out, aux, cache). `idx` forces the choice of experts (see route).
    """
    bs = cfg.get("branch_scale", 1.0) or 1.0
    h1, ca = attention_block_fwd(x, W, cfg)
    bn, r2 = rmsnorm_fwd(h1, W["ffn_norm"], cfg["rms_eps"])
    y, aux, cm = moe_fwd(bn, W, cfg, idx)
    if cfg.get("shared_ffn", 0):
        ys, cm["shared"] = shared_fwd(bn, W, cfg)
        y = y + ys
    return h1 + bs * y, aux, dict(attn=ca, moe=cm, h1=h1, r2=r2)


def layer_bwd(cache, W, cfg, dout):
    """Backward of layer_fwd for the objective <out, dout> + aux."""
    bs = cfg.get("branch_scale", 1.0) or 1.0
    # <h1 + s y, dout> + aux: the branch sees s dout, the aux term is unscaled
    db, g = moe_bwd(cache["moe"], W, cfg, bs * dout)
    if cfg.get("shared_ffn", 0):
        fs = cfg["shared_ffn"]
        G, U, A = cache["moe"]["shared"]
        dy = bs * dout
        g["w_down_s"] = dy.T @ A
        dG, dU = swiglu_bwd(G, U, dy @ W["w_down_s"])
        dgu = np.concatenate([dG, dU], axis=1)
        g["w_gate_up_s"] = dgu.T @ cache["moe"]["b"]
        db = db + dgu @ W["w_gate_up_s"]
    dh1n, g["ffn_norm"] = rmsnorm_bwd(cache["h1"], W["ffn_norm"], cache["r2"], db)
    dx, ga = attention_block_bwd(cache["attn"], W, cfg, dout + dh1n)
    g.update(ga)
    return dx, g


def layer_fwd_rows(x, W, cfg, rows, with_logits=False):
    """MoE layer output at selected token rows only (the same definition).

    Attention needs every key, so it runs through dense.layer_fwd_rows'
    pieces; the routed FFN of a token depends on that token alone. With
    with_logits, also returns the router logits of those rows.
    """
    from . import dense
    h, nh, nkv, d, hq, hkv = dense._dims(cfg)
    rows = np.asarray(rows)
    # h1 at the selected rows: attention block only (FFN of the dense helper unused)
    B, S, base = cfg["batch"], cfg["seq"], cfg["rope_base"]
    T = x.shape[0]
    a, _ = dense.rmsnorm_fwd(x, W["attn_norm"], cfg["rms_eps"])
    wq, wk, wv = W["w_qkv"][:hq], W["w_qkv"][hq:hq + hkv], W["w_qkv"][hq + hkv:]
    k_ = dense.rope_fwd((a @ wk.T).reshape(T, nkv, d), B, S, base)
    v_ = (a @ wv.T).reshape(T, nkv, d)
    phi = dense.rope_angles(S, d, base)[rows % S]
    cs, sn = np.cos(phi)[:, None, :], np.sin(phi)[:, None, :]
    q = (a[rows] @ wq.T).reshape(len(rows), nh, d)
    q1, q2 = q[..., : d // 2], q[..., d // 2:]
    q = np.concatenate([q1 * cs - q2 * sn, q2 * cs + q1 * sn], axis=-1)
    grp = nh // nkv
    o = np.zeros((len(rows), nh, d))
    for r, t in enumerate(rows):
        keys = slice((t // S) * S, t + 1)
        for n in range(nh):
            s = (k_[keys, n // grp] @ q[r, n]) / np.sqrt(d)
            p = np.exp(s - s.max())
            o[r, n] = (p / p.sum()) @ v_[keys, n // grp]
    h1 = x[rows] + o.reshape(len(rows), hq) @ W["w_o"].T
    bn, _ = dense.rmsnorm_fwd(h1, W["ffn_norm"], cfg["rms_eps"])
    out = h1 + moe_fwd_per_token(bn, W, cfg)
    return (out, bn @ W["w_router"].T) if with_logits else out
