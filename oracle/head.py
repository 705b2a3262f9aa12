"""Oracle: embedding, final norm + LM head + softmax cross-entropy, model step.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The output head is the fp32 softmax cross-entropy the engines fuse
(App. A, framework-level trajectory, fused cross-entropy steps; App. G,
fused NPU cross-entropy in FP32), after a final RMSNorm, optionally with the LM head tied to the input
embedding (App. B, "Tied input/output embeddings").

Readings where the paper is silent:
  * loss = (1/T) sum_t (logsumexp(z_t) - z_t[y_t]) over all T tokens, no
    ignore index; the targets are given (not derived by shifting the ids).
  * Tied head: the LM head matrix is the embedding matrix, and its gradient is
    the sum of the head's weight gradient and the embedding scatter-add.
  * muP scalars of the MiniCPM models (App. B: scale_emb, dim_model_base,
    scale_depth), read as in their public model definition: the embedding
    output is multiplied by scale_emb, each residual branch by
    scale_depth / sqrt(n_layers) (the layers' branch_scale), and the logits
    by dim_model_base / hidden (the final hidden state divided by
    hidden / dim_model_base before the LM head). Off unless the config sets
    them.
  * dense_first_layers (MiniCPM5 16B-A3B, App. B): the first layers of a MoE
    model use the dense FFN of width ffn; the others are routed.
"""
from __future__ import annotations

import numpy as np

from . import dense, moe


def embed_fwd(ids, E, scale=1.0):
    """x0[t] = scale * E[ids[t]]."""
    return scale * E[np.asarray(ids)]


def embed_bwd(ids, dx0, vocab, scale=1.0):
    """dE[v] = scale * sum over t with ids[t] = v of dx0[t]."""
    dE = np.zeros((vocab, dx0.shape[1]))
    np.add.at(dE, np.asarray(ids), scale * dx0)
    return dE


def logsumexp(z):
    m = np.max(z, axis=1)
    return m + np.log(np.sum(np.exp(z - m[:, None]), axis=1))


def cross_entropy(z, targets):
    """Mean over tokens of logsumexp(z_t) - z_t[y_t], and dloss/dz."""
    T = z.shape[0]
    lse = logsumexp(z)
    t = np.asarray(targets)
    loss = np.mean(lse - z[np.arange(T), t])
    dz = np.exp(z - lse[:, None])
    dz[np.arange(T), t] -= 1.0
    return loss, dz / T


def head_fwd_bwd(xL, gf, w_lm, targets, eps, logit_scale=1.0):
    """Final RMSNorm, logits z = logit_scale RMSNorm(xL) W_lm^T, mean CE, and
    all grads.

    Returns (loss, dxL, dgf, dW_lm).
    """
    xn, r = dense.rmsnorm_fwd(xL, gf, eps)
    z = logit_scale * (xn @ w_lm.T)
    loss, dz = cross_entropy(z, targets)
    dz = logit_scale * dz
    dw = dz.T @ xn
    dxn = dz @ w_lm
    dxL, dgf = dense.rmsnorm_bwd(xL, gf, r, dxn)
    return loss, dxL, dgf, dw


def layer_cfg(cfg, i):
    """Configuration of layer i of a model: dense for the first
    cfg["dense_first_layers"] layers of a MoE model, else cfg itself."""
    if cfg.get("n_experts", 0) and i < cfg.get("dense_first_layers", 0):
        return dict(cfg, n_experts=0, top_k=0, expert_ffn=0, shared_ffn=0)
    return cfg


def model_fwd_bwd(P, ids, targets, cfg, route_idx=None):
    """Whole model: embedding, layers, final norm, head, CE; then backward.

    P holds 'embedding' [V, h], 'layers' (list of weight dicts),
    'final_norm' [h] and 'w_lm' [V, h] (None when tied). Returns
    (loss, grads) with grads mirroring P. For MoE layers the loss includes
    the per-layer aux losses. route_idx: optional {layer index: [T, k]
    experts} forcing those layers' choice of experts (see moe.route).
    """
    V = cfg["vocab"]
    tied = P["w_lm"] is None
    w_lm = P["embedding"] if tied else P["w_lm"]
    es = cfg.get("embed_scale", 1.0) or 1.0
    ls = cfg.get("logit_scale", 1.0) or 1.0
    x = embed_fwd(ids, P["embedding"], es)
    caches, aux_total = [], 0.0
    for i, W in enumerate(P["layers"]):
        lc = layer_cfg(cfg, i)
        if lc["n_experts"]:
            x, aux, c = moe.layer_fwd(x, W, lc, (route_idx or {}).get(i))
            aux_total += aux
        else:
            x, c = dense.layer_fwd(x, W, lc)
        caches.append(c)
    loss, dx, dgf, dw_lm = head_fwd_bwd(x, P["final_norm"], w_lm, targets,
                                        cfg["rms_eps"], ls)
    grads = {"layers": [None] * len(P["layers"]), "final_norm": dgf}
    for i in reversed(range(len(P["layers"]))):
        lc = layer_cfg(cfg, i)
        mod = moe if lc["n_experts"] else dense
        dx, grads["layers"][i] = mod.layer_bwd(caches[i], P["layers"][i], lc, dx)
    dE = embed_bwd(ids, dx, V, es)
    if tied:
        grads["embedding"] = dE + dw_lm
        grads["w_lm"] = None
    else:
        grads["embedding"] = dE
        grads["w_lm"] = dw_lm
    return loss + aux_total, grads
