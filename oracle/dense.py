"""Oracle: dense pre-norm decoder layer, forward and backward, fp64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The layer is the decoder block of App. B ("Model Architectures"): grouped-query
attention, SwiGLU feed-forward, pre-normalisation RMSNorm, RoPE. Attention is
causal (App. C, the causal factor of the attention-core count). The backward
is written out by hand (the paper's engines use a static hand-written
backward, App. J, and count the backward of every GEMM as one data-gradient
and one weight-gradient product, App. C).

Readings where the paper is silent:
  * RMSNorm: y = x * (mean(x^2) + eps)^(-1/2) * g, per token over the hidden dim.
  * RoPE: rotate-half pairs (i, i + d/2), angle pos * base^(-2i/d), i < d/2;
    positions restart at 0 in every batch row; q and k rotated, v not.
  * GQA: contiguous groups, query head n reads key/value head n // (n_h / n_kv).
  * Attention scale 1/sqrt(d); key j visible to query i iff j <= i, same row.
  * Fused weight order: w_qkv rows [q heads; k heads; v heads], head-major;
    w_gate_up rows [gate; up]; nn.Linear convention y = x W^T.
  * Layer order (Llama): a = RMSNorm(x); h1 = x + Attn(a) W_o^T;
    b = RMSNorm(h1); out = h1 + (silu(b W_g^T) * (b W_u^T)) W_d^T.

Model variants of App. B, each off unless the config asks for it:
  * qk_norm (Qwen3's per-head QK-Norm): every q and k head vector is
    RMS-normalised over head_dim with gains q_norm / k_norm [head_dim] (shared
    by the heads), before RoPE: q <- RoPE(RMSNorm_d(q; q_norm)), same for k.
  * positions (document-aware RoPE, App. A step 23): cfg["positions"] [T]
    gives each token's RoPE position (e.g. its offset inside its document in
    a packed row); absent, a token's position is its index in its batch row.
    Attention stays causal over the whole batch row.
  * branch_scale (MiniCPM's muP scale_depth / sqrt(n_layers)): both residual
    branches are multiplied by it, h1 = x + s Attn, out = h1 + s FFN.

Shapes: x is [T, h] with T = batch * seq, batch-row major.
"""
from __future__ import annotations

import numpy as np


# --------------------------------------------------------------------------
# RMSNorm
# --------------------------------------------------------------------------

def rmsnorm_fwd(x, g, eps):
    """y = x * r * g with r = (mean_j x_j^2 + eps)^(-1/2). Returns (y, r)."""
    r = 1.0 / np.sqrt(np.mean(x * x, axis=-1) + eps)
    return x * r[:, None] * g[None, :], r


def rmsnorm_bwd(x, g, r, dy):
    """Gradients of y = x r g.

    With dr/dx_k = -r^3 x_k / h:
      dx_k = r (g dy)_k - r^3 x_k / h * sum_j (g dy)_j x_j
      dg_j = sum_t dy_tj x_tj r_t
    """
    h = x.shape[-1]
    gd = dy * g[None, :]
    proj = np.sum(gd * x, axis=-1)
    dx = gd * r[:, None] - x * (r ** 3 * proj / h)[:, None]
    dg = np.sum(dy * x * r[:, None], axis=0)
    return dx, dg


# --------------------------------------------------------------------------
# RoPE
# --------------------------------------------------------------------------

def rope_angles(seq, head_dim, base, pos=None):
    """phi[s, i] = pos_s * base^(-2i/d) for i < d/2 (fp64); pos defaults to
    0 .. seq-1."""
    i = np.arange(head_dim // 2, dtype=np.float64)
    inv_freq = base ** (-2.0 * i / head_dim)
    p = np.arange(seq, dtype=np.float64) if pos is None else np.asarray(pos, np.float64)
    return p[:, None] * inv_freq[None, :]


def _positions(batch, seq, pos=None):
    return np.tile(np.arange(seq), batch) if pos is None else np.asarray(pos)


def rope_fwd(x, batch, seq, base, pos=None):
    """Rotate each head of x [T, n, d] by its token's angles (rotate-half).

    y_i = x_i cos - x_{i+d/2} sin,  y_{i+d/2} = x_{i+d/2} cos + x_i sin.
    pos [T]: the tokens' positions (default: index within the batch row).
    """
    d = x.shape[-1]
    phi = rope_angles(0, d, base, _positions(batch, seq, pos))      # [T, d/2]
    c, s = np.cos(phi)[:, None, :], np.sin(phi)[:, None, :]
    x1, x2 = x[..., : d // 2], x[..., d // 2:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def rope_bwd(dy, batch, seq, base, pos=None):
    """Transpose of the rotation (rotation by -phi)."""
    d = dy.shape[-1]
    phi = rope_angles(0, d, base, _positions(batch, seq, pos))
    c, s = np.cos(phi)[:, None, :], np.sin(phi)[:, None, :]
    d1, d2 = dy[..., : d // 2], dy[..., d // 2:]
    return np.concatenate([d1 * c + d2 * s, d2 * c - d1 * s], axis=-1)


# --------------------------------------------------------------------------
# Causal grouped-query attention (naive, full score matrix per head)
# --------------------------------------------------------------------------

def attention_probs(q, k, scale):
    """Causal row-softmax of q k^T * scale for one (row, head): [S, S]."""
    S = q.shape[0]
    s = (q @ k.T) * scale
    s = np.where(np.tril(np.ones((S, S), dtype=bool)), s, -np.inf)
    m = np.max(s, axis=1, keepdims=True)
    e = np.exp(s - m)
    l = np.sum(e, axis=1, keepdims=True)
    return e / l, (m + np.log(l))[:, 0]


# Threads for the per-(batch row, kv head) loops of attention_fwd / _bwd. Each
# task runs one kv head's query group in head order, exactly the serial
# arithmetic, on slices no other task writes; more than one thread only
# shortens the wall time on long sequences (NumPy releases the interpreter
# lock inside its array operations).
ATTENTION_WORKERS = 1
# Optional callable(b, m), told when a kv head's group is done (for callers
# that report progress on long sequences).
ATTENTION_PROGRESS = None


def _for_each_kv_head(batch, nkv, task, workers):
    jobs = [(b, m) for b in range(batch) for m in range(nkv)]

    def run(b, m):
        task(b, m)
        if ATTENTION_PROGRESS is not None:
            ATTENTION_PROGRESS(b, m)

    if workers <= 1:
        for j in jobs:
            run(*j)
        return
    from concurrent.futures import ThreadPoolExecutor
    with ThreadPoolExecutor(workers) as ex:
        for f in [ex.submit(run, *j) for j in jobs]:
            f.result()


def attention_fwd(q, k, v, batch, seq, workers=None):
    """o_i = sum_{j<=i} softmax_j(q_i.k_j / sqrt(d)) v_j per head.

    q [T, n_h, d], k/v [T, n_kv, d]. Returns o [T, n_h, d] and the row
    log-sum-exp lse [batch, n_h, seq].
    """
    T, nh, d = q.shape
    nkv = k.shape[1]
    grp = nh // nkv
    scale = 1.0 / np.sqrt(d)
    o = np.zeros_like(q)
    lse = np.zeros((batch, nh, seq))

    def group(b, m):
        rows = slice(b * seq, (b + 1) * seq)
        for n in range(m * grp, (m + 1) * grp):
            P, lse[b, n] = attention_probs(q[rows, n], k[rows, m], scale)
            o[rows, n] = P @ v[rows, m]

    _for_each_kv_head(batch, nkv, group, ATTENTION_WORKERS if workers is None else workers)
    return o, lse


def attention_bwd(q, k, v, do, batch, seq, workers=None):
    """Softmax-attention backward, per head, summed over each GQA group.

      dv_j = sum_i P_ij do_i
      dP_ij = do_i . v_j
      ds_ij = P_ij (dP_ij - sum_l P_il dP_il)
      dq_i = scale sum_j ds_ij k_j,   dk_j = scale sum_i ds_ij q_i
    """
    T, nh, d = q.shape
    nkv = k.shape[1]
    grp = nh // nkv
    scale = 1.0 / np.sqrt(d)
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)

    def group(b, m):
        rows = slice(b * seq, (b + 1) * seq)
        for n in range(m * grp, (m + 1) * grp):
            P, _ = attention_probs(q[rows, n], k[rows, m], scale)
            dO = do[rows, n]
            dv[rows, m] += P.T @ dO
            dP = dO @ v[rows, m].T
            ds = P * (dP - np.sum(P * dP, axis=1, keepdims=True))
            dq[rows, n] = scale * (ds @ k[rows, m])
            dk[rows, m] += scale * (ds.T @ q[rows, n])

    _for_each_kv_head(batch, nkv, group, ATTENTION_WORKERS if workers is None else workers)
    return dq, dk, dv


# --------------------------------------------------------------------------
# SwiGLU
# --------------------------------------------------------------------------

def sigmoid(x):
    return 0.5 * (1.0 + np.tanh(0.5 * x))


def silu(x):
    return x * sigmoid(x)


def swiglu_fwd(G, U):
    """A = silu(G) * U."""
    return silu(G) * U


def swiglu_bwd(G, U, dA):
    """dG = dA U silu'(G) with silu'(G) = s (1 + G (1 - s)), s = sigmoid(G);
    dU = dA silu(G)."""
    s = sigmoid(G)
    return dA * U * s * (1.0 + G * (1.0 - s)), dA * G * s


# --------------------------------------------------------------------------
# Dense layer
# --------------------------------------------------------------------------

def _dims(cfg):
    d = cfg["head_dim"]
    return cfg["hidden"], cfg["n_heads"], cfg["n_kv_heads"], d, \
        cfg["n_heads"] * d, cfg["n_kv_heads"] * d


def head_rmsnorm_fwd(x, g, eps):
    """RMSNorm of every head vector x [T, n, d] over d with gain g [d]."""
    T, n, d = x.shape
    y, r = rmsnorm_fwd(x.reshape(T * n, d), g, eps)
    return y.reshape(T, n, d), r.reshape(T, n)


def head_rmsnorm_bwd(x, g, r, dy):
    T, n, d = x.shape
    dx, dg = rmsnorm_bwd(x.reshape(T * n, d), g, r.reshape(T * n), dy.reshape(T * n, d))
    return dx.reshape(T, n, d), dg


def attention_block_fwd(x, W, cfg):
    """a = RMSNorm(x; g1); qkv = a W_qkv^T; [QK-Norm]; RoPE; attention;
    h1 = x + s o W_o^T (s = branch_scale, 1 unless set)."""
    h, nh, nkv, d, hq, hkv = _dims(cfg)
    B, S, base = cfg["batch"], cfg["seq"], cfg["rope_base"]
    pos = cfg.get("positions")
    bs = cfg.get("branch_scale", 1.0) or 1.0
    T = x.shape[0]
    a, r1 = rmsnorm_fwd(x, W["attn_norm"], cfg["rms_eps"])
    qkv = a @ W["w_qkv"].T
    q = qkv[:, :hq].reshape(T, nh, d)
    k = qkv[:, hq:hq + hkv].reshape(T, nkv, d)
    v = qkv[:, hq + hkv:].reshape(T, nkv, d)
    cache = dict(x=x, a=a, r1=r1, v=v, q_raw=q, k_raw=k)
    if cfg.get("qk_norm"):
        q, cache["rq"] = head_rmsnorm_fwd(q, W["q_norm"], cfg["rms_eps"])
        k, cache["rk"] = head_rmsnorm_fwd(k, W["k_norm"], cfg["rms_eps"])
    qr = rope_fwd(q, B, S, base, pos)
    kr = rope_fwd(k, B, S, base, pos)
    o, lse = attention_fwd(qr, kr, v, B, S)
    o = o.reshape(T, hq)
    h1 = x + bs * (o @ W["w_o"].T)
    cache.update(qr=qr, kr=kr, o=o, lse=lse)
    return h1, cache


def attention_block_bwd(c, W, cfg, dh1):
    """Backward of attention_block_fwd; dh1 flows through the residual."""
    h, nh, nkv, d, hq, hkv = _dims(cfg)
    B, S, base = cfg["batch"], cfg["seq"], cfg["rope_base"]
    pos = cfg.get("positions")
    bs = cfg.get("branch_scale", 1.0) or 1.0
    T = dh1.shape[0]
    g = {}
    db = bs * dh1
    g["w_o"] = db.T @ c["o"]
    do = (db @ W["w_o"]).reshape(T, nh, d)
    dqr, dkr, dv = attention_bwd(c["qr"], c["kr"], c["v"], do, B, S)
    dq = rope_bwd(dqr, B, S, base, pos)
    dk = rope_bwd(dkr, B, S, base, pos)
    if cfg.get("qk_norm"):
        dq, g["q_norm"] = head_rmsnorm_bwd(c["q_raw"], W["q_norm"], c["rq"], dq)
        dk, g["k_norm"] = head_rmsnorm_bwd(c["k_raw"], W["k_norm"], c["rk"], dk)
    dqkv = np.concatenate([dq.reshape(T, hq), dk.reshape(T, hkv), dv.reshape(T, hkv)], axis=1)
    g["w_qkv"] = dqkv.T @ c["a"]
    da = dqkv @ W["w_qkv"]
    dxn, g["attn_norm"] = rmsnorm_bwd(c["x"], W["attn_norm"], c["r1"], da)
    return dh1 + dxn, g


def ffn_fwd(h1, W, cfg):
    """b = RMSNorm(h1; g2); [G|U] = b W_gu^T; out = h1 + s (silu(G) U) W_d^T."""
    f = cfg["ffn"]
    bs = cfg.get("branch_scale", 1.0) or 1.0
    b, r2 = rmsnorm_fwd(h1, W["ffn_norm"], cfg["rms_eps"])
    gu = b @ W["w_gate_up"].T
    G, U = gu[:, :f], gu[:, f:]
    A = swiglu_fwd(G, U)
    out = h1 + bs * (A @ W["w_down"].T)
    return out, dict(h1=h1, b=b, r2=r2, G=G, U=U, A=A)


def ffn_bwd(c, W, cfg, dout):
    bs = cfg.get("branch_scale", 1.0) or 1.0
    g = {}
    dy = bs * dout
    g["w_down"] = dy.T @ c["A"]
    dA = dy @ W["w_down"]
    dG, dU = swiglu_bwd(c["G"], c["U"], dA)
    dgu = np.concatenate([dG, dU], axis=1)
    g["w_gate_up"] = dgu.T @ c["b"]
    db = dgu @ W["w_gate_up"]
    dh1n, g["ffn_norm"] = rmsnorm_bwd(c["h1"], W["ffn_norm"], c["r2"], db)
    return dout + dh1n, g


def layer_fwd(x, W, cfg):
    """Dense decoder layer forward. Returns (out [T, h], cache)."""
    h1, ca = attention_block_fwd(x, W, cfg)
    out, cf = ffn_fwd(h1, W, cfg)
    return out, dict(attn=ca, ffn=cf)


def layer_bwd(cache, W, cfg, dout):
    """Dense decoder layer backward. Returns (dx [T, h], grads by weight name)."""
    dh1, gf = ffn_bwd(cache["ffn"], W, cfg, dout)
    dx, ga = attention_block_bwd(cache["attn"], W, cfg, dh1)
    ga.update(gf)
    return dx, ga


def layer_fwd_rows(x, W, cfg, rows):
    """The layer output at selected token rows only (the same definition).

    Keys and values need every token, so RMSNorm and the k/v projections run
    over all rows; the query projection, attention, output projection and FFN
    run only for `rows`. Used to check very long sequences one row at a time.
    """
    h, nh, nkv, d, hq, hkv = _dims(cfg)
    B, S, base = cfg["batch"], cfg["seq"], cfg["rope_base"]
    rows = np.asarray(rows)
    T = x.shape[0]
    a, _ = rmsnorm_fwd(x, W["attn_norm"], cfg["rms_eps"])
    wq, wk, wv = W["w_qkv"][:hq], W["w_qkv"][hq:hq + hkv], W["w_qkv"][hq + hkv:]
    k = rope_fwd((a @ wk.T).reshape(T, nkv, d), B, S, base)
    v = (a @ wv.T).reshape(T, nkv, d)
    pos = rows % S
    phi = rope_angles(S, d, base)[pos]
    cs, sn = np.cos(phi)[:, None, :], np.sin(phi)[:, None, :]
    q = (a[rows] @ wq.T).reshape(len(rows), nh, d)
    q1, q2 = q[..., : d // 2], q[..., d // 2:]
    q = np.concatenate([q1 * cs - q2 * sn, q2 * cs + q1 * sn], axis=-1)
    grp = nh // nkv
    o = np.zeros((len(rows), nh, d))
    for r, t in enumerate(rows):
        b0 = (t // S) * S
        keys = slice(b0, t + 1)
        for n in range(nh):
            s = (k[keys, n // grp] @ q[r, n]) / np.sqrt(d)
            p = np.exp(s - s.max())
            o[r, n] = (p / p.sum()) @ v[keys, n // grp]
    h1 = x[rows] + o.reshape(len(rows), hq) @ W["w_o"].T
    out, _ = ffn_fwd(h1, W, cfg)
    return out
