"""Pins for the oracle's model variants (App. B, App. A step 23): per-head
QK-Norm, document-aware RoPE positions, the muP scalars (embedding scale,
residual-branch scale, logit scale), the shared expert and dense first
layers of the sparse model.

Each variant's backward is held to central finite differences, and its
forward to a closed form that a plausible mistake breaks: QK-Norm makes a
head invariant to the scale of its projection rows and gives every
normalised head vector squared norm d; RoPE attention depends on position
differences only, so shifting a row's positions changes nothing; a branch
scale s makes (out - x) / s independent of s; the shared expert with the
routed experts silenced is the dense SwiGLU FFN; the embedding and logit
scales are the same as scaling the embedding or LM-head matrix.
"""
import numpy as np

from oracle import dense, moe, head
from fdcheck import central_diff, sample_indices, rel_err
from test_oracle_dense import MICRO, micro_weights
from test_oracle_moe import MOE, moe_weights


def _x(cfg, rng):
    return rng.standard_normal((cfg["batch"] * cfg["seq"], cfg["hidden"]))


def _qk(cfg, W, rng):
    d = cfg["head_dim"]
    W["q_norm"] = 1.0 + 0.2 * rng.standard_normal(d)
    W["k_norm"] = 1.0 + 0.2 * rng.standard_normal(d)
    return W


def _fd_layer(mod, cfg, W, x, R, names, n=96):
    def objective():
        if mod is moe:
            out, aux, _ = moe.layer_fwd(x, W, cfg)
            return float(np.sum(out * R)) + aux
        out, _ = dense.layer_fwd(x, W, cfg)
        return float(np.sum(out * R))
    if mod is moe:
        _, _, cache = moe.layer_fwd(x, W, cfg)
    else:
        _, cache = dense.layer_fwd(x, W, cfg)
    dx, g = mod.layer_bwd(cache, W, cfg, R)
    srng = np.random.default_rng(0)
    idx = sample_indices(x.size, n, srng)
    assert rel_err(dx.ravel()[idx], central_diff(objective, x, idx)) <= 1e-6
    for name in names:
        idx = sample_indices(W[name].size, n, srng)
        assert rel_err(g[name].ravel()[idx], central_diff(objective, W[name], idx)) <= 1e-6, name


def test_dense_variants_backward_finite_differences():
    rng = np.random.default_rng(51)
    T = MICRO["batch"] * MICRO["seq"]
    cfg = dict(MICRO, qk_norm=1, branch_scale=0.7,
               positions=np.array([4, 0, 1, 0, 1, 2]))
    assert len(cfg["positions"]) == T
    W = _qk(cfg, micro_weights(cfg, rng), rng)
    _fd_layer(dense, cfg, W, _x(cfg, rng), rng.standard_normal((T, cfg["hidden"])),
              ("q_norm", "k_norm", "w_qkv", "w_o", "attn_norm", "w_gate_up", "w_down",
               "ffn_norm"))


def test_moe_shared_expert_backward_finite_differences():
    rng = np.random.default_rng(52)
    cfg = dict(MOE, shared_ffn=8, branch_scale=0.6, aux_coef=0.3)
    W = moe_weights(cfg, rng)
    W["w_gate_up_s"] = 0.3 * rng.standard_normal((16, cfg["hidden"]))
    W["w_down_s"] = 0.3 * rng.standard_normal((cfg["hidden"], 8))
    T = cfg["batch"] * cfg["seq"]
    _fd_layer(moe, cfg, W, _x(cfg, rng), rng.standard_normal((T, cfg["hidden"])),
              ("w_gate_up_s", "w_down_s", "w_router", "w_gate_up_e", "w_down_e", "ffn_norm",
               "w_o"))


def test_qk_norm_head_scale_invariance_and_unit_rms():
    rng = np.random.default_rng(53)
    cfg = dict(MICRO, qk_norm=1, rms_eps=0.0)
    W = micro_weights(cfg, rng)
    d, hq = cfg["head_dim"], cfg["n_heads"] * cfg["head_dim"]
    W["q_norm"] = np.ones(d)
    W["k_norm"] = np.ones(d)
    x = _x(cfg, rng)
    out, cache = dense.layer_fwd(x, W, cfg)
    # RoPE keeps the norm: every normalised head vector has |q|^2 = |k|^2 = d
    assert np.allclose(np.sum(cache["attn"]["qr"] ** 2, -1), d, rtol=1e-12)
    assert np.allclose(np.sum(cache["attn"]["kr"] ** 2, -1), d, rtol=1e-12)
    # a head's projection rows scaled by c > 0: the normalised head is the same
    W2 = {k: v.copy() for k, v in W.items()}
    W2["w_qkv"][d:2 * d] *= 3.5               # query head 1
    W2["w_qkv"][hq:hq + d] *= 0.25            # key head 0
    out2, _ = dense.layer_fwd(x, W2, cfg)
    assert np.allclose(out2, out, rtol=1e-11, atol=1e-12)
    # the norm comes before RoPE: rotating the final head vectors back by
    # their angles and dividing by the gain leaves unit-RMS vectors (a norm
    # applied after the rotation would not, for a non-uniform gain)
    W3 = _qk(cfg, {k: v.copy() for k, v in W.items()}, rng)
    _, c3 = dense.layer_fwd(x, W3, cfg)
    B, S, base = cfg["batch"], cfg["seq"], cfg["rope_base"]
    qb = dense.rope_bwd(c3["attn"]["qr"], B, S, base) / W3["q_norm"]
    kb = dense.rope_bwd(c3["attn"]["kr"], B, S, base) / W3["k_norm"]
    assert np.allclose(np.mean(qb ** 2, -1), 1.0, rtol=1e-12)
    assert np.allclose(np.mean(kb ** 2, -1), 1.0, rtol=1e-12)
    # without QK-Norm the same change moves the output
    out3, _ = dense.layer_fwd(x, W2, dict(cfg, qk_norm=0))
    out4, _ = dense.layer_fwd(x, W, dict(cfg, qk_norm=0))
    assert not np.allclose(out3, out4, rtol=1e-6)


def test_rope_positions_default_and_shift_invariance():
    rng = np.random.default_rng(54)
    cfg = dict(MICRO, batch=1, seq=6)
    W = micro_weights(cfg, rng)
    x = _x(cfg, rng)
    base_out, _ = dense.layer_fwd(x, W, cfg)
    out, _ = dense.layer_fwd(x, W, dict(cfg, positions=np.arange(6)))
    assert np.array_equal(out, base_out)
    # attention scores depend on position differences only
    shifted, _ = dense.layer_fwd(x, W, dict(cfg, positions=np.arange(6) + 37))
    assert np.allclose(shifted, base_out, rtol=1e-11, atol=1e-12)
    # a document that restarts at position 0 inside the row changes its rows
    docs = np.array([0, 1, 2, 0, 1, 2])
    packed, _ = dense.layer_fwd(x, W, dict(cfg, positions=docs))
    assert np.array_equal(packed[:3], base_out[:3])       # first document: same positions
    assert not np.allclose(packed[3:], base_out[3:], rtol=1e-6)


def test_branch_scale_is_linear_in_each_branch():
    rng = np.random.default_rng(55)
    W = micro_weights(MICRO, rng)
    x = _x(MICRO, rng)
    for zero in ("w_down", "w_o"):
        Wz = dict(W, **{zero: np.zeros_like(W[zero])})
        plain, _ = dense.layer_fwd(x, Wz, MICRO)
        for s in (0.25, 1.4 / np.sqrt(24)):
            out, _ = dense.layer_fwd(x, Wz, dict(MICRO, branch_scale=s))
            assert np.allclose((out - x) / s, plain - x, rtol=1e-11, atol=1e-12), (zero, s)
    one, _ = dense.layer_fwd(x, W, dict(MICRO, branch_scale=1.0))
    plain, _ = dense.layer_fwd(x, W, MICRO)
    assert np.array_equal(one, plain)


def test_shared_expert_alone_is_the_dense_ffn():
    rng = np.random.default_rng(56)
    cfg = dict(MOE, shared_ffn=8, branch_scale=0.5)
    W = moe_weights(cfg, rng)
    W["w_down_e"][:] = 0.0
    W["w_gate_up_s"] = 0.3 * rng.standard_normal((16, cfg["hidden"]))
    W["w_down_s"] = 0.3 * rng.standard_normal((cfg["hidden"], 8))
    x = _x(cfg, rng)
    out, _, _ = moe.layer_fwd(x, W, cfg)
    Wd = dict(W, w_gate_up=W["w_gate_up_s"], w_down=W["w_down_s"])
    want, _ = dense.layer_fwd(x, Wd, dict(cfg, n_experts=0, ffn=8))
    assert np.allclose(out, want, rtol=1e-13, atol=1e-13)


def test_embedding_and_logit_scales_equal_scaled_matrices():
    rng = np.random.default_rng(57)
    T, h, V = 7, 16, 32
    xL = rng.standard_normal((T, h))
    g = 1.0 + 0.1 * rng.standard_normal(h)
    w = rng.standard_normal((V, h))
    tg = rng.integers(0, V, T)
    c = 256.0 / 1024.0
    a = head.head_fwd_bwd(xL, g, w, tg, 1e-5, logit_scale=c)
    b = head.head_fwd_bwd(xL, g, c * w, tg, 1e-5)
    assert np.isclose(a[0], b[0], rtol=1e-13)
    assert np.allclose(a[1], b[1], rtol=1e-10, atol=1e-15)
    assert np.allclose(a[3], c * b[3], rtol=1e-10, atol=1e-15)
    ids = rng.integers(0, V, T)
    assert np.array_equal(head.embed_fwd(ids, w, 12.0), head.embed_fwd(ids, 12.0 * w))
    assert np.allclose(head.embed_bwd(ids, xL, V, 12.0), 12.0 * head.embed_bwd(ids, xL, V))


def test_mup_moe_model_with_dense_first_layer_finite_differences():
    rng = np.random.default_rng(58)
    cfg = dict(MOE, vocab=32, n_layers=2, dense_first_layers=1, ffn=20, shared_ffn=8,
               embed_scale=12.0, logit_scale=0.25, branch_scale=1.4 / np.sqrt(2), aux_coef=0.1)
    h = cfg["hidden"]
    dense_w = micro_weights(dict(cfg, n_experts=0), rng)
    moe_w = moe_weights(cfg, rng)
    moe_w["w_gate_up_s"] = 0.3 * rng.standard_normal((16, h))
    moe_w["w_down_s"] = 0.3 * rng.standard_normal((h, 8))
    P = {"embedding": 0.1 * rng.standard_normal((32, h)), "layers": [dense_w, moe_w],
         "final_norm": 1.0 + 0.1 * rng.standard_normal(h), "w_lm": None}
    T = cfg["batch"] * cfg["seq"]
    ids, tg = rng.integers(0, 32, T), rng.integers(0, 32, T)
    assert head.layer_cfg(cfg, 0)["n_experts"] == 0 and head.layer_cfg(cfg, 1)["n_experts"] == 8
    loss, grads = head.model_fwd_bwd(P, ids, tg, cfg)
    f = lambda: head.model_fwd_bwd(P, ids, tg, cfg)[0]
    srng = np.random.default_rng(2)
    for name, theta, gr in [("embedding", P["embedding"], grads["embedding"]),
                            ("0.w_gate_up", dense_w["w_gate_up"], grads["layers"][0]["w_gate_up"]),
                            ("1.w_down_s", moe_w["w_down_s"], grads["layers"][1]["w_down_s"]),
                            ("1.w_router", moe_w["w_router"], grads["layers"][1]["w_router"])]:
        idx = sample_indices(theta.size, 48, srng)
        assert rel_err(gr.ravel()[idx], central_diff(f, theta, idx)) <= 1e-6, name
