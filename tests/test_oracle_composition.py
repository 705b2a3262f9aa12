"""Pins for how the oracle composes a layer and a model, not just its pieces.

The per-function pins (finite differences, closed forms, brute force) cannot
see a composition mistake shared by the forward and the backward: a dropped
or misplaced residual, a norm applied to the wrong tensor, a missing final
norm before the LM head. The pre-norm decoder of App. B fixes closed forms
for exactly those:

* residual identity: with both branch output projections zero the layer is
  the identity (out == x bit for bit), and with one zero the other branch
  alone is added;
* pre-norm placement: a branch sees x only through RMSNorm(x), which (eps = 0)
  is invariant to x -> c x, so out(c x) - c x == out(x) - x when the other
  branch is zero; a post-norm or a norm on the wrong tensor breaks this;
* final norm: with eps = 0 the head's loss is invariant to scaling a row of
  x_L (its input gradient row scales by 1/c), and a zero final-norm gain
  makes every logit zero, so the loss is ln V exactly;
* model chain: with every layer the identity, the model's loss is the head's
  loss on the embedding rows, and the input gradient reaches the embedding
  unchanged through every layer.
"""
import numpy as np

from oracle import dense, moe, head
from test_oracle_dense import MICRO, micro_weights
from test_oracle_moe import MOE, moe_weights


def _x(cfg, rng):
    return rng.standard_normal((cfg["batch"] * cfg["seq"], cfg["hidden"]))


def test_dense_layer_with_zero_branch_outputs_is_identity():
    rng = np.random.default_rng(31)
    W = micro_weights(MICRO, rng)
    W["w_o"][:] = 0.0
    W["w_down"][:] = 0.0
    x = _x(MICRO, rng)
    out, _ = dense.layer_fwd(x, W, MICRO)
    assert np.array_equal(out, x)


def test_dense_layer_adds_each_branch_to_the_residual_stream():
    # attention alone: out = x + o W_o^T; FFN alone: out = x + FFN(RMSNorm(x))
    rng = np.random.default_rng(32)
    W = micro_weights(MICRO, rng)
    x = _x(MICRO, rng)
    Wa = dict(W, w_down=np.zeros_like(W["w_down"]))
    out_a, cache = dense.layer_fwd(x, Wa, MICRO)
    assert np.array_equal(out_a, x + cache["attn"]["o"] @ W["w_o"].T)
    Wf = dict(W, w_o=np.zeros_like(W["w_o"]))
    out_f, _ = dense.layer_fwd(x, Wf, MICRO)
    b, _ = dense.rmsnorm_fwd(x, W["ffn_norm"], MICRO["rms_eps"])
    G = b @ W["w_gate_up"][:MICRO["ffn"]].T
    U = b @ W["w_gate_up"][MICRO["ffn"]:].T
    A = G / (1.0 + np.exp(-G)) * U
    assert np.allclose(out_f, x + A @ W["w_down"].T, rtol=1e-13, atol=1e-13)


def test_dense_layer_branches_are_pre_normalised():
    rng = np.random.default_rng(33)
    cfg = dict(MICRO, rms_eps=0.0)
    W = micro_weights(cfg, rng)
    x = _x(cfg, rng)
    for zero in ("w_down", "w_o"):     # attention branch alone, FFN branch alone
        Wz = dict(W, **{zero: np.zeros_like(W[zero])})
        base, _ = dense.layer_fwd(x, Wz, cfg)
        for c in (0.25, 3.0):
            out, _ = dense.layer_fwd(c * x, Wz, cfg)
            assert np.allclose(out - c * x, base - x, rtol=1e-11, atol=1e-12), (zero, c)
        # a row-wise scale too: each token's norm is its own
        s = rng.uniform(0.5, 2.0, (x.shape[0], 1))
        out, _ = dense.layer_fwd(s * x, Wz, cfg)
        assert np.allclose(out - s * x, base - x, rtol=1e-11, atol=1e-12), zero


def test_dense_layer_backward_through_identity_layer():
    # identity layer: d_in == d_out exactly; only the two zero projections
    # get a gradient (their inputs times d_out), the weights behind them none
    rng = np.random.default_rng(34)
    W = micro_weights(MICRO, rng)
    W["w_o"][:] = 0.0
    W["w_down"][:] = 0.0
    x = _x(MICRO, rng)
    dy = rng.standard_normal(x.shape)
    _, cache = dense.layer_fwd(x, W, MICRO)
    dx, g = dense.layer_bwd(cache, W, MICRO, dy)
    assert np.array_equal(dx, dy)
    for n in ("w_qkv", "attn_norm", "w_gate_up", "ffn_norm"):
        assert np.all(g[n] == 0.0), n
    assert np.allclose(g["w_o"], dy.T @ cache["attn"]["o"], rtol=1e-13, atol=1e-13)
    assert np.allclose(g["w_down"], dy.T @ cache["ffn"]["A"], rtol=1e-13, atol=1e-13)


def test_moe_layer_with_zero_expert_outputs_returns_h1():
    rng = np.random.default_rng(35)
    W = moe_weights(MOE, rng)
    W["w_down_e"][:] = 0.0
    x = _x(MOE, rng)
    out, _, cache = moe.layer_fwd(x, W, MOE)
    assert np.array_equal(out, cache["h1"])
    W["w_o"][:] = 0.0
    out, _, _ = moe.layer_fwd(x, W, MOE)
    assert np.array_equal(out, x)


def test_moe_layer_branch_is_pre_normalised():
    rng = np.random.default_rng(36)
    cfg = dict(MOE, rms_eps=0.0)
    W = moe_weights(cfg, rng)
    W["w_o"][:] = 0.0
    x = _x(cfg, rng)
    base, aux0, c0 = moe.layer_fwd(x, W, cfg)
    for c in (0.5, 4.0):
        out, aux, c1 = moe.layer_fwd(c * x, W, cfg)
        assert np.array_equal(c1["moe"]["idx"], c0["moe"]["idx"])
        assert np.allclose(out - c * x, base - x, rtol=1e-11, atol=1e-12)
        assert np.isclose(aux, aux0, rtol=1e-12)


def test_head_loss_invariant_to_row_scale_of_its_input():
    rng = np.random.default_rng(37)
    T, h, V = 7, 16, 32
    xL = rng.standard_normal((T, h))
    g = 1.0 + 0.1 * rng.standard_normal(h)
    w = 0.5 * rng.standard_normal((V, h))
    tg = rng.integers(0, V, T)
    loss, dx, dg, dw = head.head_fwd_bwd(xL, g, w, tg, 0.0)
    s = rng.uniform(0.2, 5.0, (T, 1))
    loss2, dx2, dg2, dw2 = head.head_fwd_bwd(s * xL, g, w, tg, 0.0)
    assert np.isclose(loss2, loss, rtol=1e-13)
    assert np.allclose(dx2 * s, dx, rtol=1e-10, atol=1e-14)
    assert np.allclose(dg2, dg, rtol=1e-10, atol=1e-14)
    assert np.allclose(dw2, dw, rtol=1e-10, atol=1e-14)


def test_head_zero_final_norm_gives_uniform_logits():
    rng = np.random.default_rng(38)
    T, h, V = 5, 16, 1024
    xL = rng.standard_normal((T, h))
    w = rng.standard_normal((V, h))
    loss, dx, dg, dw = head.head_fwd_bwd(xL, np.zeros(h), w, rng.integers(0, V, T), 1e-5)
    assert loss == np.log(V) == 6.931471805599453
    assert np.all(dx == 0.0) and np.all(dw == 0.0)


def test_model_with_identity_layers_is_the_head_on_the_embedding():
    rng = np.random.default_rng(39)
    cfg = dict(MICRO, vocab=32, n_layers=3)
    T, h = cfg["batch"] * cfg["seq"], cfg["hidden"]
    layers = []
    for _ in range(3):
        W = micro_weights(cfg, rng)
        W["w_o"][:] = 0.0
        W["w_down"][:] = 0.0
        layers.append(W)
    for tied in (False, True):
        P = {"embedding": rng.standard_normal((32, h)), "layers": layers,
             "final_norm": 1.0 + 0.1 * rng.standard_normal(h),
             "w_lm": None if tied else rng.standard_normal((32, h))}
        ids, tg = rng.integers(0, 32, T), rng.integers(0, 32, T)
        loss, grads = head.model_fwd_bwd(P, ids, tg, cfg)
        w_lm = P["embedding"] if tied else P["w_lm"]
        ref_loss, ref_dx, ref_dg, ref_dw = head.head_fwd_bwd(
            P["embedding"][ids], P["final_norm"], w_lm, tg, cfg["rms_eps"])
        assert loss == ref_loss
        assert np.array_equal(grads["final_norm"], ref_dg)
        dE = np.zeros_like(P["embedding"])
        np.add.at(dE, ids, ref_dx)
        want = dE + ref_dw if tied else dE
        assert np.allclose(grads["embedding"], want, rtol=1e-13, atol=1e-15)
        if not tied:
            assert np.array_equal(grads["w_lm"], ref_dw)


def test_dense_layer_is_ffn_layer_after_attention_layer():
    # the FFN branch reads the attention branch's output h1: the full layer is
    # the FFN-only layer (w_o = 0) applied to the attention-only layer's
    # output (w_down = 0); an FFN norm on x instead of h1 breaks this
    rng = np.random.default_rng(40)
    W = micro_weights(MICRO, rng)
    x = _x(MICRO, rng)
    out, _ = dense.layer_fwd(x, W, MICRO)
    h1, _ = dense.layer_fwd(x, dict(W, w_down=np.zeros_like(W["w_down"])), MICRO)
    want, _ = dense.layer_fwd(h1, dict(W, w_o=np.zeros_like(W["w_o"])), MICRO)
    assert np.allclose(out, want, rtol=1e-13, atol=1e-13)


def test_moe_layer_is_moe_branch_after_attention_layer():
    rng = np.random.default_rng(41)
    W = moe_weights(MOE, rng)
    x = _x(MOE, rng)
    out, aux, _ = moe.layer_fwd(x, W, MOE)
    h1, _, _ = moe.layer_fwd(x, dict(W, w_down_e=np.zeros_like(W["w_down_e"])), MOE)
    want, aux2, _ = moe.layer_fwd(h1, dict(W, w_o=np.zeros_like(W["w_o"])), MOE)
    assert np.allclose(out, want, rtol=1e-13, atol=1e-13)
    assert np.isclose(aux, aux2, rtol=1e-13)
