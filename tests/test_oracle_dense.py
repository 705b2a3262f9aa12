"""Pins for the dense-layer oracle: finite differences, closed forms, invariants.

Each test fixes the oracle against something other than itself: central
finite differences of a scalar objective (the whole hand-derived backward),
closed forms of RMSNorm / RoPE / attention on special inputs, a RoPE worked
example computed by hand, the causal-mask invariant and brute-force loops.
"""
import numpy as np
import pytest

from oracle import dense
from fdcheck import central_diff, sample_indices, rel_err

MICRO = dict(batch=2, seq=3, hidden=16, n_heads=4, n_kv_heads=2, head_dim=4,
             ffn=24, rope_base=10000.0, rms_eps=1e-5, n_experts=0)


def micro_weights(cfg, rng, std=0.3):
    h, d = cfg["hidden"], cfg["head_dim"]
    hq, hkv, f = cfg["n_heads"] * d, cfg["n_kv_heads"] * d, cfg["ffn"]
    return {
        "attn_norm": 1.0 + 0.1 * rng.standard_normal(h),
        "w_qkv": std * rng.standard_normal((hq + 2 * hkv, h)),
        "w_o": std * rng.standard_normal((h, hq)),
        "ffn_norm": 1.0 + 0.1 * rng.standard_normal(h),
        "w_gate_up": std * rng.standard_normal((2 * f, h)),
        "w_down": std * rng.standard_normal((h, f)),
    }


# --------------------------------------------------------------------------
# whole-layer backward vs central differences
# --------------------------------------------------------------------------

def test_layer_backward_matches_finite_differences():
    rng = np.random.default_rng(7)
    cfg = MICRO
    T = cfg["batch"] * cfg["seq"]
    W = micro_weights(cfg, rng)
    x = rng.standard_normal((T, cfg["hidden"]))
    R = rng.standard_normal((T, cfg["hidden"]))

    def objective():
        out, _ = dense.layer_fwd(x, W, cfg)
        return float(np.sum(out * R))

    out, cache = dense.layer_fwd(x, W, cfg)
    dx, grads = dense.layer_bwd(cache, W, cfg, R)
    srng = np.random.default_rng(0)
    idx = sample_indices(x.size, 96, srng)
    assert rel_err(dx.ravel()[idx], central_diff(objective, x, idx)) <= 1e-6
    for name, g in grads.items():
        idx = sample_indices(W[name].size, 160, srng)
        fd = central_diff(objective, W[name], idx)
        assert rel_err(g.ravel()[idx], fd) <= 1e-6, name


# --------------------------------------------------------------------------
# RMSNorm
# --------------------------------------------------------------------------

def test_rmsnorm_constant_row_closed_form():
    h, c, eps = 8, 0.37, 1e-5
    g = np.linspace(0.5, 1.5, h)
    y, r = dense.rmsnorm_fwd(np.full((1, h), c), g, eps)
    assert np.allclose(y[0], c / np.sqrt(c * c + eps) * g, rtol=0, atol=1e-15)
    assert np.isclose(r[0], 1.0 / np.sqrt(c * c + eps), rtol=1e-15)


def test_rmsnorm_scale_invariance_of_gradient():
    # with g = 1 and eps = 0, y(x) = y(a x), so the gradient is orthogonal to x
    rng = np.random.default_rng(3)
    x = rng.standard_normal((5, 12))
    g = np.ones(12)
    _, r = dense.rmsnorm_fwd(x, g, 0.0)
    dx, _ = dense.rmsnorm_bwd(x, g, r, rng.standard_normal((5, 12)))
    assert np.max(np.abs(np.sum(dx * x, axis=1))) < 1e-13


# --------------------------------------------------------------------------
# RoPE
# --------------------------------------------------------------------------

def test_rope_worked_example():
    # d = 4, base 1e4: angles at position 1 are 1 rad (i = 0) and 1e-2 rad
    # (i = 1). The unit vector e0 rotates into (cos 1, 0, sin 1, 0) and e1
    # into (0, cos .01, 0, sin .01): the pair (i, i + d/2) turns counter-clockwise.
    x = np.zeros((2, 2, 4))
    x[:, 0, 0] = 1.0
    x[:, 1, 1] = 1.0
    y = dense.rope_fwd(x, 1, 2, 10000.0)
    assert np.allclose(y[0], x[0], atol=0)                   # position 0
    assert np.allclose(y[1, 0], [np.cos(1.0), 0, np.sin(1.0), 0], atol=1e-15)
    assert np.allclose(y[1, 1], [0, np.cos(0.01), 0, np.sin(0.01)], atol=1e-15)


def test_rope_preserves_pair_norms_and_inverts():
    rng = np.random.default_rng(4)
    B, S, n, d = 2, 9, 3, 8
    x = rng.standard_normal((B * S, n, d))
    y = dense.rope_fwd(x, B, S, 500000.0)
    pn = lambda a: a[..., : d // 2] ** 2 + a[..., d // 2:] ** 2
    assert np.allclose(pn(x), pn(y), rtol=1e-13)
    # backward is the inverse rotation: R(-phi) R(phi) = I
    assert np.allclose(dense.rope_bwd(y, B, S, 500000.0), x, atol=1e-13)
    # positions restart per batch row
    assert np.allclose(y[:S], dense.rope_fwd(x[:S], 1, S, 500000.0))
    assert np.allclose(y[S:], dense.rope_fwd(x[S:], 1, S, 500000.0))


def test_rope_relative_position_property():
    rng = np.random.default_rng(5)
    d, S = 8, 12
    q = rng.standard_normal(d)
    k = rng.standard_normal(d)
    Q = dense.rope_fwd(np.tile(q, (S, 1))[:, None, :], 1, S, 10000.0)[:, 0]
    K = dense.rope_fwd(np.tile(k, (S, 1))[:, None, :], 1, S, 10000.0)[:, 0]
    # <R(m) q, R(n) k> depends on m - n only
    for delta in range(-3, 4):
        vals = [Q[m] @ K[m - delta] for m in range(max(0, delta), min(S, S + delta))]
        assert np.ptp(vals) < 1e-12


# --------------------------------------------------------------------------
# attention
# --------------------------------------------------------------------------

def test_attention_rows_sum_to_one_and_are_causal():
    rng = np.random.default_rng(6)
    S, d = 11, 8
    P, lse = dense.attention_probs(rng.standard_normal((S, d)),
                                   rng.standard_normal((S, d)), 1 / np.sqrt(d))
    assert np.max(np.abs(P.sum(1) - 1.0)) <= 1e-12
    assert np.all(P[np.triu_indices(S, 1)] == 0.0)


def test_attention_brute_force_loops():
    rng = np.random.default_rng(8)
    B, S, nh, nkv, d = 2, 5, 4, 2, 3
    q = rng.standard_normal((B * S, nh, d))
    k = rng.standard_normal((B * S, nkv, d))
    v = rng.standard_normal((B * S, nkv, d))
    o, lse = dense.attention_fwd(q, k, v, B, S)
    for b in range(B):
        for n in range(nh):
            m = n // (nh // nkv)
            for i in range(S):
                ti = b * S + i
                w = [np.exp(q[ti, n] @ k[b * S + j, m] / np.sqrt(d)) for j in range(i + 1)]
                ref = sum(wj * v[b * S + j, m] for j, wj in enumerate(w)) / sum(w)
                assert np.allclose(o[ti, n], ref, rtol=1e-12, atol=1e-14)
                assert np.isclose(lse[b, n, i], np.log(sum(w)), rtol=1e-13)


def test_attention_equal_keys_gives_prefix_mean():
    rng = np.random.default_rng(9)
    S, d = 7, 4
    q = rng.standard_normal((S, 1, d))
    k = np.tile(rng.standard_normal(d), (S, 1))[:, None, :]
    v = rng.standard_normal((S, 1, d))
    o, _ = dense.attention_fwd(q, k, v, 1, S)
    means = np.cumsum(v[:, 0], axis=0) / np.arange(1, S + 1)[:, None]
    assert np.allclose(o[:, 0], means, atol=1e-14)


def test_attention_single_token_returns_v():
    rng = np.random.default_rng(10)
    q, k, v = (rng.standard_normal((1, 2, 4)) for _ in range(3))
    o, lse = dense.attention_fwd(q, k[:, :1], v[:, :1], 1, 1)
    assert np.array_equal(o[0, 0], v[0, 0]) and np.array_equal(o[0, 1], v[0, 0])


def test_gqa_group_reads_its_own_kv_head():
    rng = np.random.default_rng(11)
    S, nh, nkv, d = 6, 4, 2, 4
    q = rng.standard_normal((S, nh, d))
    k = rng.standard_normal((S, nkv, d))
    v = rng.standard_normal((S, nkv, d))
    o, _ = dense.attention_fwd(q, k, v, 1, S)
    k2, v2 = k.copy(), v.copy()
    k2[:, 1] += 5.0
    v2[:, 1] -= 3.0
    o2, _ = dense.attention_fwd(q, k2, v2, 1, S)
    assert np.array_equal(o[:, :2], o2[:, :2])          # heads 0,1 -> kv head 0
    assert not np.allclose(o[:, 2:], o2[:, 2:])         # heads 2,3 -> kv head 1


def test_layer_causal_invariance():
    rng = np.random.default_rng(12)
    cfg = dict(MICRO, batch=1, seq=6)
    W = micro_weights(cfg, rng)
    x = rng.standard_normal((6, cfg["hidden"]))
    out, _ = dense.layer_fwd(x, W, cfg)
    x2 = x.copy()
    x2[4] += rng.standard_normal(cfg["hidden"])
    out2, _ = dense.layer_fwd(x2, W, cfg)
    assert np.array_equal(out[:4], out2[:4])
    assert not np.allclose(out[4], out2[4])


# --------------------------------------------------------------------------
# SwiGLU
# --------------------------------------------------------------------------

def test_silu_special_values():
    assert dense.silu(np.array(0.0)) == 0.0
    dG, dU = dense.swiglu_bwd(np.array(0.0), np.array(1.0), np.array(1.0))
    assert dG == 0.5 and dU == 0.0
    # large |x|: silu(x) -> x, silu(-x) -> 0
    assert np.isclose(dense.silu(np.array(40.0)), 40.0, rtol=1e-15)
    assert abs(dense.silu(np.array(-40.0))) < 1e-15


def test_swiglu_backward_finite_differences():
    rng = np.random.default_rng(13)
    G, U, dA = rng.standard_normal((3, 20))
    dG, dU = dense.swiglu_bwd(G, U, dA)
    f = lambda: float(np.sum(dense.swiglu_fwd(G, U) * dA))
    idx = np.arange(20)
    assert rel_err(dG, central_diff(f, G, idx)) <= 1e-8
    assert rel_err(dU, central_diff(f, U, idx)) <= 1e-8


def test_layer_rows_equals_full_layer():
    rng = np.random.default_rng(14)
    cfg = dict(MICRO, batch=2, seq=5)
    W = micro_weights(cfg, rng)
    x = rng.standard_normal((10, cfg["hidden"]))
    out, _ = dense.layer_fwd(x, W, cfg)
    rows = [0, 3, 4, 5, 9]
    assert np.allclose(dense.layer_fwd_rows(x, W, cfg, rows), out[rows], rtol=1e-12, atol=1e-13)


def test_attention_threaded_equals_serial():
    # the per-kv-head tasks run the serial arithmetic: identical bits
    rng = np.random.default_rng(12)
    B, S, nh, nkv, d = 2, 9, 6, 3, 4
    q = rng.standard_normal((B * S, nh, d))
    k = rng.standard_normal((B * S, nkv, d))
    v = rng.standard_normal((B * S, nkv, d))
    do = rng.standard_normal((B * S, nh, d))
    o1, l1 = dense.attention_fwd(q, k, v, B, S, workers=1)
    o4, l4 = dense.attention_fwd(q, k, v, B, S, workers=4)
    assert np.array_equal(o1, o4) and np.array_equal(l1, l4)
    for a, b in zip(dense.attention_bwd(q, k, v, do, B, S, workers=1),
                    dense.attention_bwd(q, k, v, do, B, S, workers=4)):
        assert np.array_equal(a, b)
