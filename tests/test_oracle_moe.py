"""Pins for the MoE oracle: routing brute force, aux loss, grouped vs per token, FD."""
import numpy as np

from oracle import moe
from fdcheck import central_diff, sample_indices, rel_err
from test_oracle_dense import MICRO, micro_weights

MOE = dict(MICRO, ffn=0, n_experts=8, top_k=2, expert_ffn=12, aux_coef=1e-2)


def moe_weights(cfg, rng, std=0.3):
    W = micro_weights(dict(cfg, ffn=4), rng, std)
    del W["w_gate_up"], W["w_down"]
    E, h, fe = cfg["n_experts"], cfg["hidden"], cfg["expert_ffn"]
    W["w_router"] = std * rng.standard_normal((E, h))
    W["w_gate_up_e"] = std * rng.standard_normal((E, 2 * fe, h))
    W["w_down_e"] = std * rng.standard_normal((E, h, fe))
    return W


def test_topk_brute_force_with_ties():
    l = np.array([[0.5, 2.0, 2.0, -1.0, 2.0],
                  [1.0, 1.0, 1.0, 1.0, 1.0],
                  [-3.0, 0.0, 4.0, 0.0, 1.0]], np.float32)
    assert np.array_equal(moe.topk(l, 3), [[1, 2, 4], [0, 1, 2], [2, 4, 1]])
    rng = np.random.default_rng(1)
    l = rng.standard_normal((50, 16)).astype(np.float32)
    l[:, 5] = l[:, 9]                      # force exact ties
    idx = moe.topk(l, 4)
    for t in range(50):
        want = sorted(range(16), key=lambda e: (-float(l[t, e]), e))[:4]
        assert list(idx[t]) == want


def test_route_counts_offsets_perm():
    rng = np.random.default_rng(2)
    T, E, k = 37, 8, 3
    l = rng.standard_normal((T, E)).astype(np.float32)
    idx, gates, p, counts, offsets, perm = moe.route(l, k)
    assert counts.sum() == T * k and offsets[-1] == T * k
    assert np.all(np.diff(offsets) == counts)
    assert np.array_equal(np.sort(perm), np.arange(T * k))
    flat = idx.reshape(-1)
    for e in range(E):
        seg = perm[offsets[e]:offsets[e + 1]]
        assert np.all(flat[seg] == e) and np.all(np.diff(seg) > 0)
    assert np.allclose(p.sum(1), 1.0, atol=1e-15)
    assert np.allclose(gates, np.take_along_axis(p, idx, 1))


def test_aux_loss_balanced_routing_equals_alpha():
    T, E, k, alpha = 16, 8, 2, 1e-2
    p = np.full((T, E), 1.0 / E)
    counts = np.full(E, T * k // E)
    assert np.isclose(moe.aux_loss(p, counts, k, alpha), alpha, rtol=1e-15)


def test_grouped_equals_per_token():
    rng = np.random.default_rng(3)
    cfg = MOE
    W = moe_weights(cfg, rng)
    b = rng.standard_normal((10, cfg["hidden"]))
    y, aux, _ = moe.moe_fwd(b, W, cfg)
    assert np.allclose(y, moe.moe_fwd_per_token(b, W, cfg), rtol=1e-12, atol=1e-14)


def test_moe_layer_backward_finite_differences():
    rng = np.random.default_rng(4)
    cfg = MOE
    T = cfg["batch"] * cfg["seq"]
    W = moe_weights(cfg, rng)
    x = rng.standard_normal((T, cfg["hidden"]))
    R = rng.standard_normal((T, cfg["hidden"]))
    out, aux, cache = moe.layer_fwd(x, W, cfg)
    idx0 = cache["moe"]["idx"].copy()

    def objective():
        o, a, c = moe.layer_fwd(x, W, cfg)
        assert np.array_equal(c["moe"]["idx"], idx0)   # no routing flips under FD
        return float(np.sum(o * R) + a)

    dx, grads = moe.layer_bwd(cache, W, cfg, R)
    srng = np.random.default_rng(0)
    idx = sample_indices(x.size, 64, srng)
    assert rel_err(dx.ravel()[idx], central_diff(objective, x, idx)) <= 1e-6
    for name in ("w_router", "w_gate_up_e", "w_down_e", "ffn_norm", "w_qkv"):
        idx = sample_indices(W[name].size, 96, srng)
        fd = central_diff(objective, W[name], idx)
        assert rel_err(grads[name].ravel()[idx], fd) <= 1e-6, name


def test_aux_loss_gradient_reaches_router():
    # with dy = 0 the only gradient is the aux loss's, through softmax
    rng = np.random.default_rng(5)
    cfg = dict(MOE, aux_coef=0.7)
    W = moe_weights(cfg, rng)
    b = rng.standard_normal((9, cfg["hidden"]))
    _, aux, c = moe.moe_fwd(b, W, cfg)
    db, g = moe.moe_bwd(c, W, cfg, np.zeros_like(b))
    f = lambda: moe.moe_fwd(b, W, cfg)[1]
    idx = np.arange(W["w_router"].size)
    assert rel_err(g["w_router"].ravel(), central_diff(f, W["w_router"], idx)) <= 1e-6
    assert np.all(g["w_down_e"] == 0)


def test_moe_layer_rows_equals_full_layer():
    rng = np.random.default_rng(6)
    cfg = dict(MOE, batch=2, seq=5)
    W = moe_weights(cfg, rng)
    x = rng.standard_normal((10, cfg["hidden"]))
    out, _, cache = moe.layer_fwd(x, W, cfg)
    rows = [0, 4, 5, 9]
    assert np.allclose(moe.layer_fwd_rows(x, W, cfg, rows), out[rows], rtol=1e-12, atol=1e-13)
    o2, l2 = moe.layer_fwd_rows(x, W, cfg, rows, with_logits=True)
    assert np.allclose(l2, cache["moe"]["l"][rows], rtol=1e-12, atol=1e-13)


def test_topk_margin_brute_force():
    rng = np.random.default_rng(7)
    l = rng.standard_normal((40, 12)).astype(np.float32)
    l[3, 4] = l[3, 9]                                   # a tie is a zero margin
    for k in (1, 3, 11):
        m = moe.topk_margin(l, k)
        idx = moe.topk(l, k)
        for t in range(40):
            inside = float(min(l[t, e] for e in idx[t]))
            outside = float(max(l[t, e] for e in range(12) if e not in idx[t]))
            assert m[t] == inside - outside and m[t] >= 0
    assert np.all(np.isinf(moe.topk_margin(l, 12)))
    # a perturbation below half the margin leaves the top-k set unchanged
    k = 3
    m = moe.topk_margin(l, k)
    d = (0.49 * m[:, None] * rng.uniform(-1, 1, l.shape)).astype(np.float32)
    keep = m > 1e-3
    assert np.array_equal(np.sort(moe.topk(l + d, k)[keep], 1), np.sort(moe.topk(l, k)[keep], 1))


def test_forced_routing_reproduces_free_routing_and_stays_valid():
    rng = np.random.default_rng(9)
    T, E, k = 41, 16, 4
    l = rng.standard_normal((T, E))
    free = moe.route(l, k)
    forced = moe.route(l, k, moe.topk(np.asarray(l, np.float32), k))
    for a, b in zip(free, forced):
        assert np.array_equal(a, b)
    # another valid choice: swap the k-th expert of token 3 for its (k+1)-th
    order = np.argsort(-l[3], kind="stable")
    alt = free[0].copy()
    alt[3, k - 1] = order[k]
    idx, gates, p, counts, offsets, perm = moe.route(l, k, alt)
    assert counts[order[k]] == free[3][order[k]] + 1
    assert counts[order[k - 1]] == free[3][order[k - 1]] - 1
    assert np.array_equal(gates, np.take_along_axis(p, alt, 1))
    flat = alt.reshape(-1)
    for e in range(E):
        seg = perm[offsets[e]:offsets[e + 1]]
        assert np.all(flat[seg] == e) and np.all(np.diff(seg) > 0)


def test_topk_order_of_signed_zero_and_nan():
    # -0 and +0 tie (lower id first); NaN ranks below every number, -inf too
    l = np.array([[np.nan, -np.inf, -0.0, 0.0, -1.0],
                  [0.0, -0.0, np.nan, np.nan, -np.inf]], np.float32)
    assert np.array_equal(moe.topk(l, 5), [[2, 3, 4, 1, 0], [0, 1, 4, 2, 3]])
