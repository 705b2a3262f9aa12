"""Pins for the embedding / LM head / cross-entropy oracle and the model step."""
import numpy as np

from oracle import head
from fdcheck import central_diff, sample_indices, rel_err
from test_oracle_dense import MICRO, micro_weights


def test_uniform_logits_loss_is_log_vocab():
    for V, exact in ((1024, 6.931471805599453), (32000, 10.373491181781864)):
        z = np.full((3, V), 0.25)
        loss, dz = head.cross_entropy(z, np.array([0, 5, V - 1]))
        assert abs(loss - exact) < 1e-12
        assert np.max(np.abs(dz.sum(axis=1))) < 1e-15


def test_cross_entropy_brute_force():
    rng = np.random.default_rng(1)
    z = rng.standard_normal((4, 6)) * 3
    y = np.array([1, 0, 5, 2])
    loss, dz = head.cross_entropy(z, y)
    ref = np.mean([-np.log(np.exp(z[t, y[t]]) / np.exp(z[t]).sum()) for t in range(4)])
    assert abs(loss - ref) < 1e-14
    f = lambda: head.cross_entropy(z, y)[0]
    assert rel_err(dz, central_diff(f, z, np.arange(z.size))) <= 1e-7


def test_embedding_backward_scatter_brute_force():
    rng = np.random.default_rng(2)
    ids = np.array([3, 1, 3, 0, 3])
    dx = rng.standard_normal((5, 4))
    dE = head.embed_bwd(ids, dx, 6)
    for v in range(6):
        assert np.allclose(dE[v], dx[ids == v].sum(axis=0), atol=1e-15)
    assert np.array_equal(head.embed_fwd(ids, np.arange(24.0).reshape(6, 4))[1],
                          [4.0, 5.0, 6.0, 7.0])


def test_loss_at_init_is_near_log_vocab():
    # weights N(0, 0.02): logits are tiny, so the mean CE is close to ln V
    rng = np.random.default_rng(4)
    T, h, V = 64, 256, 1024
    x = rng.standard_normal((T, h))
    w = 0.02 * rng.standard_normal((V, h))
    loss, *_ = head.head_fwd_bwd(x, np.ones(h), w, rng.integers(0, V, T), 1e-5)
    assert abs(loss - np.log(V)) < 0.05


def _micro_model(tied, rng):
    cfg = dict(MICRO, vocab=32, n_layers=2)
    P = {"embedding": 0.5 * rng.standard_normal((32, cfg["hidden"])),
         "layers": [micro_weights(cfg, rng) for _ in range(2)],
         "final_norm": 1.0 + 0.1 * rng.standard_normal(cfg["hidden"]),
         "w_lm": None if tied else 0.5 * rng.standard_normal((32, cfg["hidden"]))}
    T = cfg["batch"] * cfg["seq"]
    return cfg, P, rng.integers(0, 32, T), rng.integers(0, 32, T)


def _check_model_fd(tied):
    rng = np.random.default_rng(20 + tied)
    cfg, P, ids, tg = _micro_model(tied, rng)
    loss, grads = head.model_fwd_bwd(P, ids, tg, cfg)
    f = lambda: head.model_fwd_bwd(P, ids, tg, cfg)[0]
    srng = np.random.default_rng(1)
    tensors = [("embedding", P["embedding"], grads["embedding"]),
               ("final_norm", P["final_norm"], grads["final_norm"])]
    if not tied:
        tensors.append(("w_lm", P["w_lm"], grads["w_lm"]))
    for li in range(2):
        for name in ("w_qkv", "w_down", "attn_norm"):
            tensors.append((f"{li}.{name}", P["layers"][li][name],
                            grads["layers"][li][name]))
    for name, theta, g in tensors:
        idx = sample_indices(theta.size, 48, srng)
        assert rel_err(g.ravel()[idx], central_diff(f, theta, idx)) <= 1e-6, name


def test_model_backward_finite_differences_untied():
    _check_model_fd(False)


def test_model_backward_finite_differences_tied():
    _check_model_fd(True)
