"""Pins for the AdamW oracle, the clip coefficient and bf16 rounding."""
import numpy as np

from oracle import adamw


def test_constant_gradient_closed_form():
    # m0 = v0 = 0 and a constant g give m_hat = g and v_hat = g^2 at every
    # step, so p_t = p_{t-1} - lr (g / (|g| + eps) + wd p_{t-1}) exactly.
    g = np.array([3e-3, -2e-2, 1e-6, 0.5])
    lr, b1, b2, eps, wd = 1e-3, 0.9, 0.95, 1e-8, 0.1
    p = np.array([0.01, -0.02, 0.3, 0.0])
    m = np.zeros(4)
    v = np.zeros(4)
    ref = p.copy()
    for t in range(1, 6):
        p, m, v = adamw.adamw_step(p, g, m, v, lr, b1, b2, eps, wd, t)
        ref = ref - lr * (g / (np.abs(g) + eps) + wd * ref)
        assert np.allclose(p, ref, rtol=1e-12, atol=1e-15)


def test_single_step_term_by_term():
    # one element, arbitrary state, every term of the update written out
    p, g, m, v = 0.2, -0.04, 0.01, 3e-4
    lr, b1, b2, eps, wd, t, clip = 2e-3, 0.9, 0.95, 1e-8, 0.1, 3, 0.5
    gc = g * clip
    m1 = b1 * m + (1 - b1) * gc
    v1 = b2 * v + (1 - b2) * gc * gc
    upd = (m1 / (1 - b1 ** t)) / (np.sqrt(v1 / (1 - b2 ** t)) + eps) + wd * p
    pn, mn, vn = adamw.adamw_step(np.array([p]), np.array([g]), np.array([m]),
                                  np.array([v]), lr, b1, b2, eps, wd, t, clip)
    assert np.isclose(pn[0], p - lr * upd, rtol=1e-15)
    assert np.isclose(mn[0], m1, rtol=1e-15) and np.isclose(vn[0], v1, rtol=1e-15)


def test_weight_decay_only_when_gradient_is_zero():
    p = np.array([0.5, -1.0])
    pn, _, _ = adamw.adamw_step(p, np.zeros(2), np.zeros(2), np.zeros(2),
                                1e-2, 0.9, 0.95, 1e-8, 0.1, 1)
    assert np.allclose(pn, p * (1 - 1e-3), rtol=1e-15)


def test_clip_coefficient():
    assert adamw.clip_coeff(0.25, 1.0, 1e-6) == 1.0             # norm 0.5 < 1
    assert np.isclose(adamw.clip_coeff(16.0, 1.0, 0.0), 0.25)    # norm 4
    assert adamw.clip_coeff(-1.0, 1.0, 1e-6) == 1.0              # clamped at 0
    assert np.isclose(adamw.grad_norm_sq([np.array([3.0]), np.array([[4.0]])]), 25.0)


def test_bf16_rounding_known_values():
    # bf16 spacing in [1, 2) is 2^-7 = 0.0078125
    cases = {
        1.0: 1.0,
        1.00390625: 1.0,            # exactly half an ulp above 1: tie -> even (1.0)
        1.01171875: 1.015625,       # half-way between 1.0078125 and 1.015625 -> even
        1.0078125: 1.0078125,       # representable
        1.005: 1.0078125,           # above the half-way point
        -3.14159265: -3.140625,
        65504.0: 65536.0,
        1e-40: np.float64(np.float32(1e-40)),  # subnormal range, spacing 2^-133
    }
    for x, want in cases.items():
        x32 = np.float64(np.float32(x))
        got = adamw.bf16_rne(np.array([x32]))[0]
        if x == 1e-40:
            want = np.rint(x32 / 2.0 ** -133) * 2.0 ** -133
        assert got == want, (x, got, want)


def test_bf16_rounding_matches_bit_definition():
    # against the integer definition: add 0x7FFF + lsb, truncate 16 bits
    rng = np.random.default_rng(3)
    x = (rng.standard_normal(20000) * 10.0 ** rng.integers(-20, 20, 20000)).astype(np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    want = r.astype(np.uint32).view(np.float32).astype(np.float64)
    assert np.array_equal(adamw.bf16_rne(x.astype(np.float64)), want)
