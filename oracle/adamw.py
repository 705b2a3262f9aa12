"""Oracle: fused clip + AdamW + bf16 write-back, gradient norm, clip coefficient.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The update is the one the paper's fused optimizer kernel performs per element
(App. F, "Vertical integration", fused clip / Adam / cast): scale the gradient
by the clip coefficient, update both moments, divide by the bias corrections,
add eps outside the square root, add decoupled weight decay on the pre-update
master, step by lr, then write the new master back as bf16. The per-step
scalars (lr, clip coefficient, both bias corrections) are read from device
buffers refreshed once per step (App. F, "Deep customization"); the clip
coefficient is min(1, max_norm / (||g|| + eps)) with the norm clamped at 0
(same passage).

Arithmetic: fp64 on the exact values of the fp32 inputs.
"""
from __future__ import annotations

import numpy as np


def bias_corrections(beta1, beta2, step):
    """bc1 = 1 - beta1^t, bc2 = 1 - beta2^t for step t >= 1."""
    return 1.0 - beta1 ** step, 1.0 - beta2 ** step


def adamw_step(p, g, m, v, lr, beta1, beta2, eps, wd, step, clip=1.0):
    """One AdamW step. Returns (p_new, m_new, v_new), all fp64."""
    p = np.asarray(p, np.float64)
    g = np.asarray(g, np.float64) * clip
    m = beta1 * np.asarray(m, np.float64) + (1.0 - beta1) * g
    v = beta2 * np.asarray(v, np.float64) + (1.0 - beta2) * g * g
    bc1, bc2 = bias_corrections(beta1, beta2, step)
    update = (m / bc1) / (np.sqrt(v / bc2) + eps) + wd * p
    return p - lr * update, m, v


def grad_norm_sq(grads):
    """Sum of squares over every gradient tensor."""
    return float(sum(np.sum(np.asarray(g, np.float64) ** 2) for g in grads))


def clip_coeff(norm_sq, max_norm, eps):
    """min(1, max_norm / (sqrt(max(norm_sq, 0)) + eps))."""
    return min(1.0, max_norm / (np.sqrt(max(norm_sq, 0.0)) + eps))


def bf16_rne(x):
    """Round fp32-representable values to bfloat16, nearest, ties to even.

    Written from the format: bf16 keeps 8 significant bits and fp32's
    exponent range, so a normal value m 2^e (0.5 <= |m| < 1) is quantised to a
    multiple of 2^(e-8); below 2^-126 the quantum is the subnormal one,
    2^-133. np.rint rounds halves to even.
    """
    x = np.asarray(x, np.float64)
    _, e = np.frexp(x)
    q = np.ldexp(1.0, np.maximum(e, -125) - 8)
    return np.rint(x / q) * q
