"""Central finite differences in fp64, used to pin the oracle's backward."""
import numpy as np


def central_diff(f, theta, idx, rel_step=1e-6):
    """(f(theta + h e_i) - f(theta - h e_i)) / 2h at each flat index i in idx.

    theta is perturbed in place and restored; h = rel_step * max(1, |theta_i|).
    """
    flat = theta.reshape(-1)
    out = np.empty(len(idx))
    for n, i in enumerate(idx):
        old = flat[i]
        h = rel_step * max(1.0, abs(old))
        flat[i] = old + h
        fp = f()
        flat[i] = old - h
        fm = f()
        flat[i] = old
        out[n] = (fp - fm) / (2.0 * h)
    return out


def sample_indices(size, max_n, rng):
    if size <= max_n:
        return np.arange(size)
    return np.sort(rng.choice(size, max_n, replace=False))


def rel_err(a, b):
    a = np.asarray(a, np.float64).ravel()
    b = np.asarray(b, np.float64).ravel()
    return np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300)
