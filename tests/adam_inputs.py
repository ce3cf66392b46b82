"""Gradient rows for the Adam parity cases where the placement of eps matters (Sec. 5.7; Kingma & Ba,
Algorithm 1): N(0, 0.01) values with, in half the elements, magnitudes 0, 1e-10 .. 1e-5 and
eps / sqrt(1 - b2^t) for t = 1, 2, 3 (eps = 1e-8, b2 = 0.999), random signs; every 7th row entirely
in that regime and every 11th row zero.  Seeded numpy draws; nothing here computes the update."""
import numpy as np

SPECIAL = np.array([0.0, 1e-10, 1e-9, 1e-8, 3e-8, 1e-7, 3.16e-7, 2.24e-7, 1.83e-7, 1e-6, 1e-5])


def eps_regime_grads(rng, n, D):
    g = rng.normal(0.0, 0.01, (n, D)).astype(np.float32)
    vals = (SPECIAL[rng.integers(0, SPECIAL.size, (n, D))] * rng.choice([-1.0, 1.0], (n, D))).astype(np.float32)
    mask = rng.random((n, D)) < 0.5
    g[mask] = vals[mask]
    g[::7] = vals[::7]
    g[::11] = 0.0
    return g
