"""Global gradient-norm clipping, Adam and RMSprop, over the flat parameter buffer.

Test infrastructure: only the tests, the smoke check and the benchmark's CPU baseline use
this package.

Algorithm 1 clips the maximum gradient norm of all parameters (policy and value share the
trunk) before the optimiser step; Appendix B sets the threshold (PPO 0.5, IMPALA 40) and
Adam's epsilon (1e-5). beta1 = 0.9, beta2 = 0.999 and bias correction are the standard Adam
(Kingma and Ba, 2015) values, as used by optax. Appendix B's IMPALA table gives RMSprop with
epsilon 0.01 and decay 0.99; where epsilon sits is not stated, and it is read as optax's
RMSprop does it: inside the square root, with the second-moment estimate starting at zero
(the paper's learner is written in JAX).
"""
from __future__ import annotations

import numpy as np


def global_norm(g):
    return float(np.sqrt(np.sum(np.asarray(g, np.float64) ** 2)))


def clip_by_global_norm(g, max_norm, dtype=np.float64):
    """g * (max_norm / ||g||) when ||g|| > max_norm, else g unchanged; max_norm <= 0 disables.
    Returns (clipped g, pre-clip norm)."""
    g = np.asarray(g, dtype)
    n = np.sqrt(np.sum(g * g))
    if max_norm > 0 and n > max_norm:
        g = g * (max_norm / n)
    return g, n


def adam(p, g, m, v, step, lr, beta1=0.9, beta2=0.999, eps=1e-5, dtype=np.float64):
    """One Adam update at 1-based ``step``; returns new (p, m, v).

    m <- b1 m + (1-b1) g;  v <- b2 v + (1-b2) g^2
    p <- p - lr * (m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps)
    """
    p, g, m, v = (np.asarray(a, dtype) for a in (p, g, m, v))
    m = beta1 * m + (1 - beta1) * g
    v = beta2 * v + (1 - beta2) * g * g
    mhat = m / (1 - beta1 ** step)
    vhat = v / (1 - beta2 ** step)
    return p - lr * mhat / (np.sqrt(vhat) + eps), m, v


def rmsprop(p, g, nu, lr, decay=0.99, eps=0.01, dtype=np.float64):
    """One RMSprop update; returns new (p, nu).

    nu <- decay nu + (1 - decay) g^2
    p  <- p - lr * g / sqrt(nu + eps)
    """
    p, g, nu = (np.asarray(a, dtype) for a in (p, g, nu))
    nu = decay * nu + (1 - decay) * g * g
    return p - lr * g / np.sqrt(nu + eps), nu
