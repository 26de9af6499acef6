"""CPU oracle of the optimiser step (test infrastructure only).

Alg. 1 updates the weights with ADAM after each backward pass.  This is Adam
as its authors define it (Kingma and Ba, ICLR 2015, Algorithm 1), in float64:

    m <- beta1 m + (1 - beta1) g
    v <- beta2 v + (1 - beta2) g^2
    p <- p - lr * (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + eps)

with t the 1-based step count.  No weight decay (the paper names none).
"""
from __future__ import annotations

import numpy as np


def adam(param, grad, m, v, t: int, lr: float, beta1: float = 0.9, beta2: float = 0.999, eps: float = 1e-8):
    """One Adam step; returns (param, m, v) as new float64 arrays."""
    if t < 1:
        raise ValueError("t counts steps from 1")
    g = np.asarray(grad, dtype=np.float64)
    m = beta1 * np.asarray(m, dtype=np.float64) + (1.0 - beta1) * g
    v = beta2 * np.asarray(v, dtype=np.float64) + (1.0 - beta2) * g * g
    m_hat = m / (1.0 - beta1 ** t)
    v_hat = v / (1.0 - beta2 ** t)
    p = np.asarray(param, dtype=np.float64) - lr * m_hat / (np.sqrt(v_hat) + eps)
    return p, m, v
