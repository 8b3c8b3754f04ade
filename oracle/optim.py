"""Adam, the optimiser of the paper's training listings (CPU oracle).

Part of the CPU oracle (test infrastructure).

The paper's step (section 2.2, eq. (3)) is plain SGD, which the training step
uses by default; its DGL listings (section 5) construct torch.optim.Adam with
elided arguments.  Reading: Adam as defined by Kingma and Ba ("Adam: A Method
for Stochastic Optimization", ICLR 2015, Algorithm 1) with the common defaults
beta1 = 0.9, beta2 = 0.999, eps = 1e-8, no weight decay.  Step t (1, 2, ...):

    m = beta1 m + (1 - beta1) g
    v = beta2 v + (1 - beta2) g^2
    w = w - lr * (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + eps)
"""
from __future__ import annotations

import numpy as np

BETA1, BETA2, EPS = 0.9, 0.999, 1e-8


def adam(w, g, m, v, t: int, lr: float, beta1: float = BETA1, beta2: float = BETA2,
         eps: float = EPS):
    """One Adam step on float64 arrays; returns (w, m, v) (new arrays)."""
    assert t >= 1
    w = np.asarray(w, dtype=np.float64)
    g = np.asarray(g, dtype=np.float64)
    m = beta1 * np.asarray(m, dtype=np.float64) + (1.0 - beta1) * g
    v = beta2 * np.asarray(v, dtype=np.float64) + (1.0 - beta2) * g * g
    m_hat = m / (1.0 - beta1 ** t)
    v_hat = v / (1.0 - beta2 ** t)
    return w - lr * m_hat / (np.sqrt(v_hat) + eps), m, v
