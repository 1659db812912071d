"""Per-tenant optimizer step (AdamW) in fp64 -- oracle (test infrastructure only).

After its backward, each tenant applies its own optimizer step to its own
parameters and advances only its own version (Sec. 5.2, training-side group
execution; App. A.3, actor consumption).  The paper does not name the
optimizer; the reading used is AdamW (decoupled weight decay, bias-corrected
first and second moments), each tenant with its own hyperparameters and step
count.  Written from the update's definition:

    m <- b1 m + (1 - b1) g
    v <- b2 v + (1 - b2) g^2
    p <- p (1 - lr wd) - (lr / (1 - b1^t)) m / (sqrt(v) / sqrt(1 - b2^t) + eps)

Pinned in ``tests/test_oracle_optim.py`` against torch.optim.AdamW (float64),
the first-step closed form and the zero-gradient decay-only case.
"""
from __future__ import annotations

import numpy as np


def adamw_step(p, g, m, v, step: int, lr: float, beta1: float, beta2: float, eps: float, weight_decay: float):
    """One AdamW update of one tensor; returns new (p, m, v) as fp64 arrays.
    ``step`` is the 1-based index of this update."""
    p = np.asarray(p, np.float64)
    g = np.asarray(g, np.float64)
    m = beta1 * np.asarray(m, np.float64) + (1.0 - beta1) * g
    v = beta2 * np.asarray(v, np.float64) + (1.0 - beta2) * g * g
    bc1 = 1.0 - beta1 ** step
    bc2 = 1.0 - beta2 ** step
    p = p * (1.0 - lr * weight_decay) - (lr / bc1) * m / (np.sqrt(v) / np.sqrt(bc2) + eps)
    return p, m, v


def tenant_step(tensors, hyper: dict, step: int):
    """Apply ``adamw_step`` to every (p, g, m, v) of one tenant."""
    return [adamw_step(p, g, m, v, step, **hyper) for p, g, m, v in tensors]
