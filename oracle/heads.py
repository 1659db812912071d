"""Tenant-private action heads: forward, loss, weight gradients, in fp64 --
oracle (test infrastructure only).

Sec. 5.2: after the shared forward, features are split for tenant-private
loss computation and backward passes; App. A.3 (actor consumption): each
optimizer microbatch holds one tenant-schema group, and losses and
gradients are never averaged across tenants.  Hence every function here
sees exactly one tenant's rows.

Readings: an MLP head ``y = W_L gelu(... gelu(W_1 p + b_1) ...) + b_L``
(tanh GELU between layers, none after the last), output reshaped to
[chunk, action_dim]; the loss is the tenant's mean squared error over all
of its n * chunk * action_dim elements; gradients are w.r.t. the head's
weights and biases only (the backbone is frozen, so no gradient flows into
the shared features).
"""
from __future__ import annotations

from typing import List, Sequence, Tuple

import numpy as np

from .backbone import gelu, gelu_grad


def head_forward(P: np.ndarray, layers: Sequence[Tuple[np.ndarray, np.ndarray]]):
    """Returns (pre-activations Z_k, layer inputs X_k, output Y)."""
    X = [np.asarray(P, np.float64)]
    Z = []
    for k, (W, b) in enumerate(layers):
        z = X[-1] @ np.asarray(W, np.float64).T + np.asarray(b, np.float64)
        Z.append(z)
        if k + 1 < len(layers):
            X.append(gelu(z))
    return Z, X, Z[-1]


def mse_loss(Y: np.ndarray, target: np.ndarray) -> Tuple[float, np.ndarray]:
    """Mean squared error over every element and its gradient dL/dY."""
    t = np.asarray(target, np.float64).reshape(Y.shape)
    diff = Y - t
    n = diff.size
    return float(np.sum(diff * diff) / n), 2.0 * diff / n


def head_backward(layers, Z, X, dY) -> List[Tuple[np.ndarray, np.ndarray]]:
    """Weight and bias gradients of every layer, by the chain rule."""
    grads: List[Tuple[np.ndarray, np.ndarray]] = [None] * len(layers)
    dz = dY
    for k in range(len(layers) - 1, -1, -1):
        grads[k] = (dz.T @ X[k], dz.sum(axis=0))
        if k > 0:
            dh = dz @ np.asarray(layers[k][0], np.float64)
            dz = dh * gelu_grad(Z[k - 1])
    return grads


def tenant_step(P: np.ndarray, layers, target: np.ndarray) -> dict:
    """Forward, loss and gradients of one tenant's head over its rows P."""
    Z, X, Y = head_forward(P, layers)
    loss, dY = mse_loss(Y, target)
    return {"actions": Y, "loss": loss, "grads": head_backward(layers, Z, X, dY)}
