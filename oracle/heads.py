"""Embedding lookup, output heads and losses, forward and backward.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The model programs end with ``compute_loss(outputs)`` (Figure 1); the losses
below are the ones of the five training-step workloads.  Each function
returns the scalar loss and the gradients of its inputs, derived by hand.
"""
from __future__ import annotations

import numpy as np


def embed_forward(E, ids):
    """Row lookup x[r] = E[ids[r]] for an int array of any shape."""
    return np.asarray(E, dtype=np.float64)[np.asarray(ids, dtype=np.int64)]


def embed_backward(V, dx, ids):
    """dE[v] = sum of dx[r] over the rows r with ids[r] == v (0 elsewhere)."""
    ids = np.asarray(ids, dtype=np.int64).reshape(-1)
    dx = np.asarray(dx, dtype=np.float64).reshape(ids.shape[0], -1)
    dE = np.zeros((V, dx.shape[1]))
    for r in range(ids.shape[0]):
        dE[ids[r]] += dx[r]
    return dE


def sumsq(h):
    """L = sum of h^2 over all entries; dL/dh = 2 h."""
    h = np.asarray(h, dtype=np.float64)
    return float(np.sum(h * h)), 2.0 * h


def mean_all(h):
    """L = mean of all entries; dL/dh = 1 / count."""
    h = np.asarray(h, dtype=np.float64)
    return float(h.mean()), np.full(h.shape, 1.0 / h.size)


def log_softmax(z):
    m = z.max(axis=1, keepdims=True)
    s = z - m
    return s - np.log(np.exp(s).sum(axis=1, keepdims=True))


def softmax_xent(h, W, b, targets):
    """Mean softmax cross-entropy of logits = h W^T + b against integer
    targets.  h [R, H], W [V, H], b [V], targets [R].

    Returns (loss, dh, dW, db, logits)."""
    h = np.asarray(h, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    R = h.shape[0]
    t = np.asarray(targets, dtype=np.int64)
    logits = h @ W.T + b
    lp = log_softmax(logits)
    loss = float(-lp[np.arange(R), t].mean())
    dlogits = np.exp(lp)
    dlogits[np.arange(R), t] -= 1.0
    dlogits /= R
    return loss, dlogits @ W, dlogits.T @ h, dlogits.sum(axis=0), logits


def linear_mse(h, W, b, target):
    """L = mean over all entries of (h W^T + b - target)^2.
    h [R, H], W [P, H], b [P], target [R, P].

    Returns (loss, dh, dW, db, y)."""
    h = np.asarray(h, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    y = h @ W.T + b
    d = y - np.asarray(target, dtype=np.float64)
    loss = float(np.mean(d * d))
    dy = 2.0 * d / d.size
    return loss, dy @ W, dy.T @ h, dy.sum(axis=0), y
