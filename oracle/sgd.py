"""Parameter update of the training step: SGD whose step is scaled down when
the gradients' global L2 norm exceeds a threshold.

TEST INFRASTRUCTURE ONLY (see the package docstring).

JANUS inserts the parameter update into the generated graph after the
operations of automatic differentiation (Section 3.1, symbolic graph
generation); Figure 1 calls it as ``optimize(...)`` once per training step.
The paper names no optimizer.  The reading taken here is plain SGD,
p <- p - lr * s * g, with s = min(1, max_norm / (norm + 1e-6)) where norm is
the L2 norm over all gradients of the step (the clipping coefficient of
``torch.nn.utils.clip_grad_norm_``), and s = 1 when clipping is off
(max_norm <= 0 or infinite).

Model state changes all-or-nothing (Section 4.2.3): when the norm is not
finite, no parameter changes.  Everything here is float64.
"""
from __future__ import annotations

import math

import numpy as np

CLIP_EPS = 1e-6


def global_norm(grads) -> float:
    """L2 norm over all entries of all gradients (tensors in order)."""
    total = 0.0
    for g in grads:
        v = np.asarray(g, dtype=np.float64).ravel()
        total += float(np.dot(v, v))
    return math.sqrt(total)


def clip_scale(norm: float, max_norm: float) -> float:
    """Scale applied to the step: 0 when the norm is not finite (no update),
    1 when clipping is off or the norm is within the threshold."""
    if not math.isfinite(norm):
        return 0.0
    if not (max_norm > 0.0) or not math.isfinite(max_norm):
        return 1.0
    return min(1.0, max_norm / (norm + CLIP_EPS))


def sgd_clip_update(params, grads, lr: float, max_norm: float):
    """Returns (new parameters as float64 arrays, norm, scale, applied)."""
    norm = global_norm(grads)
    if not math.isfinite(norm):
        return [np.array(p, dtype=np.float64) for p in params], norm, 0.0, False
    s = clip_scale(norm, max_norm)
    new = [np.asarray(p, dtype=np.float64) - lr * s * np.asarray(g, dtype=np.float64)
           for p, g in zip(params, grads)]
    return new, norm, s, True
