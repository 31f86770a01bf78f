"""Pins of the parameter-update oracle (oracle/sgd.py) against what does not
depend on it: torch's own gradient clipping and SGD step in float64 on the
CPU, a closed form of the norm, the invariants of a clipped step, and the
all-or-nothing rule for non-finite gradients (Section 4.2.3)."""
import math

import numpy as np
import pytest
import torch

from oracle import sgd


def _tensors(seed, shapes, scale=1.0):
    rng = np.random.default_rng(seed)
    p = [rng.uniform(-1, 1, s) for s in shapes]
    g = [scale * rng.normal(0, 1, s) for s in shapes]
    return p, g


def _torch_step(p, g, lr, max_norm):
    tp = [torch.tensor(x, dtype=torch.float64, requires_grad=True) for x in p]
    for t, x in zip(tp, g):
        t.grad = torch.tensor(x, dtype=torch.float64)
    norm = None
    if max_norm is not None:
        norm = float(torch.nn.utils.clip_grad_norm_(tp, max_norm))
    opt = torch.optim.SGD(tp, lr=lr)
    opt.step()
    return [t.detach().numpy() for t in tp], norm


SHAPES = [(64, 32), (32,), (0,), (7, 5, 3), (1,)]


@pytest.mark.parametrize("scale,max_norm", [(1.0, 5.0), (10.0, 1.0), (0.01, 5.0), (3.0, 0.25)])
def test_matches_torch_clip_and_sgd(scale, max_norm):
    p, g = _tensors(3, SHAPES, scale)
    ref, tnorm = _torch_step(p, g, lr=0.1, max_norm=max_norm)
    new, norm, s, applied = sgd.sgd_clip_update(p, g, 0.1, max_norm)
    assert applied
    assert norm == pytest.approx(tnorm, rel=1e-14)
    for a, b in zip(new, ref):
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-14)


@pytest.mark.parametrize("max_norm", [0.0, -1.0, math.inf])
def test_clipping_off_is_plain_sgd(max_norm):
    p, g = _tensors(4, SHAPES, 50.0)
    ref, _ = _torch_step(p, g, lr=0.05, max_norm=None)
    new, _, s, applied = sgd.sgd_clip_update(p, g, 0.05, max_norm)
    assert applied and s == 1.0
    for a, b in zip(new, ref):
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-14)


def test_norm_closed_form():
    # c in every entry of n entries: norm = |c| sqrt(n)
    g = [np.full((30, 7), -0.75), np.full((11,), -0.75), np.zeros((0, 4))]
    n = 30 * 7 + 11
    assert sgd.global_norm(g) == pytest.approx(0.75 * math.sqrt(n), rel=1e-15)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_clipped_step_invariants(seed):
    p, g = _tensors(seed, SHAPES, 7.0)
    lr, max_norm = 0.3, 2.0
    new, norm, s, _ = sgd.sgd_clip_update(p, g, lr, max_norm)
    step = np.concatenate([(a - b).ravel() for a, b in zip(p, new)])
    gv = np.concatenate([np.ravel(x) for x in g])
    # the step is -lr s g: same direction as g, norm lr * min(norm, ~max_norm)
    assert np.linalg.norm(step) <= lr * max_norm * (1 + 1e-12)
    assert np.linalg.norm(step) == pytest.approx(lr * max_norm * norm / (norm + sgd.CLIP_EPS), rel=1e-12)
    cos = float(step @ gv) / (np.linalg.norm(step) * np.linalg.norm(gv))
    assert cos == pytest.approx(1.0, abs=1e-12)


@pytest.mark.parametrize("bad", [math.nan, math.inf, -math.inf])
def test_non_finite_gradient_changes_nothing(bad):
    p, g = _tensors(5, SHAPES, 1.0)
    g[3] = g[3].copy()
    g[3][2, 1, 0] = bad
    new, norm, s, applied = sgd.sgd_clip_update(p, g, 0.1, 1.0)
    assert not applied and s == 0.0 and not math.isfinite(norm)
    for a, b in zip(new, p):
        assert np.array_equal(a, b)
