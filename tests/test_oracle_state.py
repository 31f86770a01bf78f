"""Pins of the state carried between batches (oracle.lstm.carry_state):
running T1 steps, carrying the state and running T2 more steps must give
exactly the outputs of one run over T1 + T2 steps (the recurrence only sees
h and c), also with variable lengths; a row that ends in the first part
keeps its final state through the second; and the ragged-batch rules
(rows continue, start from 0 or end) hold element by element."""
import numpy as np
import pytest

from oracle import lstm


def _params(rng, L, I, H):
    a = 1.0 / np.sqrt(H)
    Wx = [rng.uniform(-a, a, (4 * H, I if l == 0 else H)) for l in range(L)]
    Wh = [rng.uniform(-a, a, (4 * H, H)) for l in range(L)]
    b = [rng.uniform(-a, a, (4 * H,)) for l in range(L)]
    return Wx, Wh, b


@pytest.mark.parametrize("ragged", [False, True])
def test_split_run_equals_one_run(ragged):
    rng = np.random.default_rng(5)
    L, I, H, B, T1, T2 = 2, 6, 8, 5, 4, 3
    Wx, Wh, b = _params(rng, L, I, H)
    x = rng.normal(0, 1, (T1 + T2, B, I))
    h0 = rng.uniform(-0.5, 0.5, (L, B, H))
    c0 = rng.uniform(-0.5, 0.5, (L, B, H))
    lens = rng.integers(0, T1 + T2 + 1, B) if ragged else None
    y, hT, cT, _, _ = lstm.stack_forward(x, lens, Wx, Wh, b, h0, c0)
    l1 = None if lens is None else np.minimum(lens, T1)
    l2 = None if lens is None else np.maximum(lens - T1, 0)
    y1, hA, cA, _, _ = lstm.stack_forward(x[:T1], l1, Wx, Wh, b, h0, c0)
    h1, c1 = lstm.carry_state(hA, cA, B)
    y2, hB, cB, _, _ = lstm.stack_forward(x[T1:], l2, Wx, Wh, b, h1, c1)
    np.testing.assert_allclose(np.concatenate([y1, y2]), y, rtol=0, atol=1e-15)
    np.testing.assert_allclose(hB, hT, rtol=0, atol=1e-15)
    np.testing.assert_allclose(cB, cT, rtol=0, atol=1e-15)


@pytest.mark.parametrize("B_prev,B_next", [(6, 4), (4, 6), (5, 5)])
def test_ragged_batch_rows(B_prev, B_next):
    rng = np.random.default_rng(6)
    hT = rng.normal(0, 1, (2, B_prev, 3))
    cT = rng.normal(0, 1, (2, B_prev, 3))
    h0, c0 = lstm.carry_state(hT, cT, B_next)
    assert h0.shape == (2, B_next, 3)
    for r in range(B_next):
        if r < B_prev:
            assert np.array_equal(h0[:, r], hT[:, r]) and np.array_equal(c0[:, r], cT[:, r])
        else:
            assert not h0[:, r].any() and not c0[:, r].any()


def test_first_batch_starts_from_zero():
    assert lstm.carry_state(None, None, 4) == (None, None)
