"""LSTM recurrence over variable-length sequences, forward and backward.

TEST INFRASTRUCTURE ONLY (see the package docstring).

What is computed (float64 throughout):

* The cell called once per sequence item by the loop of Figure 1
  (``state = rnn_cell(state, item)``), in the standard LSTM form of the
  models of Section 6.1 (Table 2, [51], [21]):
      a = W_x x + W_h h + b            (4H values, gate blocks i, f, g, o)
      i = sigma(a_i), f = sigma(a_f), g = tanh(a_g), o = sigma(a_o)
      c' = f c + i g,   h' = o tanh(c')
* The loop over time with a data-dependent trip count (Section 2.1 "dynamic
  control flow", Section 4.2.1 loops): sequence b is advanced only while
  t < len_b; afterwards its state is carried unchanged and its output is 0.
  The loop runs max(len) times.
* Stacked layers: the output h of layer l at step t is the input of layer
  l+1 at step t.
* The backward pass through time (the differentiation inserted into the
  graph, Section 3.1), derived by hand from the forward equations.
"""
from __future__ import annotations

from typing import List, Optional

import numpy as np


def sigmoid(z):
    with np.errstate(over="ignore"):
        return 1.0 / (1.0 + np.exp(-z))


def cell_forward(x, h, c, Wx, Wh, b):
    """One cell application for a block of rows.

    x [n, I], h [n, H], c [n, H]; returns (h', c', (i, f, g, o))."""
    H = h.shape[1]
    a = x @ Wx.T + h @ Wh.T + b
    i = sigmoid(a[:, 0:H])
    f = sigmoid(a[:, H:2 * H])
    g = np.tanh(a[:, 2 * H:3 * H])
    o = sigmoid(a[:, 3 * H:4 * H])
    c_new = f * c + i * g
    h_new = o * np.tanh(c_new)
    return h_new, c_new, (i, f, g, o)


def cell_backward(dh, dc, c_prev, c_new, gates):
    """Backward of one cell application for a block of rows.

    Given dL/dh' and the gradient dc' carried from the next step, returns
    (da [n, 4H], dc_prev [n, H]).  With tau = tanh(c'):
        do = dh tau;   dc_total = dc + dh o (1 - tau^2)
        di = dc_total g;  dg = dc_total i;  df = dc_total c;  dc_prev = dc_total f
        da_i = di i(1-i), da_f = df f(1-f), da_g = dg (1-g^2), da_o = do o(1-o)
    """
    i, f, g, o = gates
    tau = np.tanh(c_new)
    do = dh * tau
    dct = dc + dh * o * (1.0 - tau * tau)
    di = dct * g
    dg = dct * i
    df = dct * c_prev
    dc_prev = dct * f
    da = np.concatenate([di * i * (1.0 - i), df * f * (1.0 - f),
                         dg * (1.0 - g * g), do * o * (1.0 - o)], axis=1)
    return da, dc_prev


class LayerCache:
    def __init__(self):
        self.steps = []   # per step t: (rows, x_t, h_prev, c_prev, c_new, gates)


def layer_forward(x, lengths, Wx, Wh, b, h0=None, c0=None):
    """Run one LSTM layer over x [T, B, I].

    lengths: int array [B] with 0 <= len_b <= T, or None (all T).
    Returns y [T, B, H], hT [B, H], cT [B, H], cache."""
    T, B, _ = x.shape
    H = Wh.shape[1]
    lengths = np.full(B, T, dtype=np.int64) if lengths is None else np.asarray(lengths)
    h = np.zeros((B, H)) if h0 is None else np.array(h0, dtype=np.float64)
    c = np.zeros((B, H)) if c0 is None else np.array(c0, dtype=np.float64)
    y = np.zeros((T, B, H))
    cache = LayerCache()
    trip = int(lengths.max()) if B > 0 else 0
    for t in range(trip):
        rows = np.nonzero(lengths > t)[0]          # sequences still running
        h_prev, c_prev = h[rows], c[rows]
        h_new, c_new, gates = cell_forward(x[t, rows], h_prev, c_prev, Wx, Wh, b)
        h[rows] = h_new
        c[rows] = c_new
        y[t, rows] = h_new                         # finished rows keep y = 0
        cache.steps.append((rows, x[t, rows], h_prev, c_prev, c_new, gates))
    return y, h, c, cache


def layer_backward(cache, Wx, Wh, dy=None, dhT=None, dcT=None, shape=None):
    """Backward of ``layer_forward``.

    dy [T, B, H] is dL/dy (entries at finished positions are ignored: y is
    the constant 0 there); dhT, dcT are dL/dhT and dL/dcT.  ``shape`` is
    (T, B, I, H).  Returns dx [T, B, I], dh0, dc0, dWx, dWh, db."""
    T, B, I, H = shape
    dh = np.zeros((B, H)) if dhT is None else np.array(dhT, dtype=np.float64)
    dc = np.zeros((B, H)) if dcT is None else np.array(dcT, dtype=np.float64)
    dx = np.zeros((T, B, I))
    dWx = np.zeros_like(Wx, dtype=np.float64)
    dWh = np.zeros_like(Wh, dtype=np.float64)
    db = np.zeros(4 * H)
    for t in range(len(cache.steps) - 1, -1, -1):
        rows, x_t, h_prev, c_prev, c_new, gates = cache.steps[t]
        dh_t = dh[rows] + (dy[t, rows] if dy is not None else 0.0)
        da, dc_prev = cell_backward(dh_t, dc[rows], c_prev, c_new, gates)
        dWx += da.T @ x_t
        dWh += da.T @ h_prev
        db += da.sum(axis=0)
        dx[t, rows] = da @ Wx
        dh[rows] = da @ Wh                         # rows not running pass through
        dc[rows] = dc_prev
    return dx, dh, dc, dWx, dWh, db


def stack_forward(x, lengths, Wx: List, Wh: List, b: List, h0=None, c0=None):
    """Stacked layers; h0, c0 are [L, B, H] or None.  Returns
    (y [T, B, H] of the top layer, hT [L, B, H], cT [L, B, H], caches, ys)."""
    L = len(Wx)
    inp = np.asarray(x, dtype=np.float64)
    hT, cT, caches, ys = [], [], [], []
    for layer in range(L):
        y, h, c, cache = layer_forward(inp, lengths, Wx[layer], Wh[layer], b[layer],
                                       None if h0 is None else h0[layer],
                                       None if c0 is None else c0[layer])
        hT.append(h); cT.append(c); caches.append(cache); ys.append(inp)
        inp = y
    return inp, np.stack(hT), np.stack(cT), caches, ys


def stack_backward(caches, ys, Wx, Wh, dy=None, dhT=None, dcT=None):
    """Backward of ``stack_forward``.  ``ys[l]`` is the input of layer l.
    Returns dx [T, B, I], dh0 [L, B, H], dc0 [L, B, H], dWx, dWh, db lists."""
    L = len(Wx)
    dWx, dWh, db = [None] * L, [None] * L, [None] * L
    dh0, dc0 = [None] * L, [None] * L
    g = dy
    for layer in range(L - 1, -1, -1):
        T, B, I = ys[layer].shape
        H = Wh[layer].shape[1]
        dx, dh, dc, dWx[layer], dWh[layer], db[layer] = layer_backward(
            caches[layer], Wx[layer], Wh[layer], g,
            None if dhT is None else dhT[layer], None if dcT is None else dcT[layer],
            (T, B, I, H))
        dh0[layer], dc0[layer] = dh, dc
        g = dx
    return g, np.stack(dh0), np.stack(dc0), dWx, dWh, db


def carry_state(hT, cT, B_next):
    """Initial state of the next batch from the final state of the previous
    one: the program keeps the recurrent state in ``self.state`` between
    calls (Figure 1).  Rows both batches have continue; rows only the next
    batch has start from 0; rows past the next batch end (a smaller last
    batch, the shape the paper relaxes when its specialized value changes).
    ``hT`` is None for the first batch (all zeros)."""
    if hT is None:
        return None, None
    hT = np.asarray(hT, dtype=np.float64)
    cT = np.asarray(cT, dtype=np.float64)
    L, B_prev, H = hT.shape
    h0 = np.zeros((L, B_next, H))
    c0 = np.zeros((L, B_next, H))
    n = min(B_prev, B_next)
    h0[:, :n] = hT[:, :n]
    c0[:, :n] = cT[:, :n]
    return h0, c0
